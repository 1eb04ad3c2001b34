// soma_api.hip -- C ABI of the SOMA SPSA hot path on gfx950 (see soma.h).
//
// A step of the stacked LSTM enqueues, per chunk of directions (all experts
// at once, both signs of each direction side by side):
//   k_fold          layer-1 gate inputs per byte value (embedding times the
//                   input weights, perturbed rows formed on the fly)
//   per layer l:    for l >= 2, h^(l-1) times the input weights, weights
//                   held in registers: k_proj_dma where the previous layer's
//                   k_rec_xchg stored its h pre-split (B % 16 = 0,
//                   H = 128, 256, 512), else k_proj_stream; then the
//                   recurrence:
//                   k_rec_xchg (one cooperative launch, four row tiles of
//                   the batch pipelined, h exchanged pre-split by LDS DMA)
//                   or k_rec_persist (one cooperative launch; blocks of a
//                   group share the recurrent weights and stage h each step),
//                   k_rec_local (H = 64: one block per perturbed model, h in
//                   LDS, for L = 1 with the head and cross entropy fused), or
//                   one launch per time step (k_rec_step_split / k_rec_step)
//   k_head_stream + k_ce_combine   head and softmax cross entropy (unless
//                   fused into the recurrence)
//   k_loss_reduce   fixed-order sums -> L_{e,j,+-} (fp64 means)
// and then, once for the step:
//   k_coef          c_{e,j} (independent) or dF_j / (2 eps_e P) (summed)
//   k_update / k_update_adam   theta -= lr sum_j c_j z_j, regenerating z_j
// The paper's width-32 body (SOMA_ARCH_BODY) runs its whole perturbed
// forward in k_body (soma_body.hpp); the wide controls' body
// (SOMA_ARCH_WIDE) forms each slot's perturbed weights once (k_wide_form)
// and runs split-fp16 products (k_wide_mm), LayerNorms and the decoder
// (soma_wide.hpp) around k_rec_persist on the pre-formed weights.  Every kernel that forms split fp16
// weights checks their range and the persistent recurrence bounds its waits:
// either failure sets a sticky flag, and the step is then aborted on the
// device (NaN losses, theta untouched).  The step writes theta only in the
// update kernel, after every loss exists.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "soma.h"
#include "soma_kernels.hpp"
#include "soma_body.hpp"
#include "soma_wide.hpp"

namespace {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int ok() {
  g_last_error.clear();
  return SOMA_OK;
}

constexpr size_t kAlign = 256;
constexpr int kMaxGroups = 1024;              // persistent-recurrence groups (counters in the workspace)
constexpr unsigned kSpinLimit = 1u << 20;     // polls (~1 s) before a persistent launch gives up
constexpr size_t kAutoBudget = size_t(64) << 30;  // automatic pair_chunk keeps the workspace below this

size_t round_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Layout {
  int64_t d = 0;
  int64_t off_layer[64] = {};
  int64_t off_head = 0;
  int pc = 0;          // directions per pass
  int row_tiles = 0;   // head tiles per slot
  size_t sync = 0, rates = 0, coef = 0, lossd = 0, part = 0, U = 0, gin = 0, hseq = 0, cst = 0, hpart = 0, htgt = 0,
         total = 0;
  // the exchange recurrence: published h ring, flags and placement counters
  size_t xch = 0, xch_bytes = 0;
  // the paper's body (SOMA_ARCH_BODY) and the wide controls' body
  // (SOMA_ARCH_WIDE): decoder inputs, log-sum-exps and delta-rule partials
  // of an evaluation pass
  size_t fdec = 0, lse = 0, dpart = 0;
  int delta_chunks = 0;
  // SOMA_ARCH_WIDE: pre-formed weights and the residual stream per slot
  // (hseq holds the normalised rows and the recurrence's h, gin the gate
  // inputs and the MLP hidden layer)
  size_t wform = 0, xres = 0;
};

// Directions per update: n_pairs per accumulation batch, accum batches.
int dirs(const soma_config& c) { return c.n_pairs * (c.accum > 1 ? c.accum : 1); }

static_assert(SOMA_PERTURB_EMBEDDING == soma::kGroupEmb && SOMA_PERTURB_LSTM == soma::kGroupLstm &&
                  SOMA_PERTURB_HEAD == soma::kGroupHead,
              "the mask bits of the boundary are the kernels' group bits");

// The perturbed parameter groups of a configuration (0 in the config: all).
unsigned group_mask(const soma_config& c) { return c.perturb_mask ? c.perturb_mask : unsigned(SOMA_PERTURB_ALL); }

int64_t param_count_of(const soma_config& c) {
  if (c.arch == SOMA_ARCH_BODY) return c.n_layers * soma::body_block(c.hidden) + c.hidden;
  if (c.arch == SOMA_ARCH_WIDE)
    return 16LL * c.n_layers * c.hidden * c.hidden + (2LL * c.n_layers + 1) * c.hidden + 2LL * c.embed * c.hidden;
  int64_t d = int64_t(SOMA_VOCAB) * c.embed;
  for (int l = 0; l < c.n_layers; ++l)
    d += 4LL * c.hidden * ((l == 0 ? c.embed : c.hidden) + c.hidden);
  return d + int64_t(SOMA_VOCAB) * c.hidden;
}

int validate(const soma_config* c) {
  if (!c) return fail(SOMA_EINVAL, "config is NULL");
  if (c->n_experts < 1 || c->n_layers < 1 || c->n_pairs < 1 || c->batch < 1)
    return fail(SOMA_ESHAPE, "n_experts, n_layers, n_pairs and batch must be >= 1");
  if (c->n_layers > 64) return fail(SOMA_ESHAPE, "at most 64 layers");
  if (c->seq_len < 2) return fail(SOMA_ESHAPE, "seq_len must be >= 2 (T-1 targets)");
  if (c->arch == SOMA_ARCH_WIDE) {
    if (c->embed != soma::kWideHeadWidth || c->hidden < 4 || c->hidden > 512)
      return fail(SOMA_ESHAPE, "the wide body needs embed = %d and 4 <= hidden <= 512 (got %d, %d)",
                  soma::kWideHeadWidth, c->embed, c->hidden);
  } else if (c->embed < 16 || c->embed % 16 || c->hidden < 16 || c->hidden % 16) {
    return fail(SOMA_ESHAPE, "embed and hidden must be positive multiples of 16 (got %d, %d)",
                c->embed, c->hidden);
  }
  if (c->loss_mode != SOMA_LOSS_INDEPENDENT && c->loss_mode != SOMA_LOSS_SUMMED)
    return fail(SOMA_EINVAL, "loss_mode must be 0 (independent) or 1 (summed)");
  if (c->accum < 0) return fail(SOMA_ESHAPE, "accum must be >= 0 (0 or 1: one batch)");
  if (int64_t(c->n_pairs) * (c->accum > 1 ? c->accum : 1) >= (int64_t(1) << 24))
    return fail(SOMA_ESHAPE, "n_pairs * accum must stay below 2^24");
  if (c->pair_chunk < 0 || c->pair_chunk > dirs(*c))
    return fail(SOMA_ESHAPE, "pair_chunk must be in [0, n_pairs * accum]");
  if (c->flags & ~(SOMA_FLAG_PER_STEP_RECURRENCE | SOMA_FLAG_TILED_WEIGHTS | SOMA_FLAG_STAGED_RECURRENCE |
                   SOMA_FLAG_FP32_SEQUENCE))
    return fail(SOMA_EINVAL, "unknown flags");
  if (c->probe != SOMA_PROBE_GAUSSIAN && c->probe != SOMA_PROBE_SPARSE_RADEMACHER &&
      c->probe != SOMA_PROBE_RADEMACHER)
    return fail(SOMA_EINVAL, "probe must be 0 (Gaussian), 1 (sparse Rademacher) or 2 (Rademacher)");
  if (c->arch != SOMA_ARCH_LSTM && c->arch != SOMA_ARCH_BODY && c->arch != SOMA_ARCH_WIDE)
    return fail(SOMA_EINVAL, "arch must be 0 (stacked LSTM), 1 (the paper's body) or 2 (the wide controls' body)");
  if (c->perturb_mask > SOMA_PERTURB_ALL)
    return fail(SOMA_EINVAL, "perturb_mask must be a combination of SOMA_PERTURB_* bits (got %u)", c->perturb_mask);
  if (c->arch != SOMA_ARCH_LSTM && !(group_mask(*c) & SOMA_PERTURB_LSTM))
    return fail(SOMA_EINVAL, "the body's parameters are one group: perturb_mask must include SOMA_PERTURB_LSTM");
  if (c->arch == SOMA_ARCH_BODY) {
    if (c->embed != c->hidden || (c->hidden != 16 && c->hidden != 32) || c->n_layers > 2)
      return fail(SOMA_ESHAPE, "the body needs embed = hidden in {16, 32} and n_layers in {1, 2} (got %d, %d, %d)",
                  c->embed, c->hidden, c->n_layers);
    if (c->flags) return fail(SOMA_EINVAL, "flags select stacked-LSTM kernels and must be 0 for the body");
    const int64_t blocks = int64_t((c->batch + soma::kBodySeqs - 1) / soma::kBodySeqs) * c->n_experts * 2 *
                           (int64_t(c->n_pairs) * (c->accum > 1 ? c->accum : 1));
    if (blocks >= (int64_t(1) << 31)) return fail(SOMA_ESHAPE, "too many body blocks in one step");
  }
  if (c->arch == SOMA_ARCH_WIDE) {
    if (c->flags) return fail(SOMA_EINVAL, "flags select stacked-LSTM kernels and must be 0 for the wide body");
    if (c->batch > 64) return fail(SOMA_ESHAPE, "the wide body's recurrence takes batch <= 64 (got %d)", c->batch);
    const int64_t dp = soma::wide_padded(c->hidden);
    if (int64_t(c->seq_len - 1) * c->batch * 4 * dp * int64_t(sizeof(float)) >= (int64_t(1) << 31))
      return fail(SOMA_ESHAPE, "one slot's gate inputs, B (T-1) 4 d_p floats, must stay below 2^31 bytes");
  }
  const int64_t d = param_count_of(*c);
  if (d >= (int64_t(1) << 40)) return fail(SOMA_ESHAPE, "expert too large (d >= 2^40)");
  const int64_t rows = int64_t(c->seq_len - 1) * c->batch;
  if (rows >= (int64_t(1) << 31)) return fail(SOMA_ESHAPE, "B (T-1) must stay below 2^31");
  return SOMA_OK;
}

Layout layout_for_body(const soma_config& c, int pc) {
  Layout L;
  L.d = param_count_of(c);
  L.pc = pc;
  const size_t N = c.n_experts, R = size_t(c.seq_len - 1) * c.batch, dm = c.hidden;
  L.row_tiles = (c.batch + soma::kBodySeqs - 1) / soma::kBodySeqs;
  L.delta_chunks = int((R + soma::kDeltaChunk - 1) / soma::kDeltaChunk);
  const size_t slots = N * size_t(pc) * 2;
  size_t at = 0;
  L.sync = at; at += round_up(sizeof(unsigned) * (kMaxGroups + 1));
  L.rates = at; at += round_up(sizeof(float) * 2 * N);
  L.coef = at; at += round_up(sizeof(float) * N * dirs(c));
  L.lossd = at; at += round_up(sizeof(double) * N * dirs(c) * 2);
  L.part = at; at += round_up(sizeof(double) * slots * L.row_tiles);
  L.fdec = at; at += round_up(sizeof(float) * N * R * dm);
  L.lse = at; at += round_up(sizeof(float) * N * R);
  L.dpart = at; at += round_up(sizeof(float) * N * L.delta_chunks * SOMA_VOCAB * dm);
  L.total = at;
  return L;
}

// The wide controls' body: per slot of a pass its pre-formed weights, the
// per-byte input projection U, the residual stream x, the normalised rows
// (shared with the recurrence's h: each reader is done before the next
// writer) and the gate inputs (shared with the MLP hidden layer).
Layout layout_for_wide(const soma_config& c, int pc) {
  Layout L;
  L.d = param_count_of(c);
  L.pc = pc;
  const size_t N = c.n_experts, R = size_t(c.seq_len - 1) * c.batch, dp = soma::wide_padded(c.hidden);
  L.row_tiles = int((R + soma::kWideHeadRows - 1) / soma::kWideHeadRows);
  L.delta_chunks = int((R + soma::kDeltaChunk - 1) / soma::kDeltaChunk);
  const size_t slots = std::max(N * size_t(pc) * 2, N);
  const size_t form = size_t(soma::wide_form_layout(int(dp), c.n_layers).total);
  const size_t E = soma::kWideHeadWidth;
  size_t at = 0;
  L.sync = at; at += round_up(sizeof(unsigned) * (kMaxGroups + 1));
  L.rates = at; at += round_up(sizeof(float) * 2 * N);
  L.coef = at; at += round_up(sizeof(float) * N * dirs(c));
  L.lossd = at; at += round_up(sizeof(double) * N * dirs(c) * 2);
  L.part = at; at += round_up(sizeof(double) * slots * L.row_tiles);
  L.wform = at; at += round_up(sizeof(float) * slots * form);
  L.U = at; at += round_up(sizeof(float) * slots * SOMA_VOCAB * dp);
  L.xres = at; at += round_up(sizeof(float) * slots * R * dp);
  L.hseq = at; at += round_up(sizeof(float) * slots * R * dp);
  L.gin = at; at += round_up(sizeof(float) * slots * R * 4 * dp);
  L.fdec = at; at += round_up(sizeof(float) * N * R * E);
  L.lse = at; at += round_up(sizeof(float) * N * R);
  L.dpart = at; at += round_up(sizeof(float) * N * L.delta_chunks * SOMA_VOCAB * E);
  L.total = at;
  return L;
}

bool stream_weights(const soma_config& c);
bool local_embedding(const soma_config& c);

// The pipelined exchange recurrence (k_rec_xchg) runs for the stacked LSTM
// with four row tiles (48 < B <= 64) at the widths it has been validated on:
// H = 128, 256, 512 and 704.  At H = 192 a launch faulted the device, with no
// cause found in the kernel's indexing; that width and the others not yet
// validated take the staged recurrence.  Whether it runs also depends on the
// device (compute units per XCD).
bool xchg_shape(const soma_config& c) {
  const int H = c.hidden;
  return c.arch == SOMA_ARCH_LSTM && c.batch > 48 && c.batch <= 64 &&
         (H == 128 || H == 256 || H == 512 || H == 704) && !(c.flags & SOMA_FLAG_PER_STEP_RECURRENCE) &&
         !(c.flags & SOMA_FLAG_STAGED_RECURRENCE);
}

int xchg_tiles(int) { return soma::kXchgTiles; }

// Groups the exchange recurrence can have at width H: 8 XCDs of at most 64
// compute units, one block each, H / 32 blocks a group.
int xchg_max_groups(int H) { return std::min(soma::kXchgMaxGroups, 8 * 64 / (H / 32)); }

// Ring of two published steps per group: 16 NB rows x H, split (4 bytes a value).
size_t xchg_ring_bytes(const soma_config& c) {
  return size_t(xchg_max_groups(c.hidden)) * 2 * 16 * xchg_tiles(c.batch) * c.hidden * 4;
}

// Flags, then the per-compute-unit and per-rank placement counters.
int xchg_counter_words() { return soma::kXchgMaxGroups * soma::kXchgFlagWords + soma::kXchgCuSlots + 8 * soma::kXchgMaxPerCu; }

Layout layout_for(const soma_config& c, int pc) {
  if (c.arch == SOMA_ARCH_BODY) return layout_for_body(c, pc);
  if (c.arch == SOMA_ARCH_WIDE) return layout_for_wide(c, pc);
  Layout L;
  L.d = param_count_of(c);
  int64_t off = int64_t(SOMA_VOCAB) * c.embed;
  for (int l = 0; l < c.n_layers; ++l) {
    L.off_layer[l] = off;
    off += 4LL * c.hidden * ((l == 0 ? c.embed : c.hidden) + c.hidden);
  }
  L.off_head = off;
  L.pc = pc;
  const size_t N = c.n_experts, H = c.hidden, B = c.batch, R = size_t(c.seq_len - 1) * B;
  L.row_tiles = int((R + 63) / 64);
  const size_t slots = N * size_t(pc) * 2;
  size_t at = 0;
  L.sync = at; at += round_up(sizeof(unsigned) * (kMaxGroups + 1));
  L.rates = at; at += round_up(sizeof(float) * 2 * N);            // eps[N], lr[N] of a scalar-rate step
  L.coef = at; at += round_up(sizeof(float) * N * dirs(c));
  L.lossd = at; at += round_up(sizeof(double) * N * dirs(c) * 2);
  L.part = at; at += round_up(sizeof(double) * slots * L.row_tiles);
  // U: the perturbed slots' folded inputs, or only the N unperturbed ones
  // of an evaluation where the H = 64 recurrence forms them in the block.
  const size_t uslots = local_embedding(c) ? N : slots;
  L.U = at;    at += round_up(sizeof(float) * uslots * SOMA_VOCAB * 4 * H);
  L.hseq = at; at += round_up(sizeof(float) * slots * R * H);
  L.cst = at;  at += round_up(sizeof(float) * slots * B * H);
  // Head partials of k_head_stream only (H > 128; k_head_fused keeps its own).
  const size_t hslots = stream_weights(c) && H > 128 ? slots : 0;
  L.hpart = at; at += round_up(sizeof(float) * 2 * hslots * 2 * R);   // (m, s) per vocabulary half
  L.htgt = at; at += round_up(sizeof(float) * hslots * R);
  L.gin = at;
  if (c.n_layers > 1) at += round_up(sizeof(float) * slots * R * 4 * H);
  if (xchg_shape(c)) {
    L.xch = at;
    L.xch_bytes = xchg_ring_bytes(c);
    at += round_up(L.xch_bytes + sizeof(unsigned) * xchg_counter_words());
  }
  L.total = at;
  return L;
}

int choose_chunk(const soma_config& c) {
  if (c.pair_chunk > 0) return c.pair_chunk;
  if (c.arch == SOMA_ARCH_BODY) return dirs(c);   // no per-direction buffers
  int pc = dirs(c);
  while (pc > 1 && layout_for(c, pc).total > kAutoBudget) --pc;
  if (c.arch == SOMA_ARCH_WIDE) {
    // Chunks of equal size: each chunk's recurrence runs its jobs in rounds
    // of the concurrent groups, and a small last chunk would leave most of
    // them idle.
    const int n = (dirs(c) + pc - 1) / pc;
    pc = (dirs(c) + n - 1) / n;
  }
  return pc;
}

}  // namespace

enum Phase { kPhaseStart = -1, kPhaseFold, kPhaseProj, kPhaseRec, kPhaseHead, kPhaseReduce, kPhaseUpdate };

struct soma_ctx {
  soma_config cfg;
  Layout lay;
  char* ws;
  size_t ws_bytes;
  bool have_coef;
  // phase timing
  bool timing;
  unsigned spin_limit;              // polls per group barrier of the persistent recurrence
  bool have_times;
  // device facts for the persistent recurrence
  int coop_blocks;                  // co-resident k_rec_persist blocks (0: path unavailable)
  int xchg_per_cu;                  // co-resident k_rec_xchg blocks per compute unit (0: unavailable)
  int xchg_cus_per_xcd;
  int xchg_pad_lds;                 // unused dynamic LDS per block that caps its occupancy at xchg_per_cu
  float* head;                      // SOMA_ARCH_BODY, SOMA_ARCH_WIDE: the tied matrix E of expert 0 (caller owned)
  int64_t head_stride;              // floats from one expert's E to the next
  std::vector<hipEvent_t> events;   // pool, grows on demand
  std::vector<int> phase;           // phase closed by events[i]
  size_t nmarks;
  int rec_launches, proj_launches, xchg_launches;
};

namespace soma {

// z values for a contiguous index range (probe dump).
__global__ void k_gaussian(uint64_t seed, uint64_t step, uint32_t pair, uint64_t k0, uint64_t count,
                           float* out) {
  const uint64_t q = (k0 >> 2) + blockIdx.x * uint64_t(blockDim.x) + threadIdx.x;
  const uint64_t qend = (k0 + count + 3) >> 2;
  if (q >= qend) return;
  const float4 z = gauss_quad(stream_key(seed, step), pair, static_cast<uint32_t>(step), q);
  const float zz[4] = {z.x, z.y, z.z, z.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint64_t k = 4 * q + i;
    if (k >= k0 && k < k0 + count) out[k - k0] = zz[i];
  }
}

__global__ void k_probe(int law, uint64_t seed, uint64_t step, uint32_t pair, uint64_t k0, uint64_t count,
                        float* out) {
  const uint64_t q = (k0 >> 2) + blockIdx.x * uint64_t(blockDim.x) + threadIdx.x;
  const uint64_t qend = (k0 + count + 3) >> 2;
  if (q >= qend) return;
  const float4 z = probe_quad(law, stream_key(seed, step), pair, static_cast<uint32_t>(step), 4 * q);
  const float zz[4] = {z.x, z.y, z.z, z.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint64_t k = 4 * q + i;
    if (k >= k0 && k < k0 + count) out[k - k0] = zz[i];
  }
}

__global__ void k_philox(const uint32_t* ctr, const uint32_t* key, uint32_t* out, uint64_t n) {
  const uint64_t i = blockIdx.x * uint64_t(blockDim.x) + threadIdx.x;
  if (i >= n) return;
  const uint4 r = philox4x32_10(make_uint4(ctr[4 * i], ctr[4 * i + 1], ctr[4 * i + 2], ctr[4 * i + 3]),
                                make_uint2(key[2 * i], key[2 * i + 1]));
  out[4 * i] = r.x;
  out[4 * i + 1] = r.y;
  out[4 * i + 2] = r.z;
  out[4 * i + 3] = r.w;
}

__global__ void k_box_muller(const uint32_t* wa, const uint32_t* wb, float* za, float* zb, uint64_t n) {
  const uint64_t i = blockIdx.x * uint64_t(blockDim.x) + threadIdx.x;
  if (i >= n) return;
  const float2 z = box_muller(wa[i], wb[i]);
  za[i] = z.x;
  zb[i] = z.y;
}

// L[e][j0 + jl][s] = (sum over tiles in order) / (B (T-1)), accumulated in
// fp64; the fp64 mean is kept (lossd) so that the antithetic difference is
// taken before any rounding to fp32.  One thread per slot.
__global__ void k_loss_reduce(const double* part, int row_tiles, int N, int pcs, int PC, int NS,
                              int P, int j0, double inv_rows, float* losses, double* lossd,
                              const unsigned* err) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= N * pcs * NS) return;
  const int s = i % NS, jl = (i / NS) % pcs, e = i / (NS * pcs);
  const double* p = part + ((int64_t(e) * PC + jl) * NS + s) * row_tiles;
  double tot = 0.0;
  for (int k = 0; k < row_tiles; ++k) tot += p[k];
  if (err && *err) tot = __builtin_nan("");   // an aborted step (k_coef voids earlier chunks too)
  const int64_t o = (int64_t(e) * P + j0 + jl) * NS + s;
  losses[o] = static_cast<float>(tot * inv_rows);
  if (lossd) lossd[o] = tot * inv_rows;
}

// loss[e] = (sum over tiles in order) / (B (T-1)) of slot (e, direction 0,
// sign +) of a pass with PC directions per expert and both signs: the
// evaluation that runs the step's kernels at radius 0.
__global__ void k_eval_reduce(const double* part, int row_tiles, int N, int PC, double inv_rows, float* loss,
                              const unsigned* err) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= N) return;
  const double* p = part + (int64_t(e) * PC * 2) * row_tiles;
  double tot = 0.0;
  for (int k = 0; k < row_tiles; ++k) tot += p[k];
  if (*err) tot = __builtin_nan("");
  loss[e] = static_cast<float>(tot * inv_rows);
}

// c[e][j] = (L+ - L-) / (2 eps_e P) from the fp64 means, rounded once to fp32;
// summed mode: the loss differences of all experts added in expert order
// (the shared loss difference), divided by expert e's own radius: Eq.
// main-spsa applied to the summed loss, whose joint direction moves expert e
// by eps_e z_{e,j}.  It runs once after every direction
// chunk: if the step was aborted (the flag may have been set in a later
// chunk than some losses were reduced in), every loss and coefficient of
// the step reads NaN.
__global__ void k_coef(const double* lossd, int N, int P, int summed, const float* eps_v, int eps_stride,
                       float* coef, float* losses, const unsigned* err) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= N * P) return;
  if (*err) {
    losses[2 * int64_t(i)] = __builtin_nanf("");
    losses[2 * int64_t(i) + 1] = __builtin_nanf("");
    coef[i] = __builtin_nanf("");
    return;
  }
  const int j = i % P, e = i / P;
  auto inv_denom = [&](int x) { return 1.0 / (2.0 * double(eps_v[int64_t(x) * eps_stride]) * double(P)); };
  double c;
  if (summed) {
    double dF = 0.0;   // the shared loss difference sum_e2 (L_{e2,j,+} - L_{e2,j,-})
    for (int e2 = 0; e2 < N; ++e2) dF += lossd[(int64_t(e2) * P + j) * 2] - lossd[(int64_t(e2) * P + j) * 2 + 1];
    c = dF * inv_denom(e);
  } else {
    c = (lossd[(int64_t(e) * P + j) * 2] - lossd[(int64_t(e) * P + j) * 2 + 1]) * inv_denom(e);
  }
  coef[i] = static_cast<float>(c);
}

// Per-expert rates of a step given as scalars: eps_v[e] = eps, lr_v[e] = lr.
__global__ void k_fill_rates(float* eps_v, float* lr_v, int N, float eps, float lr) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e < N) {
    eps_v[e] = eps;
    lr_v[e] = lr;
  }
}

// A step whose per-expert radius is not finite and > 0, or whose learning
// rate is not finite, is aborted (the sticky flag; losses read NaN and the
// parameters stay as they were).
__global__ void k_check_rates(const float* eps_v, int eps_stride, const float* lr_v, int lr_stride, int N,
                              unsigned* err) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= N) return;
  const float eps = eps_v[int64_t(e) * eps_stride], lr = lr_v[int64_t(e) * lr_stride];
  if (!(eps > 0.0f) || !__builtin_isfinite(eps) || !__builtin_isfinite(lr))
    __hip_atomic_fetch_or(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The probe law of each coordinate: one law for the stacked LSTM; for the
// paper's body under the sparse law, dense +-1 on the LayerNorm gains
// (Appendix E).  Gain ranges are whole probe quads (d is a multiple of 4).
struct LawMap {
  int law;
  int layers;
  int64_t blk;         // parameters per body block; 0: every coordinate has `law`
  int64_t dm;          // body width
  int64_t emb_end;     // first coordinate of the LSTM layers (the embedding precedes it)
  int64_t head_start;  // first coordinate of the head
  unsigned mask;       // perturbed groups (kGroup* bits)
  int64_t gain0;       // the wide controls' body: first gain (all gains follow); 0: none
};

// Whether the probe quad at coordinate k4 belongs to a perturbed group.
// Group boundaries are multiples of 4, so a quad never straddles two.
__device__ __forceinline__ bool quad_perturbed(const LawMap& m, int64_t k4) {
  const unsigned g = k4 < m.emb_end ? kGroupEmb : (k4 < m.head_start ? kGroupLstm : kGroupHead);
  return (m.mask & g) != 0u;
}

__device__ __forceinline__ int law_at(const LawMap& m, int64_t k4) {
  if (m.law != kProbeSparseRademacher) return m.law;
  if (m.gain0 > 0) return k4 >= m.gain0 ? kProbeRademacher : m.law;   // gains at the end (a multiple of 4)
  if (m.blk == 0) return m.law;
  const int64_t l = k4 / m.blk;
  if (l >= m.layers) return kProbeRademacher;                 // g_f
  const int64_t r = k4 - l * m.blk, w = 8 * m.dm * m.dm;
  return (r < m.dm || (r >= m.dm + w && r < 2 * m.dm + w)) ? kProbeRademacher : m.law;   // g1, g2
}

// g_hat[4q .. 4q+3] = sum_{j<P} coef[j] z_j[4q .. 4q+3] of one expert, summed
// in j order in fp32 (each z regenerated from its counter).
__device__ __forceinline__ float4 estimate_quad(uint2 key, uint32_t step_lo, const float* coef, int P, int law,
                                                int64_t q) {
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int j = 0; j < P; ++j) {
    const float4 z = probe_quad(law, key, static_cast<uint32_t>(j), step_lo, 4 * static_cast<uint64_t>(q));
    acc = fma4(coef[j], z, acc);
  }
  return acc;
}

// theta[e][k] -= lr * sum_{j<P} coef[e][j] z_{e,j}[k], one probe quad per
// thread (Section 4, Eq. main-spsa; the plain step on the estimate).
__global__ __launch_bounds__(256) void k_update(float* theta, const uint64_t* seeds, uint64_t step,
                                                 const float* lr_v, int lr_stride, const float* coef, int64_t d,
                                                 int P, LawMap lm, const unsigned* err) {
  const int e = blockIdx.y;
  const int64_t q = blockIdx.x * int64_t(blockDim.x) + threadIdx.x;
  if (4 * q >= d) return;
  if (err && *err) return;   // the step was aborted: theta stays as it was
  if (!quad_perturbed(lm, 4 * q)) return;   // a masked group: no estimate, no update
  const float4 acc = estimate_quad(stream_key(seeds[e], step), static_cast<uint32_t>(step),
                                   coef + int64_t(e) * P, P, law_at(lm, 4 * q), q);
  const float lr = lr_v[int64_t(e) * lr_stride];
  float* t = theta + int64_t(e) * d + 4 * q;
  if (4 * q + 4 <= d) {
    float4 v = *reinterpret_cast<float4*>(t);
    v = fma4(-lr, acc, v);
    *reinterpret_cast<float4*>(t) = v;
  } else {
    const float a4[4] = {acc.x, acc.y, acc.z, acc.w};
    for (int i = 0; 4 * q + i < d; ++i) t[i] = __builtin_fmaf(-lr, a4[i], t[i]);
  }
}

// Adam hyperparameters in the form the kernel uses (fp32): bc1 = 1 - beta1^t,
// bc2 = 1 - beta2^t, omb1 = 1 - beta1, omb2 = 1 - beta2 (computed in fp64 on
// the host, rounded once).
struct AdamArgs {
  float beta1, beta2, omb1, omb2, bc1, bc2, delta, lambda;
};

// The paper's update with coupled weight decay (Appendix E, Eq. localspsa):
//   g = g_hat + lambda theta;  m' = beta1 m + (1 - beta1) g;
//   v' = beta2 v + (1 - beta2) g^2;
//   theta' = theta - lr (m' / bc1) / (sqrt(v' / bc2) + delta).
// theta, m, v [N][d] fp32 in place, one probe quad per thread.
__global__ __launch_bounds__(256) void k_update_adam(float* theta, float* m, float* v, const uint64_t* seeds,
                                                      uint64_t step, AdamArgs h, const float* lr_v, int lr_stride,
                                                      const float* coef, int64_t d, int P, LawMap lm,
                                                      const unsigned* err) {
  const int e = blockIdx.y;
  const int64_t q = blockIdx.x * int64_t(blockDim.x) + threadIdx.x;
  if (4 * q >= d) return;
  if (err && *err) return;   // the step was aborted: theta, m, v stay as they were
  if (!quad_perturbed(lm, 4 * q)) return;   // a masked group: theta, m, v stay as they were
  const float4 acc = estimate_quad(stream_key(seeds[e], step), static_cast<uint32_t>(step),
                                   coef + int64_t(e) * P, P, law_at(lm, 4 * q), q);
  const float a4[4] = {acc.x, acc.y, acc.z, acc.w};
  const float lr = lr_v[int64_t(e) * lr_stride];
  const int64_t base = int64_t(e) * d + 4 * q;
  for (int i = 0; i < 4 && 4 * q + i < d; ++i) {
    const float th = theta[base + i];
    const float g = __builtin_fmaf(h.lambda, th, a4[i]);
    const float m1 = __builtin_fmaf(h.beta1, m[base + i], h.omb1 * g);
    const float v1 = __builtin_fmaf(h.beta2, v[base + i], h.omb2 * (g * g));
    const float r = (m1 / h.bc1) / (sqrtf(v1 / h.bc2) + h.delta);
    theta[base + i] = __builtin_fmaf(-lr, r, th);
    m[base + i] = m1;
    v[base + i] = v1;
  }
}

// Moments of the single-direction estimates X_j = D c_j z_j of each expert
// (the coefficients of a step at fixed weights; Appendix estimator-iso):
//   out[e][0] += sum_k sum_g (sum_{j in g} X_jk)^2  over consecutive groups
//                of `group` directions,
//   out[e][1] += sum_k (sum_j X_jk)^2,
// in fp64, z regenerated per (quad, j).  Partial sums of a block are added
// to out with fp64 atomics (summation order is not fixed).
__global__ __launch_bounds__(256) void k_estimator_moments(const uint64_t* seeds, uint64_t step, const float* coef,
                                                            int64_t d, int D, int group, LawMap lm, double* out) {
  __shared__ double red[2][256];
  const int e = blockIdx.y;
  const int64_t q = blockIdx.x * int64_t(blockDim.x) + threadIdx.x;
  double s0 = 0.0, s1 = 0.0;
  if (4 * q < d && quad_perturbed(lm, 4 * q)) {   // masked coordinates have no estimate
    const uint2 key = stream_key(seeds[e], step);
    const uint32_t step_lo = static_cast<uint32_t>(step);
    const float* c = coef + int64_t(e) * D;
    const int law = law_at(lm, 4 * q);
    double gsum[4] = {0, 0, 0, 0}, tot[4] = {0, 0, 0, 0};
    for (int j = 0; j < D; ++j) {
      const float4 z = probe_quad(law, key, static_cast<uint32_t>(j), step_lo, 4 * static_cast<uint64_t>(q));
      const double x = double(D) * double(c[j]);
      const double zz[4] = {z.x, z.y, z.z, z.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) gsum[i] += x * zz[i];
      if ((j + 1) % group == 0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (4 * q + i < d) s0 += gsum[i] * gsum[i];
          tot[i] += gsum[i];
          gsum[i] = 0.0;
        }
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (4 * q + i < d) s1 += tot[i] * tot[i];
  }
  red[0][threadIdx.x] = s0;
  red[1][threadIdx.x] = s1;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (int(threadIdx.x) < w) {
      red[0][threadIdx.x] += red[0][threadIdx.x + w];
      red[1][threadIdx.x] += red[1][threadIdx.x + w];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    atomicAdd(&out[2 * e], red[0][0]);
    atomicAdd(&out[2 * e + 1], red[1][0]);
  }
}

__global__ void k_zero_f64(double* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0.0;
}

// The plateau schedule (Section 4; Table experimental-setup): an expert's
// learning rate and perturbation radius decay together, by `factor`, after
// `patience` updates without its validation loss improving by more than
// `threshold`, never below `floor` (and never upward).
__global__ void k_schedule_init(soma_schedule_entry* s, int n, float lr0, float eps0) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) s[i] = soma_schedule_entry{lr0, eps0, __builtin_inff(), 0};
}

__global__ void k_schedule_observe(soma_schedule_entry* s, int n, const float* val, int updates, soma_plateau rule) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  soma_schedule_entry x = s[i];
  if (double(val[i]) < double(x.best) - double(rule.threshold)) {
    x.best = val[i];
    x.since = 0;
  } else {
    x.since += updates;
  }
  if (x.since >= rule.patience) {
    x.lr = fminf(x.lr, fmaxf(x.lr * rule.factor, rule.floor));
    x.eps = fminf(x.eps, fmaxf(x.eps * rule.factor, rule.floor));
    x.since = 0;
  }
  s[i] = x;
}

}  // namespace soma

namespace {

hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

int check_launch(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(SOMA_EDEVICE, "%s: %s", what, hipGetErrorString(e));
  return SOMA_OK;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Record a phase boundary on the stream (no-op unless timing is on).
int mark(soma_ctx* ctx, int phase, hipStream_t st) {
  if (!ctx->timing) return SOMA_OK;
  if (ctx->nmarks == ctx->events.size()) {
    hipEvent_t ev;
    const hipError_t e = hipEventCreate(&ev);
    if (e != hipSuccess) return fail(SOMA_EDEVICE, "hipEventCreate: %s", hipGetErrorString(e));
    ctx->events.push_back(ev);
    ctx->phase.push_back(phase);
  }
  ctx->phase[ctx->nmarks] = phase;
  const hipError_t e = hipEventRecord(ctx->events[ctx->nmarks], st);
  if (e != hipSuccess) return fail(SOMA_EDEVICE, "hipEventRecord: %s", hipGetErrorString(e));
  ++ctx->nmarks;
  return SOMA_OK;
}

template <bool kPert>
int launch_rec(const soma::FwdArgs& a, dim3 grid, hipStream_t st) {
  const int B = a.B;
  if (B <= 16)
    hipLaunchKernelGGL((soma::k_rec_step<1, kPert>), grid, dim3(soma::kThreads), 0, st, a);
  else if (B <= 32)
    hipLaunchKernelGGL((soma::k_rec_step<2, kPert>), grid, dim3(soma::kThreads), 0, st, a);
  else
    hipLaunchKernelGGL((soma::k_rec_step<4, kPert>), grid, dim3(soma::kThreads), 0, st, a);
  return SOMA_OK;
}

// The per-step recurrence with split fp16 products (perturbed step, H % 32
// == 0, the per-step path chosen by the shape rather than by the flag).
int launch_rec_split(const soma::FwdArgs& a, dim3 grid, hipStream_t st) {
  const int B = a.B;
  if (B <= 16)
    hipLaunchKernelGGL((soma::k_rec_step_split<1>), grid, dim3(soma::kThreads), 0, st, a);
  else if (B <= 32)
    hipLaunchKernelGGL((soma::k_rec_step_split<2>), grid, dim3(soma::kThreads), 0, st, a);
  else
    hipLaunchKernelGGL((soma::k_rec_step_split<4>), grid, dim3(soma::kThreads), 0, st, a);
  return SOMA_OK;
}

int rec_row_block(int B) { return B <= 16 ? 16 : (B <= 32 ? 32 : 64); }

// Groups of H / (4 NW) blocks that the persistent recurrence can run at once
// (0 when the shape or the device rules it out; NW = persist_waves(H, B)).  The kernel addresses one
// slot's gate inputs with 32-bit offsets, so B (T-1) 4H floats must stay
// below 2^31 bytes.
int persistent_groups_h(const soma_ctx* ctx, int jobs, int H) {
  const soma_config& c = ctx->cfg;
  if (c.flags & SOMA_FLAG_PER_STEP_RECURRENCE) return 0;
  if (ctx->coop_blocks <= 0 || H > soma::kRecMaxH || H % 64 != 0 || c.batch > 64)
    return 0;
  const int64_t gin_slot_bytes = int64_t(c.seq_len - 1) * c.batch * 4 * H * int64_t(sizeof(float));
  if (gin_slot_bytes >= (int64_t(1) << 31)) return 0;
  const int ut = H / (4 * soma::persist_waves(H, c.batch));
  int groups = std::min(ctx->coop_blocks / ut, jobs);
  // Group g owns blocks g + k groups and blocks are dealt to the 8 XCDs
  // round-robin, so with a multiple of 8 groups every group sits on one XCD
  // and exchanges h through its L2; other counts spread each group over
  // every XCD (about twice the time per step), so round down.
  if (groups > 8) groups -= groups % 8;
  groups = std::min(groups, kMaxGroups);
  return groups >= 1 ? groups : 0;
}

int persistent_groups(const soma_ctx* ctx, int jobs) { return persistent_groups_h(ctx, jobs, ctx->cfg.hidden); }

template <int NB, int NCH, bool kRad>
const void* persist_kernel() {
  return reinterpret_cast<const void*>(&soma::k_rec_persist<NB, NCH, kRad, soma::persist_waves(64 * NCH, 16 * NB)>);
}

template <int NB, bool kRad>
const void* persist_kernel_for(int nch) {
  switch (nch) {
    case 1: return persist_kernel<NB, 1, kRad>();
    case 2: return persist_kernel<NB, 2, kRad>();
    case 3: return persist_kernel<NB, 3, kRad>();
    case 4: return persist_kernel<NB, 4, kRad>();
    case 5: return persist_kernel<NB, 5, kRad>();
    case 6: return persist_kernel<NB, 6, kRad>();
    case 7: return persist_kernel<NB, 7, kRad>();
    case 8: return persist_kernel<NB, 8, kRad>();
    case 9: return persist_kernel<NB, 9, kRad>();
    case 10: return persist_kernel<NB, 10, kRad>();
    case 11: return persist_kernel<NB, 11, kRad>();
    default: return nullptr;
  }
}

template <bool kRad>
const void* persist_kernel_for(int B, int H) {
  const int nch = H / 64;
  if (B <= 16) return persist_kernel_for<1, kRad>(nch);
  if (B <= 32) return persist_kernel_for<2, kRad>(nch);
  return persist_kernel_for<4, kRad>(nch);
}

// The persistent recurrence kernel for batch B, hidden width H (H % 64 == 0,
// H <= kRecMaxH) and the generator family of probe law `probe`.
const void* persist_kernel_for(int B, int H, int probe) {
  return probe == SOMA_PROBE_GAUSSIAN ? persist_kernel_for<false>(B, H) : persist_kernel_for<true>(B, H);
}

// The exchange recurrence for width H (xchg_shape) and the generator family
// of probe law `probe`.
template <bool kRad, bool kL1>
const void* xchg_kernel_for(int nch) {
  switch (nch) {
    case 2: return reinterpret_cast<const void*>(&soma::k_rec_xchg<2, kRad, kL1>);
    case 3: return reinterpret_cast<const void*>(&soma::k_rec_xchg<3, kRad, kL1>);
    case 4: return reinterpret_cast<const void*>(&soma::k_rec_xchg<4, kRad, kL1>);
    case 5: return reinterpret_cast<const void*>(&soma::k_rec_xchg<5, kRad, kL1>);
    case 6: return reinterpret_cast<const void*>(&soma::k_rec_xchg<6, kRad, kL1>);
    case 7: return reinterpret_cast<const void*>(&soma::k_rec_xchg<7, kRad, kL1>);
    case 8: return reinterpret_cast<const void*>(&soma::k_rec_xchg<8, kRad, kL1>);
    case 9: return reinterpret_cast<const void*>(&soma::k_rec_xchg<9, kRad, kL1>);
    case 10: return reinterpret_cast<const void*>(&soma::k_rec_xchg<10, kRad, kL1>);
    case 11: return reinterpret_cast<const void*>(&soma::k_rec_xchg<11, kRad, kL1>);
    default: return nullptr;
  }
}

// The instance for width H, the probe kind and the layer (layer 1 reads the
// folded table).
const void* xchg_kernel_for(int H, int probe, bool layer1) {
  const bool rad = probe != SOMA_PROBE_GAUSSIAN;
  if (layer1) return rad ? xchg_kernel_for<true, true>(H / 64) : xchg_kernel_for<false, true>(H / 64);
  return rad ? xchg_kernel_for<true, false>(H / 64) : xchg_kernel_for<false, false>(H / 64);
}

// Groups of the exchange recurrence (a multiple of 8, each on one XCD), or
// 0 where it does not run: one block per compute unit, H / 32 blocks a
// group, the compute units of an XCD past its whole groups idle.
int xchg_groups(const soma_ctx* ctx) {
  const soma_config& c = ctx->cfg;
  if (!xchg_shape(c) || ctx->xchg_per_cu <= 0) return 0;
  const int ut = c.hidden / 32;
  const int groups = 8 * (ctx->xchg_per_cu * ctx->xchg_cus_per_xcd / ut);
  return groups >= 8 && groups <= xchg_max_groups(c.hidden) ? groups : 0;
}

// Its instantiation on pre-formed weights (the wide controls' body, d_p <= 512).
template <int NB, int NCH>
const void* persist_pre_kernel() {
  return reinterpret_cast<const void*>(
      &soma::k_rec_persist<NB, NCH, false, soma::persist_waves(64 * NCH, 16 * NB), true>);
}

template <int NB>
const void* persist_pre_kernel_for(int nch) {
  switch (nch) {
    case 1: return persist_pre_kernel<NB, 1>();
    case 2: return persist_pre_kernel<NB, 2>();
    case 3: return persist_pre_kernel<NB, 3>();
    case 4: return persist_pre_kernel<NB, 4>();
    case 5: return persist_pre_kernel<NB, 5>();
    case 6: return persist_pre_kernel<NB, 6>();
    case 7: return persist_pre_kernel<NB, 7>();
    case 8: return persist_pre_kernel<NB, 8>();
    default: return nullptr;
  }
}

const void* persist_pre_kernel_for(int B, int H) {
  if (B <= 16) return persist_pre_kernel_for<1>(H / 64);
  if (B <= 32) return persist_pre_kernel_for<2>(H / 64);
  return persist_pre_kernel_for<4>(H / 64);
}

// The streaming input projection and head apply for H % 64 == 0,
// H <= kStreamMaxH and one slot's gate inputs under 2^31 bytes (32-bit
// offsets), unless the tiled kernels are asked for.
bool stream_weights(const soma_config& c) {
  if (c.flags & SOMA_FLAG_TILED_WEIGHTS) return false;
  const int64_t gin_slot_bytes = int64_t(c.seq_len - 1) * c.batch * 4 * c.hidden * int64_t(sizeof(float));
  return c.hidden % 64 == 0 && c.hidden <= soma::kStreamMaxH && gin_slot_bytes < (int64_t(1) << 31);
}

template <bool kRad>
// H > 128 (k_head_fused takes H <= 128), H % 64 == 0, H <= kStreamMaxH.
void launch_head_stream_t(const soma::FwdArgs& a, int nslots, float2* hpart, float* htgt, hipStream_t st) {
  const dim3 grid(unsigned(nslots * 2)), block(soma::kProjThreads);
  switch (a.H / 64) {
    case 3: hipLaunchKernelGGL((soma::k_head_stream<3, kRad>), grid, block, 0, st, a, nslots, hpart, htgt); break;
    case 4: hipLaunchKernelGGL((soma::k_head_stream<4, kRad>), grid, block, 0, st, a, nslots, hpart, htgt); break;
    case 5: hipLaunchKernelGGL((soma::k_head_stream<5, kRad>), grid, block, 0, st, a, nslots, hpart, htgt); break;
    case 6: hipLaunchKernelGGL((soma::k_head_stream<6, kRad>), grid, block, 0, st, a, nslots, hpart, htgt); break;
    case 7: hipLaunchKernelGGL((soma::k_head_stream<7, kRad>), grid, block, 0, st, a, nslots, hpart, htgt); break;
    case 8: hipLaunchKernelGGL((soma::k_head_stream<8, kRad>), grid, block, 0, st, a, nslots, hpart, htgt); break;
    case 9: hipLaunchKernelGGL((soma::k_head_stream<9, kRad>), grid, block, 0, st, a, nslots, hpart, htgt); break;
    case 10: hipLaunchKernelGGL((soma::k_head_stream<10, kRad>), grid, block, 0, st, a, nslots, hpart, htgt); break;
    default: hipLaunchKernelGGL((soma::k_head_stream<11, kRad>), grid, block, 0, st, a, nslots, hpart, htgt); break;   // H = 704 (stream_weights)
  }
}

// H <= 128: the whole head and cross entropy of a slot in one block.
template <bool kRad>
void launch_head_fused_t(const soma::FwdArgs& a, int nslots, hipStream_t st) {
  const dim3 grid(static_cast<unsigned>(nslots)), block(soma::kHeadFusedThreads);
  if (a.H == 64)
    hipLaunchKernelGGL((soma::k_head_fused<1, kRad>), grid, block, 0, st, a);
  else
    hipLaunchKernelGGL((soma::k_head_fused<2, kRad>), grid, block, 0, st, a);
}

void launch_head_fused(const soma::FwdArgs& a, int nslots, hipStream_t st) {
  if (a.probe == SOMA_PROBE_GAUSSIAN)
    launch_head_fused_t<false>(a, nslots, st);
  else
    launch_head_fused_t<true>(a, nslots, st);
}

void launch_head_stream(const soma::FwdArgs& a, int nslots, float2* hpart, float* htgt, hipStream_t st) {
  if (a.probe == SOMA_PROBE_GAUSSIAN)
    launch_head_stream_t<false>(a, nslots, hpart, htgt, st);
  else
    launch_head_stream_t<true>(a, nslots, hpart, htgt, st);
}

template <bool kRad>
void launch_proj_stream_t(const soma::FwdArgs& a, int nslots, hipStream_t st) {
  const int mblocks = a.H / 32;
  const dim3 grid(unsigned(nslots * mblocks)), block(soma::kProjThreads);
  switch (a.H / 64) {
    case 1: hipLaunchKernelGGL((soma::k_proj_stream<1, kRad>), grid, block, 0, st, a, mblocks, nslots); break;
    case 2: hipLaunchKernelGGL((soma::k_proj_stream<2, kRad>), grid, block, 0, st, a, mblocks, nslots); break;
    case 3: hipLaunchKernelGGL((soma::k_proj_stream<3, kRad>), grid, block, 0, st, a, mblocks, nslots); break;
    case 4: hipLaunchKernelGGL((soma::k_proj_stream<4, kRad>), grid, block, 0, st, a, mblocks, nslots); break;
    case 5: hipLaunchKernelGGL((soma::k_proj_stream<5, kRad>), grid, block, 0, st, a, mblocks, nslots); break;
    case 6: hipLaunchKernelGGL((soma::k_proj_stream<6, kRad>), grid, block, 0, st, a, mblocks, nslots); break;
    case 7: hipLaunchKernelGGL((soma::k_proj_stream<7, kRad>), grid, block, 0, st, a, mblocks, nslots); break;
    case 8: hipLaunchKernelGGL((soma::k_proj_stream<8, kRad>), grid, block, 0, st, a, mblocks, nslots); break;
    case 9: hipLaunchKernelGGL((soma::k_proj_stream<9, kRad>), grid, block, 0, st, a, mblocks, nslots); break;
    case 10: hipLaunchKernelGGL((soma::k_proj_stream<10, kRad>), grid, block, 0, st, a, mblocks, nslots); break;
    default: hipLaunchKernelGGL((soma::k_proj_stream<11, kRad>), grid, block, 0, st, a, mblocks, nslots); break;   // H = 704 (stream_weights)
  }
}

void launch_proj_stream(const soma::FwdArgs& a, int nslots, hipStream_t st) {
  if (a.probe == SOMA_PROBE_GAUSSIAN)
    launch_proj_stream_t<false>(a, nslots, st);
  else
    launch_proj_stream_t<true>(a, nslots, st);
}

// The projection from a pre-split sequence (k_proj_dma), for the widths at
// which the exchange recurrence stores it (fragment order: H = 128, 256, 512).
bool proj_dma_width(int H) { return H == 128 || H == 256 || H == 512; }

template <bool kRad>
void launch_proj_dma_t(const soma::FwdArgs& a, int nslots, hipStream_t st) {
  const int mblocks = a.H / 32;
  const dim3 grid(unsigned(nslots * mblocks)), block(soma::kProjThreads);
  switch (a.H / 64) {
    case 2: hipLaunchKernelGGL((soma::k_proj_dma<2, kRad>), grid, block, 0, st, a, mblocks, nslots); break;
    case 4: hipLaunchKernelGGL((soma::k_proj_dma<4, kRad>), grid, block, 0, st, a, mblocks, nslots); break;
    default: hipLaunchKernelGGL((soma::k_proj_dma<8, kRad>), grid, block, 0, st, a, mblocks, nslots); break;
  }
}

void launch_proj_dma(const soma::FwdArgs& a, int nslots, hipStream_t st) {
  if (a.probe == SOMA_PROBE_GAUSSIAN)
    launch_proj_dma_t<false>(a, nslots, st);
  else
    launch_proj_dma_t<true>(a, nslots, st);
}

// H = 64 (and the persistent path's other conditions: B <= 64, one slot's
// gate inputs under 2^31 bytes): the recurrence runs one block per job with
// h kept in LDS between steps (k_rec_local).
bool local_recurrence(const soma_config& c) {
  if (c.flags & SOMA_FLAG_PER_STEP_RECURRENCE) return false;
  const int64_t gin_slot_bytes = int64_t(c.seq_len - 1) * c.batch * 4 * c.hidden * int64_t(sizeof(float));
  return c.arch == SOMA_ARCH_LSTM && c.hidden == 64 && c.batch <= 64 && gin_slot_bytes < (int64_t(1) << 31);
}

// Layer 1 of the local recurrence forms its gate inputs in the block from
// LDS copies of the perturbed embedding table (E = 32 or 64) and of the
// job's bytes (B T <= kLocalBytes): no fold.
bool local_embedding(const soma_config& c) {
  return local_recurrence(c) && (c.embed == 32 || c.embed == 64) &&
         int64_t(c.batch) * c.seq_len <= soma::kLocalBytes;
}

template <bool kRad, int KX, bool kHead>
void launch_local_t(const soma::FwdArgs& a, int jobs, int B, hipStream_t st) {
  const dim3 grid(static_cast<unsigned>(jobs)), block(soma::kLocalThreads);
  if (B <= 16)
    hipLaunchKernelGGL((soma::k_rec_local<1, kRad, KX, kHead>), grid, block, 0, st, a, jobs);
  else if (B <= 32)
    hipLaunchKernelGGL((soma::k_rec_local<2, kRad, KX, kHead>), grid, block, 0, st, a, jobs);
  else
    hipLaunchKernelGGL((soma::k_rec_local<4, kRad, KX, kHead>), grid, block, 0, st, a, jobs);
}

// kx: 32-wide chunks of the embedding formed in the block (0: gate inputs
// read from U or gin); head: the head and cross entropy fused into the block
// (kx > 0 only: the targets are read from the job's bytes in LDS).
template <bool kRad>
void launch_local_k(const soma::FwdArgs& a, int jobs, int B, int kx, bool head, hipStream_t st) {
  if (kx == 0)
    launch_local_t<kRad, 0, false>(a, jobs, B, st);
  else if (kx == 1 && head)
    launch_local_t<kRad, 1, true>(a, jobs, B, st);
  else if (kx == 1)
    launch_local_t<kRad, 1, false>(a, jobs, B, st);
  else if (head)
    launch_local_t<kRad, 2, true>(a, jobs, B, st);
  else
    launch_local_t<kRad, 2, false>(a, jobs, B, st);
}

int launch_local(const soma::FwdArgs& a, int jobs, int B, int probe, int kx, bool head, hipStream_t st) {
  if (kx < 0 || kx > 2 || (head && kx == 0)) return fail(SOMA_EINVAL, "k_rec_local: embedding chunks %d", kx);
  if (probe == SOMA_PROBE_GAUSSIAN)
    launch_local_k<false>(a, jobs, B, kx, head, st);
  else
    launch_local_k<true>(a, jobs, B, kx, head, st);
  return check_launch("k_rec_local");
}

template <class Args>
int launch_persist(const void* kernel, const Args& p, int blocks, int threads, hipStream_t st,
                   unsigned dyn_lds = 0) {
  void* args[] = {const_cast<Args*>(&p)};
  const hipError_t e = hipLaunchCooperativeKernel(kernel, dim3(blocks), dim3(threads), args, dyn_lds, st);
  if (e != hipSuccess) return fail(SOMA_EDEVICE, "hipLaunchCooperativeKernel: %s", hipGetErrorString(e));
  return SOMA_OK;
}

// The paper's body: one fused launch per pass (SOMA_ARCH_BODY).
template <int DW, int D, bool kPert>
void launch_body_t(const soma::BodyArgs& a, unsigned blocks, hipStream_t st) {
  hipLaunchKernelGGL((soma::k_body<DW, D, kPert>), dim3(blocks), dim3(soma::kBodyThreads), 0, st, a);
}

template <bool kPert>
int run_body(soma_ctx* ctx, const float* theta, const uint64_t* seeds, uint64_t step, const float* eps_v,
             int eps_stride, const uint8_t* bytes, int j0, int pcs, hipStream_t st) {
  const soma_config& c = ctx->cfg;
  const Layout& L = ctx->lay;
  soma::BodyArgs a{};
  a.theta = theta;
  a.bytes = bytes;
  a.seeds = seeds;
  a.E = ctx->head;
  a.e_stride = ctx->head_stride;
  a.part = reinterpret_cast<double*>(ctx->ws + L.part);
  a.fdec = reinterpret_cast<float*>(ctx->ws + L.fdec);
  a.lse = reinterpret_cast<float*>(ctx->ws + L.lse);
  a.d = L.d;
  a.step = step;
  a.eps_v = eps_v;
  a.eps_stride = eps_stride;
  a.probe = c.probe;
  a.ppb = kPert ? c.n_pairs : 1;
  a.bstride = kPert ? int64_t(c.n_experts) * c.batch * c.seq_len : 0;
  a.N = c.n_experts;
  a.B = c.batch;
  a.T = c.seq_len;
  a.PC = kPert ? L.pc : 1;
  a.pcs = pcs;
  a.j0 = j0;
  a.btiles = L.row_tiles;
  a.err = reinterpret_cast<unsigned*>(ctx->ws + L.sync) + kMaxGroups;
  const unsigned blocks = unsigned(L.row_tiles) * unsigned(c.n_experts) * unsigned(pcs) * (kPert ? 2u : 1u);
  const bool wide = c.hidden == 32, deep = c.n_layers == 2;
  if (wide && deep) launch_body_t<2, 2, kPert>(a, blocks, st);
  else if (wide) launch_body_t<2, 1, kPert>(a, blocks, st);
  else if (deep) launch_body_t<1, 2, kPert>(a, blocks, st);
  else launch_body_t<1, 1, kPert>(a, blocks, st);
  if (int rc = check_launch("k_body")) return rc;
  ctx->rec_launches += 1;
  return mark(ctx, kPhaseRec, st);
}

// The wide controls' body: one pass of the kernels listed in soma_wide.hpp
// over the pass's slots (expert, direction, sign), or over the experts
// unperturbed (!kPert).
// epi: soma::WideEpi; a_split: A stored split (else fp32, split as staged).
int launch_wide_mm(int epi, bool a_split, soma::MmArgs m, int slots, hipStream_t st) {
  m.ntn = (m.N + 127) / 128;
  m.ntm = (m.M + 127) / 128;
  m.tiles = int64_t(m.ntn) * m.ntm * slots;
  const int64_t blocks = (m.tiles + soma::kXcds - 1) / soma::kXcds * soma::kXcds;
  if (blocks >= (int64_t(1) << 31)) return fail(SOMA_ESHAPE, "too many product tiles in one launch");
  const dim3 grid(static_cast<unsigned>(blocks)), block(256);
  if (!a_split)
    hipLaunchKernelGGL((soma::k_wide_mm<false, soma::kEpiStore>), grid, block, 0, st, m);
  else if (epi == soma::kEpiGelu)
    hipLaunchKernelGGL((soma::k_wide_mm<true, soma::kEpiGelu>), grid, block, 0, st, m);
  else if (epi == soma::kEpiAdd)
    hipLaunchKernelGGL((soma::k_wide_mm<true, soma::kEpiAdd>), grid, block, 0, st, m);
  else
    hipLaunchKernelGGL((soma::k_wide_mm<true, soma::kEpiStore>), grid, block, 0, st, m);
  return check_launch("k_wide_mm");
}

template <bool kPert>
int run_wide(soma_ctx* ctx, const float* theta, const uint64_t* seeds, uint64_t step, const float* eps_v,
             int eps_stride, const uint8_t* bytes, int j0, int pcs, hipStream_t st) {
  const soma_config& c = ctx->cfg;
  const Layout& L = ctx->lay;
  const int N = c.n_experts, D = c.n_layers, dt = c.hidden, dp = soma::wide_padded(dt);
  const int NS = kPert ? 2 : 1, PC = kPert ? L.pc : 1;
  const int slots = N * pcs * NS;
  const int64_t R = int64_t(c.seq_len - 1) * c.batch;
  const soma::WideForm F = soma::wide_form_layout(dp, D);
  const int64_t mp = 4 * int64_t(dp) * dp;
  unsigned* err = reinterpret_cast<unsigned*>(ctx->ws + L.sync) + kMaxGroups;
  const int groups = persistent_groups_h(ctx, slots, dp);
  if (groups <= 0) return fail(SOMA_EDEVICE, "the wide body needs the persistent recurrence (cooperative launch)");

  soma::WideArgs a{};
  a.theta = theta;
  a.seeds = seeds;
  a.bytes = bytes;
  a.E = ctx->head;
  a.e_stride = ctx->head_stride;
  a.wform = reinterpret_cast<float*>(ctx->ws + L.wform);
  a.U = reinterpret_cast<float*>(ctx->ws + L.U);
  a.x = reinterpret_cast<float*>(ctx->ws + L.xres);
  a.n = reinterpret_cast<float*>(ctx->ws + L.hseq);
  a.gin = reinterpret_cast<float*>(ctx->ws + L.gin);
  a.part = reinterpret_cast<double*>(ctx->ws + L.part);
  a.fdec = reinterpret_cast<float*>(ctx->ws + L.fdec);
  a.lse = reinterpret_cast<float*>(ctx->ws + L.lse);
  a.d = L.d;
  a.step = step;
  a.eps_v = eps_v;
  a.eps_stride = eps_stride;
  a.err = err;
  a.probe = c.probe;
  a.ppb = kPert ? c.n_pairs : 1;
  a.bstride = kPert ? int64_t(N) * c.batch * c.seq_len : 0;
  a.N = N;
  a.D = D;
  a.dt = dt;
  a.dp = dp;
  a.B = c.batch;
  a.T = c.seq_len;
  a.PC = PC;
  a.pcs = pcs;
  a.j0 = j0;
  a.NS = NS;
  a.row_tiles = L.row_tiles;

  // Pre-formed weights; padded entries are zero (the form kernel writes only
  // the real ones).
  const int64_t form_floats = int64_t(N) * PC * NS * F.total;
  if (dp != dt) {
    hipLaunchKernelGGL(soma::k_fill_f32, dim3(4096), dim3(256), 0, st, a.wform, form_floats);
    if (int rc = check_launch("k_fill_f32")) return rc;
  }
  const int64_t mat_quads = (L.d - (2LL * D + 1) * dt) / 4;
  hipLaunchKernelGGL((soma::k_wide_form<kPert>), dim3(unsigned((mat_quads + 255) / 256), unsigned(slots)), dim3(256),
                     0, st, a);
  if (int rc = check_launch("k_wide_form")) return rc;
  if (int rc = mark(ctx, kPhaseFold, st)) return rc;

  soma::MmArgs m{};
  m.pcs = pcs;
  m.PC = PC;
  m.NS = NS;
  m.err = err;
  m.w_slot = F.total;
  // U = E P_in^T: the input projection of every byte value.
  m.A = ctx->head;
  m.a_slot = ctx->head_stride;
  m.a_expert = 1;
  m.W = a.wform + F.pin;
  m.C = a.U;
  m.c_slot = int64_t(SOMA_VOCAB) * dp;
  m.M = SOMA_VOCAB;
  m.N = dp;
  m.K = soma::kWideHeadWidth;
  if (int rc = launch_wide_mm(soma::kEpiStore, false, m, slots, st)) return rc;
  const dim3 ln_grid(unsigned((R + 3) / 4), unsigned(slots));
  hipLaunchKernelGGL((soma::k_wide_ln<0>), ln_grid, dim3(256), 0, st, a);
  if (int rc = check_launch("k_wide_ln")) return rc;
  if (int rc = mark(ctx, kPhaseFold, st)) return rc;

  m.a_expert = 0;
  m.M = int(R);
  for (int l = 0; l < D; ++l) {
    const float* blk = a.wform + F.blk0 + l * F.blk_stride;
    // gate inputs gin = n A'^T (rows interleaved per unit)
    m.A = a.n;
    m.a_slot = R * dp;
    m.W = blk;
    m.C = a.gin;
    m.c_slot = R * 4 * dp;
    m.N = 4 * dp;
    m.K = dp;
    if (int rc = launch_wide_mm(soma::kEpiStore, true, m, slots, st)) return rc;
    if (int rc = mark(ctx, kPhaseProj, st)) return rc;
    ++ctx->proj_launches;
    // the recurrence on the pre-formed R; h into the n buffer
    soma::FwdArgs f{};
    f.theta = theta;
    f.bytes = bytes;
    f.seeds = seeds;
    f.gin = a.gin;
    f.hseq = a.n;
    f.d = L.d;
    f.step = step;
    f.eps_v = eps_v;
    f.eps_stride = eps_stride;
    f.pmask = group_mask(c);
    f.err = err;
    f.probe = c.probe;
    f.ppb = a.ppb;
    f.bstride = a.bstride;
    f.N = N;
    f.E = dp;
    f.H = dp;
    f.B = c.batch;
    f.T = c.seq_len;
    f.PC = PC;
    f.pcs = pcs;
    f.j0 = j0;
    f.layer = 1;        // gate inputs from gin
    f.in_l = dp;
    f.wpre = blk + mp;
    f.wpre_slot = F.total;
    f.ns = NS;
    soma::PersistArgs p{};
    p.a = f;
    p.bar = reinterpret_cast<unsigned*>(ctx->ws + L.sync);
    p.err = err;
    p.groups = groups;
    p.jobs = slots;
    p.spin_limit = ctx->spin_limit;
    hipLaunchKernelGGL(soma::k_zero_u32, dim3((groups + 255) / 256), dim3(256), 0, st, p.bar, groups);
    if (int rc = check_launch("k_zero_u32")) return rc;
    const int nw = soma::persist_waves(dp, c.batch);
    const void* kern = persist_pre_kernel_for(c.batch, dp);
    if (!kern) return fail(SOMA_ESHAPE, "no persistent recurrence for d_p = %d", dp);
    if (int rc = launch_persist(kern, p, groups * (dp / (4 * nw)), 64 * nw, st)) return rc;
    ctx->rec_launches += 1;
    if (int rc = mark(ctx, kPhaseRec, st)) return rc;
    // x += h; n = LN(x); m = GELU(n U'^T); x += m V^T
    hipLaunchKernelGGL((soma::k_wide_ln<1>), ln_grid, dim3(256), 0, st, a);
    if (int rc = check_launch("k_wide_ln")) return rc;
    m.A = a.n;
    m.a_slot = R * dp;
    m.W = blk + 2 * mp;
    m.C = a.gin;
    m.c_slot = R * 4 * dp;
    m.N = 4 * dp;
    m.K = dp;
    if (int rc = launch_wide_mm(soma::kEpiGelu, true, m, slots, st)) return rc;
    m.A = a.gin;
    m.a_slot = R * 4 * dp;
    m.W = blk + 3 * mp;
    m.C = a.x;
    m.c_slot = R * dp;
    m.N = dp;
    m.K = 4 * dp;
    if (int rc = launch_wide_mm(soma::kEpiAdd, true, m, slots, st)) return rc;
    if (l + 1 < D) {
      hipLaunchKernelGGL((soma::k_wide_ln<2>), ln_grid, dim3(256), 0, st, a);
      if (int rc = check_launch("k_wide_ln")) return rc;
    }
    if (int rc = mark(ctx, kPhaseProj, st)) return rc;
    ctx->proj_launches += 2;
  }
  hipLaunchKernelGGL((soma::k_wide_ln<2>), ln_grid, dim3(256), 0, st, a);
  if (int rc = check_launch("k_wide_ln")) return rc;
  // u = n P_out'^T into the (free) gate-input buffer, then the decoder.
  m.A = a.n;
  m.a_slot = R * dp;
  m.W = a.wform + F.pout;
  m.C = a.gin;
  m.c_slot = R * 4 * dp;
  m.N = soma::kWideHeadWidth;
  m.K = dp;
  if (int rc = launch_wide_mm(soma::kEpiStore, true, m, slots, st)) return rc;
  hipLaunchKernelGGL((soma::k_wide_head<!kPert>), dim3(unsigned(L.row_tiles), unsigned(slots)), dim3(256), 0, st, a,
                     a.gin, R * 4 * dp, soma::kWideHeadWidth);
  if (int rc = check_launch("k_wide_head")) return rc;
  return mark(ctx, kPhaseHead, st);
}

// Forward passes of `pcs` directions starting at j0 (kPert) or of the
// unperturbed experts (!kPert, pcs = 1), ending with per-tile loss sums.
template <bool kPert>
int run_forward(soma_ctx* ctx, const float* theta, const uint64_t* seeds, uint64_t step, const float* eps_v,
                int eps_stride, const uint8_t* bytes, int j0, int pcs, hipStream_t st) {
  const soma_config& c = ctx->cfg;
  if (c.arch == SOMA_ARCH_BODY) return run_body<kPert>(ctx, theta, seeds, step, eps_v, eps_stride, bytes, j0, pcs, st);
  if (c.arch == SOMA_ARCH_WIDE) return run_wide<kPert>(ctx, theta, seeds, step, eps_v, eps_stride, bytes, j0, pcs, st);
  const Layout& L = ctx->lay;
  soma::FwdArgs a{};
  a.theta = theta;
  a.bytes = bytes;
  a.seeds = seeds;
  a.U = reinterpret_cast<float*>(ctx->ws + L.U);
  a.gin = reinterpret_cast<float*>(ctx->ws + L.gin);
  a.hseq = reinterpret_cast<float*>(ctx->ws + L.hseq);
  a.cst = reinterpret_cast<float*>(ctx->ws + L.cst);
  a.part = reinterpret_cast<double*>(ctx->ws + L.part);
  a.d = L.d;
  a.off_head = L.off_head;
  a.step = step;
  a.eps_v = eps_v;
  a.eps_stride = eps_stride;
  a.pmask = group_mask(c);
  a.err = reinterpret_cast<unsigned*>(ctx->ws + L.sync) + kMaxGroups;
  a.ppb = kPert ? c.n_pairs : 1;
  a.bstride = kPert ? int64_t(c.n_experts) * c.batch * c.seq_len : 0;
  a.probe = c.probe;
  a.N = c.n_experts;
  a.E = c.embed;
  a.H = c.hidden;
  a.B = c.batch;
  a.T = c.seq_len;
  a.PC = kPert ? L.pc : 1;
  a.j0 = j0;
  a.pcs = pcs;
  a.row_tiles = L.row_tiles;
  const int H = c.hidden, N = c.n_experts;
  const int64_t R = int64_t(c.seq_len - 1) * c.batch;

  a.layer = 0;
  a.in_l = c.embed;
  a.off_l = L.off_layer[0];
  const bool emb_local = kPert && local_embedding(c);
  // One layer at H = 64 with the embedding in the block: the head and the
  // cross entropy run in the recurrence block too (no h in HBM, no head
  // launch), unless the tiled reference kernels are asked for.
  const bool fused_head = emb_local && c.n_layers == 1 && stream_weights(c);
  if (!emb_local) {
    hipLaunchKernelGGL((soma::k_fold<kPert>), dim3(4 * H / 64, SOMA_VOCAB / 64, N * pcs),
                       dim3(soma::kThreads), 0, st, a);
    if (int rc = check_launch("k_fold")) return rc;
  }
  if (int rc = mark(ctx, kPhaseFold, st)) return rc;
  const int rb = rec_row_block(c.batch);
  const int bgroups = (c.batch + rb - 1) / rb;
  bool split_h = false;   // hseq holds the previous layer's h split into fp16 parts
  for (int l = 0; l < c.n_layers; ++l) {
    a.layer = l;
    a.in_l = l == 0 ? c.embed : c.hidden;
    a.off_l = L.off_layer[l];
    if (l > 0) {
      if (split_h) {
        launch_proj_dma(a, 2 * N * pcs, st);
        if (int rc = check_launch("k_proj_dma")) return rc;
      } else if (kPert && stream_weights(c)) {
        launch_proj_stream(a, 2 * N * pcs, st);
        if (int rc = check_launch("k_proj_stream")) return rc;
      } else {
        hipLaunchKernelGGL((soma::k_proj<kPert>),
                           dim3(4 * H / 64, unsigned((R + 127) / 128), N * pcs),
                           dim3(soma::kThreads), 0, st, a);
        if (int rc = check_launch("k_proj")) return rc;
      }
      if (int rc = mark(ctx, kPhaseProj, st)) return rc;
      ++ctx->proj_launches;
    }
    const int groups = kPert ? persistent_groups(ctx, 2 * N * pcs) : 0;
    const int xgroups = kPert ? xchg_groups(ctx) : 0;
    bool out_split = false;   // this layer's recurrence stores its h split
    if (kPert && local_recurrence(c)) {
      // H = 64: one block per job, h kept in the block between steps.
      const int jobs = 2 * N * pcs;   // (expert, direction, sign)
      const int kx = l == 0 && emb_local ? c.embed / 32 : 0;
      if (int rc = launch_local(a, jobs, c.batch, c.probe, kx, fused_head, st)) return rc;
      ctx->rec_launches += 1;
    } else if (xgroups > 0) {
      soma::XchgArgs p{};
      p.a = a;
      p.xh = reinterpret_cast<_Float16*>(ctx->ws + L.xch);
      p.flag = reinterpret_cast<unsigned*>(ctx->ws + L.xch + L.xch_bytes);
      p.cu_count = p.flag + soma::kXchgMaxGroups * soma::kXchgFlagWords;
      p.rank_count = p.cu_count + soma::kXchgCuSlots;
      p.err = a.err;
      p.groups = xgroups;
      p.cus_per_xcd = ctx->xchg_cus_per_xcd;
      p.per_cu = ctx->xchg_per_cu;
      p.jobs = 2 * N * pcs;   // (expert, direction, sign)
      p.spin_limit = ctx->spin_limit;
      // Flags and placement counters restart at zero for every launch.
      const int words = xchg_counter_words();
      hipLaunchKernelGGL(soma::k_zero_u32, dim3((words + 255) / 256), dim3(256), 0, st, p.flag, words);
      if (int rc = check_launch("k_zero_u32")) return rc;
      const int blocks = ctx->xchg_per_cu * 8 * ctx->xchg_cus_per_xcd;
      // The next layer's projection reads this layer's h pre-split (k_proj_dma).
      p.split_out = l + 1 < c.n_layers && stream_weights(c) && proj_dma_width(H) && c.batch % 16 == 0 &&
                    !(c.flags & SOMA_FLAG_FP32_SEQUENCE) ? 1 : 0;
      out_split = p.split_out != 0;
      if (int rc = launch_persist(xchg_kernel_for(H, c.probe, l == 0), p, blocks, 512, st,
                                  unsigned(ctx->xchg_pad_lds)))
        return rc;
      ctx->rec_launches += 1;
      ctx->xchg_launches += 1;
    } else if (groups > 0) {
      soma::PersistArgs p{};
      p.a = a;
      p.bar = reinterpret_cast<unsigned*>(ctx->ws + L.sync);
      p.err = p.bar + kMaxGroups;
      p.groups = groups;
      p.jobs = 2 * N * pcs;   // (expert, direction, sign)
      p.spin_limit = ctx->spin_limit;
      // Counters restart at zero for every launch; the abort flag is kept
      // (zeroed once per step) so that a failure anywhere in the step sticks.
      hipLaunchKernelGGL(soma::k_zero_u32, dim3((groups + 255) / 256), dim3(256), 0, st, p.bar, groups);
      if (int rc = check_launch("k_zero_u32")) return rc;
      const int nw = soma::persist_waves(H, c.batch);
      const int blocks = groups * (H / (4 * nw));
      if (int rc = launch_persist(persist_kernel_for(c.batch, H, c.probe), p, blocks, 64 * nw, st)) return rc;
      ctx->rec_launches += 1;
    } else {
      const dim3 grid((H / 16) * bgroups, pcs, N);
      const bool split = kPert && !(c.flags & SOMA_FLAG_PER_STEP_RECURRENCE) && H % 32 == 0;
      for (int t = 0; t + 1 < c.seq_len; ++t) {
        a.t = t;
        if (split)
          launch_rec_split(a, grid, st);
        else
          launch_rec<kPert>(a, grid, st);
      }
      if (int rc = check_launch(split ? "k_rec_step_split" : "k_rec_step")) return rc;
      ctx->rec_launches += c.seq_len - 1;
    }
    split_h = out_split;
    if (int rc = mark(ctx, kPhaseRec, st)) return rc;
  }
  if (fused_head) {
    // formed by the recurrence block
  } else if (kPert && stream_weights(c) && H <= 128) {
    launch_head_fused(a, 2 * N * pcs, st);
    if (int rc = check_launch("k_head_fused")) return rc;
  } else if (kPert && stream_weights(c)) {
    float2* hpart = reinterpret_cast<float2*>(ctx->ws + L.hpart);
    float* htgt = reinterpret_cast<float*>(ctx->ws + L.htgt);
    launch_head_stream(a, 2 * N * pcs, hpart, htgt, st);
    if (int rc = check_launch("k_head_stream")) return rc;
    hipLaunchKernelGGL(soma::k_ce_combine, dim3(L.row_tiles, 2 * N * pcs), dim3(64), 0, st, a, hpart, htgt);
    if (int rc = check_launch("k_ce_combine")) return rc;
  } else {
    hipLaunchKernelGGL((soma::k_head_ce<kPert>), dim3(L.row_tiles, N * pcs), dim3(soma::kThreads), 0,
                       st, a);
    if (int rc = check_launch("k_head_ce")) return rc;
  }
  return mark(ctx, kPhaseHead, st);
}

// Fill a context for a shape and its workspace on the current device (no
// allocation: the persistent recurrence's occupancy is queried, not run).
void init_ctx(soma_ctx* ctx, const soma_config& cfg0, const Layout& L, char* ws, size_t ws_bytes) {
  const soma_config* cfg = &cfg0;
  ctx->cfg = cfg0;
  ctx->lay = L;
  ctx->ws = ws;
  ctx->ws_bytes = ws_bytes;
  ctx->have_coef = false;
  ctx->coop_blocks = 0;
  {
    // Co-resident blocks for the persistent recurrence on the current device.
    int dev = 0, coop = 0, cus = 0, per_cu = 0, lds_max = 0;
    hipFuncAttributes fa{};
    // The wide body's recurrence runs at the padded width on pre-formed
    // weights (the kernel's generator family is then unused).
    const int rec_h = cfg->arch == SOMA_ARCH_WIDE ? soma::wide_padded(cfg->hidden) : cfg->hidden;
    const bool shape_ok = cfg->arch != SOMA_ARCH_BODY && rec_h % 64 == 0 && rec_h <= soma::kRecMaxH &&
                          cfg->batch <= 64;
    const void* kern = !shape_ok ? nullptr
                       : cfg->arch == SOMA_ARCH_WIDE ? persist_pre_kernel_for(cfg->batch, rec_h)
                                                     : persist_kernel_for(cfg->batch, rec_h, cfg->probe);
    if (kern && hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) == hipSuccess &&
        hipFuncGetAttributes(&fa, kern) == hipSuccess &&
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, 64 * soma::persist_waves(rec_h, cfg->batch), 0) ==
            hipSuccess &&
        coop && size_t(lds_max) >= fa.sharedSizeBytes && per_cu >= 1) {
      ctx->coop_blocks = cus * per_cu;
    }
    (void)hipGetLastError();  // a failed query only disables the persistent path
  }
  ctx->xchg_per_cu = 0;
  ctx->xchg_cus_per_xcd = 0;
  ctx->xchg_pad_lds = 0;
  if (xchg_shape(*cfg)) {
    // The exchange recurrence: one block per compute unit (unused dynamic LDS
    // caps the occupancy where more would fit: every compute unit must hold
    // exactly one block for the placement), compute units per XCD (8 XCDs,
    // blocks dealt to them round-robin).  A launch that placed two of its
    // blocks on each compute unit faulted the device, with no cause found
    // in the kernel's indexing; that placement stays off.
    // Both instances (layer 1, deeper layers) must take the same geometry.
    int dev = 0, coop = 0, cus = 0, lds_cu = 0;
    const bool dev_ok = hipGetDevice(&dev) == hipSuccess &&
                        hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) == hipSuccess &&
                        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
                        hipDeviceGetAttribute(&lds_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) ==
                            hipSuccess &&
                        coop && cus % 8 == 0 && cus / 8 <= 64;
    int pad_of[2] = {-1, -1};
    for (int l1 = 0; l1 < 2 && dev_ok; ++l1) {
      const void* kern = xchg_kernel_for(cfg->hidden, cfg->probe, l1 == 1);
      hipFuncAttributes fa{};
      int occ = 0;
      if (!kern || hipFuncGetAttributes(&fa, kern) != hipSuccess ||
          hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kern, 512, 0) != hipSuccess || occ < 1)
        break;
      int pad = 0, got = occ;
      if (occ > 1) {
        pad = std::max(0, lds_cu / 2 + 2048 - int(fa.sharedSizeBytes));
        if (int(fa.sharedSizeBytes) + pad > lds_cu ||
            hipOccupancyMaxActiveBlocksPerMultiprocessor(&got, kern, 512, size_t(pad)) != hipSuccess)
          got = 0;
      }
      if (got == 1) pad_of[l1] = pad;
    }
    if (pad_of[0] >= 0 && pad_of[1] >= 0) {
      ctx->xchg_per_cu = 1;
      ctx->xchg_cus_per_xcd = cus / 8;
      ctx->xchg_pad_lds = std::max(pad_of[0], pad_of[1]);
    }
    (void)hipGetLastError();
  }
  ctx->head = nullptr;
  ctx->head_stride = 0;
  ctx->timing = false;
  ctx->spin_limit = kSpinLimit;
  ctx->have_times = false;
  ctx->nmarks = 0;
  ctx->rec_launches = ctx->proj_launches = ctx->xchg_launches = 0;
}

}  // namespace

extern "C" {

const char* soma_last_error(void) { return g_last_error.c_str(); }

int soma_param_count(const soma_config* cfg, int64_t* per_expert) {
  if (int rc = validate(cfg)) return rc;
  if (!per_expert) return fail(SOMA_EINVAL, "per_expert is NULL");
  *per_expert = param_count_of(*cfg);
  return ok();
}

int soma_workspace_size(const soma_config* cfg, size_t* bytes) {
  if (int rc = validate(cfg)) return rc;
  if (!bytes) return fail(SOMA_EINVAL, "bytes is NULL");
  *bytes = layout_for(*cfg, choose_chunk(*cfg)).total;
  return ok();
}

int soma_create(const soma_config* cfg, void* workspace, size_t ws_bytes, soma_ctx** out) {
  if (int rc = validate(cfg)) return rc;
  if (!out) return fail(SOMA_EINVAL, "out is NULL");
  const Layout L = layout_for(*cfg, choose_chunk(*cfg));
  if (!workspace) return fail(SOMA_EWORKSPACE, "workspace is NULL");
  if (!aligned(workspace, kAlign)) return fail(SOMA_EWORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < L.total)
    return fail(SOMA_EWORKSPACE, "workspace too small: %zu < %zu bytes", ws_bytes, L.total);
  soma_ctx* ctx = new (std::nothrow) soma_ctx;
  if (!ctx) return fail(SOMA_EINVAL, "out of host memory");
  init_ctx(ctx, *cfg, L, static_cast<char*>(workspace), ws_bytes);
  *out = ctx;
  return ok();
}

void soma_destroy(soma_ctx* ctx) {
  if (!ctx) return;
  for (hipEvent_t ev : ctx->events) (void)hipEventDestroy(ev);
  delete ctx;
}

int soma_set_phase_timing(soma_ctx* ctx, int enable) {
  if (!ctx) return fail(SOMA_EINVAL, "ctx is NULL");
  ctx->timing = enable != 0;
  return ok();
}

int soma_set_spin_limit(soma_ctx* ctx, uint32_t polls) {
  if (!ctx) return fail(SOMA_EINVAL, "ctx is NULL");
  ctx->spin_limit = polls == 0 ? kSpinLimit : polls;
  return ok();
}

int soma_get_phase_times(soma_ctx* ctx, soma_phase_times* out) {
  if (!ctx || !out) return fail(SOMA_EINVAL, "NULL argument");
  if (!ctx->have_times || ctx->nmarks < 2) return fail(SOMA_EINVAL, "no timed step on this context");
  hipError_t e = hipEventSynchronize(ctx->events[ctx->nmarks - 1]);
  if (e != hipSuccess) return fail(SOMA_EDEVICE, "hipEventSynchronize: %s", hipGetErrorString(e));
  float acc[6] = {0, 0, 0, 0, 0, 0};
  for (size_t i = 1; i < ctx->nmarks; ++i) {
    float ms = 0.0f;
    e = hipEventElapsedTime(&ms, ctx->events[i - 1], ctx->events[i]);
    if (e != hipSuccess) return fail(SOMA_EDEVICE, "hipEventElapsedTime: %s", hipGetErrorString(e));
    const int p = ctx->phase[i];
    if (p >= 0 && p < 6) acc[p] += ms;
  }
  out->fold_ms = acc[kPhaseFold];
  out->proj_ms = acc[kPhaseProj];
  out->rec_ms = acc[kPhaseRec];
  out->head_ms = acc[kPhaseHead];
  out->reduce_ms = acc[kPhaseReduce];
  out->update_ms = acc[kPhaseUpdate];
  out->rec_launches = ctx->rec_launches;
  out->xchg_launches = ctx->xchg_launches;
  out->proj_launches = ctx->proj_launches;
  return ok();
}

}  // extern "C"

namespace {

// Per-expert perturbation radius and learning rate of a step (device
// pointers, expert e at [e * stride]).
struct Rates {
  const float* eps_v;
  int eps_stride;
  const float* lr_v;
  int lr_stride;
};

// The scalar rates of a step, written to the workspace (no host copy).
int scalar_rates(soma_ctx* ctx, float eps, float lr, hipStream_t st, Rates* out) {
  float* r = reinterpret_cast<float*>(ctx->ws + ctx->lay.rates);
  const int N = ctx->cfg.n_experts;
  hipLaunchKernelGGL(soma::k_fill_rates, dim3((N + 255) / 256), dim3(256), 0, st, r, r + N, N, eps, lr);
  if (int rc = check_launch("k_fill_rates")) return rc;
  *out = Rates{r, 1, r + N, 1};
  return SOMA_OK;
}

Rates schedule_rates(const soma_schedule_entry* sched) {
  constexpr int kStride = int(sizeof(soma_schedule_entry) / sizeof(float));
  static_assert(sizeof(soma_schedule_entry) % sizeof(float) == 0, "entries are whole floats");
  return Rates{&sched->eps, kStride, &sched->lr, kStride};
}

// The paper's body decodes through the caller's tied matrix: it must be set.
int check_head(const soma_ctx* ctx) {
  if (ctx->cfg.arch != SOMA_ARCH_LSTM && !ctx->head)
    return fail(SOMA_EINVAL, "no tied matrix E: call soma_set_tied_head first");
  return SOMA_OK;
}

// Arguments of a step that every update checks (rates apart).
int check_step_ptrs(soma_ctx* ctx, const float* theta, const uint64_t* seeds, const uint8_t* bytes,
                    const float* losses) {
  if (!ctx) return fail(SOMA_EINVAL, "ctx is NULL");
  if (int rc = check_head(ctx)) return rc;
  if (!theta || !seeds || !bytes || !losses) return fail(SOMA_EINVAL, "NULL device pointer");
  if (!aligned(theta, 16)) return fail(SOMA_EINVAL, "theta must be 16-byte aligned");
  if (!aligned(seeds, 8) || !aligned(losses, 4)) return fail(SOMA_EINVAL, "misaligned seeds or losses");
  return SOMA_OK;
}

int check_scalar_rates(float eps, float lr) {
  if (!(eps > 0.0f) || !std::isfinite(eps)) return fail(SOMA_EINVAL, "eps must be finite and > 0");
  if (!std::isfinite(lr)) return fail(SOMA_EINVAL, "lr must be finite");
  return SOMA_OK;
}

// Steps 1-3 of the method: every perturbed forward, the losses and the
// coefficients (in the workspace).  Returns the step's abort flag, which an
// invalid per-expert rate sets.
int forwards_and_coefficients(soma_ctx* ctx, const float* theta, const uint64_t* seeds, uint64_t step,
                              const Rates& r, const uint8_t* bytes, float* losses, hipStream_t st,
                              unsigned** err_out) {
  const soma_config& c = ctx->cfg;
  const Layout& L = ctx->lay;
  ctx->nmarks = 0;
  ctx->rec_launches = ctx->proj_launches = ctx->xchg_launches = 0;
  ctx->have_times = false;
  if (int rc = mark(ctx, kPhaseStart, st)) return rc;
  unsigned* err = reinterpret_cast<unsigned*>(ctx->ws + L.sync) + kMaxGroups;
  hipLaunchKernelGGL(soma::k_zero_u32, dim3(1), dim3(64), 0, st, err, 1);
  if (int rc = check_launch("k_zero_u32")) return rc;
  hipLaunchKernelGGL(soma::k_check_rates, dim3((c.n_experts + 255) / 256), dim3(256), 0, st, r.eps_v,
                     r.eps_stride, r.lr_v, r.lr_stride, c.n_experts, err);
  if (int rc = check_launch("k_check_rates")) return rc;
  const int D = dirs(c);
  for (int j0 = 0; j0 < D; j0 += L.pc) {
    const int pcs = std::min(L.pc, D - j0);
    if (int rc = run_forward<true>(ctx, theta, seeds, step, r.eps_v, r.eps_stride, bytes, j0, pcs, st)) return rc;
    const int n = c.n_experts * pcs * 2;
    const double inv_rows = 1.0 / double(int64_t(c.seq_len - 1) * c.batch);
    hipLaunchKernelGGL(soma::k_loss_reduce, dim3((n + 255) / 256), dim3(256), 0, st,
                       reinterpret_cast<const double*>(ctx->ws + L.part), L.row_tiles, c.n_experts,
                       pcs, L.pc, 2, D, j0, inv_rows, losses,
                       reinterpret_cast<double*>(ctx->ws + L.lossd), err);
    if (int rc = check_launch("k_loss_reduce")) return rc;
    if (int rc = mark(ctx, kPhaseReduce, st)) return rc;
  }
  float* coef = reinterpret_cast<float*>(ctx->ws + L.coef);
  const int nc = c.n_experts * D;
  hipLaunchKernelGGL(soma::k_coef, dim3((nc + 255) / 256), dim3(256), 0, st,
                     reinterpret_cast<const double*>(ctx->ws + L.lossd), c.n_experts, D,
                     c.loss_mode == SOMA_LOSS_SUMMED ? 1 : 0, r.eps_v, r.eps_stride, coef, losses, err);
  if (int rc = check_launch("k_coef")) return rc;
  if (int rc = mark(ctx, kPhaseReduce, st)) return rc;
  *err_out = err;
  return SOMA_OK;
}

// Adam hyperparameters checked and converted for update number t.
int adam_args(const soma_adam* hp, int64_t t, soma::AdamArgs* out) {
  if (!hp) return fail(SOMA_EINVAL, "adam hyperparameters are NULL");
  if (t < 1) return fail(SOMA_EINVAL, "the update number t must be >= 1");
  if (!(hp->beta1 >= 0.0f && hp->beta1 < 1.0f) || !(hp->beta2 >= 0.0f && hp->beta2 < 1.0f))
    return fail(SOMA_EINVAL, "beta1 and beta2 must lie in [0, 1)");
  if (!(hp->delta > 0.0f) || !std::isfinite(hp->delta)) return fail(SOMA_EINVAL, "delta must be finite and > 0");
  if (!std::isfinite(hp->weight_decay)) return fail(SOMA_EINVAL, "weight_decay must be finite");
  const double b1 = hp->beta1, b2 = hp->beta2;
  out->beta1 = hp->beta1;
  out->beta2 = hp->beta2;
  out->omb1 = static_cast<float>(1.0 - b1);
  out->omb2 = static_cast<float>(1.0 - b2);
  out->bc1 = static_cast<float>(1.0 - std::pow(b1, double(t)));
  out->bc2 = static_cast<float>(1.0 - std::pow(b2, double(t)));
  out->delta = hp->delta;
  out->lambda = hp->weight_decay;
  return SOMA_OK;
}

int check_state(const float* m, const float* v) {
  if (!m || !v) return fail(SOMA_EINVAL, "NULL moment buffer");
  if (!aligned(m, 16) || !aligned(v, 16)) return fail(SOMA_EINVAL, "m and v must be 16-byte aligned");
  return SOMA_OK;
}

soma::LawMap law_map(const soma_config& c, const Layout& L) {
  soma::LawMap m{c.probe, c.n_layers, 0, c.hidden, 0, L.d, group_mask(c), 0};
  if (c.arch == SOMA_ARCH_BODY) {
    m.blk = soma::body_block(c.hidden);   // the whole body is the LSTM group
  } else if (c.arch == SOMA_ARCH_WIDE) {
    m.gain0 = L.d - (2LL * c.n_layers + 1) * c.hidden;   // the whole body is the LSTM group
  } else {
    m.emb_end = L.off_layer[0];
    m.head_start = L.off_head;
  }
  return m;
}

int launch_sgd(const soma_ctx* ctx, float* theta, const uint64_t* seeds, uint64_t step, const Rates& r,
               const float* coef, const unsigned* err, hipStream_t st) {
  const soma_config& c = ctx->cfg;
  const int64_t quads = (ctx->lay.d + 3) / 4;
  hipLaunchKernelGGL(soma::k_update, dim3(unsigned((quads + 255) / 256), c.n_experts), dim3(256), 0, st, theta,
                     seeds, step, r.lr_v, r.lr_stride, coef, ctx->lay.d, dirs(c), law_map(c, ctx->lay), err);
  return check_launch("k_update");
}

int launch_adam(const soma_ctx* ctx, float* theta, float* m, float* v, const uint64_t* seeds, uint64_t step,
                const soma::AdamArgs& h, const Rates& r, const float* coef, const unsigned* err, hipStream_t st) {
  const soma_config& c = ctx->cfg;
  const int64_t quads = (ctx->lay.d + 3) / 4;
  hipLaunchKernelGGL(soma::k_update_adam, dim3(unsigned((quads + 255) / 256), c.n_experts), dim3(256), 0, st,
                     theta, m, v, seeds, step, h, r.lr_v, r.lr_stride, coef, ctx->lay.d, dirs(c), law_map(c, ctx->lay), err);
  return check_launch("k_update_adam");
}

int finish_step(soma_ctx* ctx, hipStream_t st) {
  if (int rc = mark(ctx, kPhaseUpdate, st)) return rc;
  ctx->have_coef = true;
  ctx->have_times = ctx->timing;
  return ok();
}

// The whole Adam step for given rates.
int adam_step(soma_ctx* ctx, float* theta, float* m, float* v, int64_t t, const soma_adam* hp,
              const uint64_t* seeds, uint64_t step, const Rates& r, const uint8_t* bytes, float* losses,
              hipStream_t st) {
  soma::AdamArgs h{};
  if (int rc = adam_args(hp, t, &h)) return rc;
  unsigned* err = nullptr;
  if (int rc = forwards_and_coefficients(ctx, theta, seeds, step, r, bytes, losses, st, &err)) return rc;
  if (int rc = launch_adam(ctx, theta, m, v, seeds, step, h, r,
                           reinterpret_cast<const float*>(ctx->ws + ctx->lay.coef), err, st))
    return rc;
  return finish_step(ctx, st);
}

}  // namespace

extern "C" {

int soma_spsa_step(soma_ctx* ctx, float* theta, const uint64_t* seeds, uint64_t step, float eps,
                   float lr, const uint8_t* bytes, float* losses, void* stream) {
  if (int rc = check_step_ptrs(ctx, theta, seeds, bytes, losses)) return rc;
  if (int rc = check_scalar_rates(eps, lr)) return rc;
  const hipStream_t st = as_stream(stream);
  Rates r{};
  if (int rc = scalar_rates(ctx, eps, lr, st, &r)) return rc;
  unsigned* err = nullptr;
  if (int rc = forwards_and_coefficients(ctx, theta, seeds, step, r, bytes, losses, st, &err)) return rc;
  if (int rc = launch_sgd(ctx, theta, seeds, step, r, reinterpret_cast<const float*>(ctx->ws + ctx->lay.coef),
                          err, st))
    return rc;
  return finish_step(ctx, st);
}

int soma_spsa_step_adam(soma_ctx* ctx, float* theta, float* m, float* v, int64_t t, const soma_adam* hp,
                        const uint64_t* seeds, uint64_t step, float eps, float lr, const uint8_t* bytes,
                        float* losses, void* stream) {
  if (int rc = check_step_ptrs(ctx, theta, seeds, bytes, losses)) return rc;
  if (int rc = check_scalar_rates(eps, lr)) return rc;
  if (int rc = check_state(m, v)) return rc;
  soma::AdamArgs h{};
  if (int rc = adam_args(hp, t, &h)) return rc;
  const hipStream_t st = as_stream(stream);
  Rates r{};
  if (int rc = scalar_rates(ctx, eps, lr, st, &r)) return rc;
  return adam_step(ctx, theta, m, v, t, hp, seeds, step, r, bytes, losses, st);
}

int soma_spsa_step_adam_sched(soma_ctx* ctx, float* theta, float* m, float* v, int64_t t, const soma_adam* hp,
                              const uint64_t* seeds, uint64_t step, const soma_schedule_entry* sched,
                              const uint8_t* bytes, float* losses, void* stream) {
  if (int rc = check_step_ptrs(ctx, theta, seeds, bytes, losses)) return rc;
  if (int rc = check_state(m, v)) return rc;
  if (!sched) return fail(SOMA_EINVAL, "schedule is NULL");
  if (!aligned(sched, alignof(soma_schedule_entry))) return fail(SOMA_EINVAL, "misaligned schedule");
  soma::AdamArgs h{};
  if (int rc = adam_args(hp, t, &h)) return rc;
  return adam_step(ctx, theta, m, v, t, hp, seeds, step, schedule_rates(sched), bytes, losses,
                   as_stream(stream));
}

int soma_estimator_moments(soma_ctx* ctx, const uint64_t* seeds, uint64_t step, const float* coef, int32_t group,
                           double* out, void* stream) {
  if (!ctx) return fail(SOMA_EINVAL, "ctx is NULL");
  if (!seeds || !coef || !out) return fail(SOMA_EINVAL, "NULL device pointer");
  if (!aligned(out, 8) || !aligned(seeds, 8)) return fail(SOMA_EINVAL, "misaligned seeds or out");
  const soma_config& c = ctx->cfg;
  const int D = dirs(c);
  if (group < 1 || D % group != 0) return fail(SOMA_EINVAL, "group must divide D = %d", D);
  const hipStream_t st = as_stream(stream);
  hipLaunchKernelGGL(soma::k_zero_f64, dim3((2 * c.n_experts + 255) / 256), dim3(256), 0, st, out,
                     2 * c.n_experts);
  if (int rc = check_launch("k_zero_f64")) return rc;
  const int64_t quads = (ctx->lay.d + 3) / 4;
  hipLaunchKernelGGL(soma::k_estimator_moments, dim3(unsigned((quads + 255) / 256), c.n_experts), dim3(256), 0, st,
                     seeds, step, coef, ctx->lay.d, D, group, law_map(c, ctx->lay), out);
  if (int rc = check_launch("k_estimator_moments")) return rc;
  return ok();
}

int soma_schedule_init(soma_schedule_entry* sched, int32_t n, float lr0, float eps0, void* stream) {
  if (!sched) return fail(SOMA_EINVAL, "schedule is NULL");
  if (n < 1) return fail(SOMA_EINVAL, "n must be >= 1");
  if (!aligned(sched, alignof(soma_schedule_entry))) return fail(SOMA_EINVAL, "misaligned schedule");
  if (!(eps0 > 0.0f) || !std::isfinite(eps0) || !std::isfinite(lr0))
    return fail(SOMA_EINVAL, "eps0 must be finite and > 0, lr0 finite");
  hipLaunchKernelGGL(soma::k_schedule_init, dim3((n + 255) / 256), dim3(256), 0, as_stream(stream), sched, n, lr0,
                     eps0);
  if (int rc = check_launch("k_schedule_init")) return rc;
  return ok();
}

int soma_schedule_observe(soma_schedule_entry* sched, int32_t n, const float* val_loss, int32_t updates,
                          const soma_plateau* rule, void* stream) {
  if (!sched || !val_loss || !rule) return fail(SOMA_EINVAL, "NULL argument");
  if (n < 1 || updates < 0) return fail(SOMA_EINVAL, "n must be >= 1 and updates >= 0");
  if (!aligned(sched, alignof(soma_schedule_entry)) || !aligned(val_loss, 4))
    return fail(SOMA_EINVAL, "misaligned schedule or losses");
  if (!(rule->factor > 0.0f && rule->factor < 1.0f) || rule->patience < 1 || !(rule->threshold >= 0.0f) ||
      !std::isfinite(rule->threshold) || !(rule->floor >= 0.0f) || !std::isfinite(rule->floor))
    return fail(SOMA_EINVAL, "plateau rule: factor in (0, 1), patience >= 1, finite threshold and floor >= 0");
  hipLaunchKernelGGL(soma::k_schedule_observe, dim3((n + 255) / 256), dim3(256), 0, as_stream(stream), sched, n,
                     val_loss, updates, *rule);
  if (int rc = check_launch("k_schedule_observe")) return rc;
  return ok();
}

int soma_apply_adam(soma_ctx* ctx, float* theta, float* m, float* v, int64_t t, const soma_adam* hp,
                    const uint64_t* seeds, uint64_t step, float lr, const float* coef, void* stream) {
  if (!ctx) return fail(SOMA_EINVAL, "ctx is NULL");
  if (!theta || !seeds || !coef) return fail(SOMA_EINVAL, "NULL device pointer");
  if (!aligned(theta, 16)) return fail(SOMA_EINVAL, "theta must be 16-byte aligned");
  if (!std::isfinite(lr)) return fail(SOMA_EINVAL, "lr must be finite");
  if (int rc = check_state(m, v)) return rc;
  soma::AdamArgs h{};
  if (int rc = adam_args(hp, t, &h)) return rc;
  const hipStream_t st = as_stream(stream);
  Rates r{};
  if (int rc = scalar_rates(ctx, 1.0f, lr, st, &r)) return rc;
  if (int rc = launch_adam(ctx, theta, m, v, seeds, step, h, r, coef, nullptr, st)) return rc;
  return ok();
}

int soma_eval_loss(soma_ctx* ctx, const float* theta, const uint8_t* bytes, float* loss,
                   void* stream) {
  if (!ctx) return fail(SOMA_EINVAL, "ctx is NULL");
  if (int rc = check_head(ctx)) return rc;
  if (!theta || !bytes || !loss) return fail(SOMA_EINVAL, "NULL device pointer");
  if (!aligned(theta, 16)) return fail(SOMA_EINVAL, "theta must be 16-byte aligned");
  const soma_config& c = ctx->cfg;
  const Layout& L = ctx->lay;
  const hipStream_t st = as_stream(stream);
  const bool timing = ctx->timing;
  ctx->timing = false;  // evaluation is not part of the step's phase record
  // The abort flag, set by a kernel that meets a weight outside the range of
  // its split products, makes the losses NaN.
  unsigned* err = reinterpret_cast<unsigned*>(ctx->ws + L.sync) + kMaxGroups;
  hipLaunchKernelGGL(soma::k_zero_u32, dim3(1), dim3(64), 0, st, err, 1);
  if (int rc = check_launch("k_zero_u32")) return rc;
  const double inv_rows = 1.0 / double(int64_t(c.seq_len - 1) * c.batch);
  if (c.arch == SOMA_ARCH_LSTM && c.flags == 0) {
    // The step's kernels with radius 0: every weight is formed as
    // fma(+-0, z, theta) = theta, so both signs of direction 0 are the
    // unperturbed model (the probes are drawn and multiplied by zero; any
    // seeds do, so the fp64 loss area serves as their memory).  The + sign's
    // sum is the loss.
    float* r = reinterpret_cast<float*>(ctx->ws + L.rates);
    const int N = c.n_experts;
    hipLaunchKernelGGL(soma::k_fill_rates, dim3((N + 255) / 256), dim3(256), 0, st, r, r + N, N, 0.0f, 0.0f);
    if (int rc = check_launch("k_fill_rates")) return rc;
    const uint64_t* any_seeds = reinterpret_cast<const uint64_t*>(ctx->ws + L.lossd);
    const int rc0 = run_forward<true>(ctx, theta, any_seeds, 0, r, 1, bytes, 0, 1, st);
    ctx->timing = timing;
    if (rc0) return rc0;
    hipLaunchKernelGGL(soma::k_eval_reduce, dim3((N + 255) / 256), dim3(256), 0, st,
                       reinterpret_cast<const double*>(ctx->ws + L.part), L.row_tiles, N, L.pc, inv_rows, loss, err);
    if (int rc = check_launch("k_eval_reduce")) return rc;
    return ok();
  }
  const int rc0 = run_forward<false>(ctx, theta, nullptr, 0, nullptr, 0, bytes, 0, 1, st);
  ctx->timing = timing;
  if (rc0) return rc0;
  hipLaunchKernelGGL(soma::k_loss_reduce, dim3((c.n_experts + 255) / 256), dim3(256), 0, st,
                     reinterpret_cast<const double*>(ctx->ws + L.part), L.row_tiles, c.n_experts, 1,
                     1, 1, 1, 0, inv_rows, loss, static_cast<double*>(nullptr), err);
  if (int rc = check_launch("k_loss_reduce")) return rc;
  return ok();
}

int soma_set_tied_head(soma_ctx* ctx, float* E, int64_t expert_stride) {
  if (!ctx) return fail(SOMA_EINVAL, "ctx is NULL");
  if (ctx->cfg.arch == SOMA_ARCH_LSTM) return fail(SOMA_EINVAL, "the stacked LSTM has no tied matrix");
  if (!E || !aligned(E, 16)) return fail(SOMA_EINVAL, "E must be a 16-byte aligned device pointer");
  if (expert_stride < 0 || expert_stride % 4)
    return fail(SOMA_EINVAL, "expert_stride must be >= 0 and a multiple of 4 floats");
  const int width = ctx->cfg.arch == SOMA_ARCH_WIDE ? ctx->cfg.embed : ctx->cfg.hidden;
  if (expert_stride > 0 && expert_stride < int64_t(SOMA_VOCAB) * width)
    return fail(SOMA_EINVAL, "experts' tied matrices must not overlap (stride %lld < %d)",
                static_cast<long long>(expert_stride), SOMA_VOCAB * width);
  ctx->head = E;
  ctx->head_stride = expert_stride;
  return ok();
}

int soma_head_delta(soma_ctx* ctx, const float* theta, const uint8_t* bytes, float lr, float* grad, float* loss,
                    void* stream) {
  if (!ctx) return fail(SOMA_EINVAL, "ctx is NULL");
  const soma_config& c = ctx->cfg;
  if (c.arch == SOMA_ARCH_LSTM) return fail(SOMA_EINVAL, "the delta rule needs a tied head (arch 1 or 2)");
  if (int rc = check_head(ctx)) return rc;
  if (!theta || !bytes) return fail(SOMA_EINVAL, "NULL device pointer");
  if (!aligned(theta, 16)) return fail(SOMA_EINVAL, "theta must be 16-byte aligned");
  if ((grad && !aligned(grad, 4)) || (loss && !aligned(loss, 4))) return fail(SOMA_EINVAL, "misaligned output");
  if (!std::isfinite(lr)) return fail(SOMA_EINVAL, "lr must be finite");
  if (lr != 0.0f && ctx->head_stride == 0 && c.n_experts > 1)
    return fail(SOMA_EINVAL, "updating E needs one tied matrix per expert (expert_stride != 0)");
  const Layout& L = ctx->lay;
  const hipStream_t st = as_stream(stream);
  const bool timing = ctx->timing;
  ctx->timing = false;
  unsigned* err = reinterpret_cast<unsigned*>(ctx->ws + L.sync) + kMaxGroups;
  hipLaunchKernelGGL(soma::k_zero_u32, dim3(1), dim3(64), 0, st, err, 1);
  if (int rc = check_launch("k_zero_u32")) return rc;
  const int rc0 = c.arch == SOMA_ARCH_WIDE ? run_wide<false>(ctx, theta, nullptr, 0, nullptr, 0, bytes, 0, 1, st)
                                           : run_body<false>(ctx, theta, nullptr, 0, nullptr, 0, bytes, 0, 1, st);
  ctx->timing = timing;
  if (rc0) return rc0;
  const double inv_rows = 1.0 / double(int64_t(c.seq_len - 1) * c.batch);
  const int width = c.arch == SOMA_ARCH_WIDE ? c.embed : c.hidden;
  if (loss) {
    hipLaunchKernelGGL(soma::k_loss_reduce, dim3((c.n_experts + 255) / 256), dim3(256), 0, st,
                       reinterpret_cast<const double*>(ctx->ws + L.part), L.row_tiles, c.n_experts, 1, 1, 1, 1, 0,
                       inv_rows, loss, static_cast<double*>(nullptr), err);
    if (int rc = check_launch("k_loss_reduce")) return rc;
  }
  float* dpart = reinterpret_cast<float*>(ctx->ws + L.dpart);
  const dim3 pgrid(L.delta_chunks, c.n_experts);
  const float* fdec = reinterpret_cast<const float*>(ctx->ws + L.fdec);
  const float* lse = reinterpret_cast<const float*>(ctx->ws + L.lse);
  if (width == 32)
    hipLaunchKernelGGL((soma::k_head_delta_part<2>), pgrid, dim3(256), 0, st, fdec, lse, bytes, ctx->head,
                       ctx->head_stride, c.batch, c.seq_len, L.delta_chunks, dpart);
  else
    hipLaunchKernelGGL((soma::k_head_delta_part<1>), pgrid, dim3(256), 0, st, fdec, lse, bytes, ctx->head,
                       ctx->head_stride, c.batch, c.seq_len, L.delta_chunks, dpart);
  if (int rc = check_launch("k_head_delta_part")) return rc;
  const int64_t vd = int64_t(SOMA_VOCAB) * width;
  hipLaunchKernelGGL(soma::k_head_delta_reduce, dim3(unsigned((vd + 255) / 256), c.n_experts), dim3(256), 0, st,
                     dpart, L.delta_chunks, vd, inv_rows, grad, ctx->head, ctx->head_stride, lr);
  if (int rc = check_launch("k_head_delta_reduce")) return rc;
  return ok();
}

int soma_coefficients(soma_ctx* ctx, float* coef, void* stream) {
  if (!ctx || !coef) return fail(SOMA_EINVAL, "NULL argument");
  if (!ctx->have_coef) return fail(SOMA_EINVAL, "no step has run on this context");
  const size_t n = size_t(ctx->cfg.n_experts) * dirs(ctx->cfg);
  const hipError_t e = hipMemcpyAsync(coef, ctx->ws + ctx->lay.coef, n * sizeof(float),
                                      hipMemcpyDeviceToDevice, as_stream(stream));
  if (e != hipSuccess) return fail(SOMA_EDEVICE, "hipMemcpyAsync: %s", hipGetErrorString(e));
  return ok();
}

int soma_apply_update(soma_ctx* ctx, float* theta, const uint64_t* seeds, uint64_t step, float lr,
                      const float* coef, void* stream) {
  if (!ctx) return fail(SOMA_EINVAL, "ctx is NULL");
  if (!theta || !seeds || !coef) return fail(SOMA_EINVAL, "NULL device pointer");
  if (!aligned(theta, 16)) return fail(SOMA_EINVAL, "theta must be 16-byte aligned");
  if (!std::isfinite(lr)) return fail(SOMA_EINVAL, "lr must be finite");
  const hipStream_t st = as_stream(stream);
  Rates r{};
  if (int rc = scalar_rates(ctx, 1.0f, lr, st, &r)) return rc;
  if (int rc = launch_sgd(ctx, theta, seeds, step, r, coef, nullptr, st)) return rc;
  return ok();
}

int soma_gaussian(uint64_t seed, uint64_t step, uint32_t pair, uint64_t k0, uint64_t count,
                  float* out, void* stream) {
  if (!out) return fail(SOMA_EINVAL, "out is NULL");
  if (count == 0) return ok();
  if (k0 + count > (uint64_t(1) << 40) || k0 + count < k0)
    return fail(SOMA_EINVAL, "k0 + count must not exceed 2^40");
  const uint64_t quads = ((k0 + count + 3) >> 2) - (k0 >> 2);
  hipLaunchKernelGGL(soma::k_gaussian, dim3(unsigned((quads + 255) / 256)), dim3(256), 0,
                     as_stream(stream), seed, step, pair, k0, count, out);
  if (int rc = check_launch("k_gaussian")) return rc;
  return ok();
}

int soma_probe(int law, uint64_t seed, uint64_t step, uint32_t pair, uint64_t k0, uint64_t count, float* out,
               void* stream) {
  if (law != SOMA_PROBE_GAUSSIAN && law != SOMA_PROBE_SPARSE_RADEMACHER && law != SOMA_PROBE_RADEMACHER)
    return fail(SOMA_EINVAL, "unknown probe law %d", law);
  if (!out) return fail(SOMA_EINVAL, "out is NULL");
  if (count == 0) return ok();
  if (k0 + count > (uint64_t(1) << 40) || k0 + count < k0)
    return fail(SOMA_EINVAL, "k0 + count must not exceed 2^40");
  const uint64_t quads = ((k0 + count + 3) >> 2) - (k0 >> 2);
  hipLaunchKernelGGL(soma::k_probe, dim3(unsigned((quads + 255) / 256)), dim3(256), 0, as_stream(stream), law,
                     seed, step, pair, k0, count, out);
  if (int rc = check_launch("k_probe")) return rc;
  return ok();
}

int soma_philox(const uint32_t* ctr, const uint32_t* key, uint32_t* out, uint64_t n, void* stream) {
  if (!ctr || !key || !out) return fail(SOMA_EINVAL, "NULL device pointer");
  if (n == 0) return ok();
  if (n > (uint64_t(1) << 32)) return fail(SOMA_EINVAL, "n too large");
  hipLaunchKernelGGL(soma::k_philox, dim3(unsigned((n + 255) / 256)), dim3(256), 0,
                     as_stream(stream), ctr, key, out, n);
  if (int rc = check_launch("k_philox")) return rc;
  return ok();
}

int soma_box_muller(const uint32_t* wa, const uint32_t* wb, float* za, float* zb, uint64_t n,
                    void* stream) {
  if (!wa || !wb || !za || !zb) return fail(SOMA_EINVAL, "NULL device pointer");
  if (n == 0) return ok();
  if (n > (uint64_t(1) << 32)) return fail(SOMA_EINVAL, "n too large");
  hipLaunchKernelGGL(soma::k_box_muller, dim3(unsigned((n + 255) / 256)), dim3(256), 0,
                     as_stream(stream), wa, wb, za, zb, n);
  if (int rc = check_launch("k_box_muller")) return rc;
  return ok();
}

}  // extern "C"

// ---------------------------------------------------------------------------
// The step for callers that cannot allocate device memory (code under HIP
// graph capture, tight serving loops, harnesses that forbid allocation): the
// kernels of soma_spsa_step with their scratch space in a file-scope device
// array instead of a caller's workspace.  Each GPU the library runs on holds
// its own copy of the array (kStaticScratchBytes) until the process ends; its
// device address is looked up once per device with hipGetSymbolAddress, with
// that device current, and only that address is handed to kernels.  Every
// call on one GPU shares the array: the step clears what must start at zero
// (the abort flag and the group counters, by kernels) and writes everything
// else before reading it, and calls that overlap on one GPU race.
// ---------------------------------------------------------------------------
namespace {

constexpr size_t kStaticScratchBytes = size_t(32) << 20;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxDevices] = {};

// The device address of the current device's scratch array (looked up on
// the first call on that device).
int scratch_address(char** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(SOMA_EDEVICE, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(SOMA_EDEVICE, "device %d beyond the %d supported", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return fail(SOMA_EDEVICE, "hipGetSymbolAddress: %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = static_cast<char*>(p);
  }
  *out = g_scratch_ptr[dev];
  return SOMA_OK;
}

// The largest direction chunk whose workspace fits `budget` bytes (the
// configured chunk if one is set), or 0 if none does.
int chunk_within(const soma_config& c, size_t budget) {
  if (c.pair_chunk > 0) return layout_for(c, c.pair_chunk).total <= budget ? c.pair_chunk : 0;
  for (int pc = dirs(c); pc >= 1; --pc)
    if (layout_for(c, pc).total <= budget) return pc;
  return 0;
}

}  // namespace

extern "C" int soma_spsa_step_noalloc(const soma_config* cfg, float* theta, const uint64_t* seeds, uint64_t step,
                                      float eps, float lr, const uint8_t* bytes, float* losses, void* stream) {
  if (int rc = validate(cfg)) return rc;
  if (cfg->arch != SOMA_ARCH_LSTM) return fail(SOMA_EINVAL, "soma_spsa_step_noalloc runs the stacked LSTM only");
  const int pc = chunk_within(*cfg, kStaticScratchBytes);
  if (pc == 0)
    return fail(SOMA_ESHAPE, "this shape needs %zu bytes of scratch per direction; the static scratch holds %zu",
                layout_for(*cfg, 1).total, kStaticScratchBytes);
  char* ws = nullptr;
  if (int rc = scratch_address(&ws)) return rc;
  const Layout L = layout_for(*cfg, pc);
  soma_ctx ctx;   // host stack: its event pool stays empty (no phase timing here)
  init_ctx(&ctx, *cfg, L, ws, kStaticScratchBytes);
  return soma_spsa_step(&ctx, theta, seeds, step, eps, lr, bytes, losses, stream);
}

// soma_wide.hpp -- the body of the paper's wider fixed-size controls
// (SOMA_ARCH_WIDE; Appendix C, counting rules and Table
// fixed-parameter-counts; Appendix E): D pre-norm residual blocks (a
// bias-free LSTM and a GELU MLP of hidden width 4 d_t, gain-only LayerNorm)
// at width d_t, between an input projection P_in from the head width d_E and
// an output projection P_out back to it, decoded by the expert's own tied
// matrix E [256][d_E], which is never perturbed.
//
// Canonical parameter order of one expert (every matrix row a multiple of 4
// long, so that a probe quad lies in one row of one matrix):
//   P_in [d_t][d_E]; per block A, R, U, V [d_t][4 d_t] (LSTM input and
//   recurrent weights with columns j = g d_t + u for gates g = i, f, g, o;
//   MLP up weights; MLP down weights, row = output feature); P_out [d_t][d_E];
//   gains g1, g2 per block, then g_f (each d_t long).
//
// A pass of this body runs, for every slot (expert, direction, sign):
//   k_wide_form   perturbed weights, gains folded into the matrices that
//                 read a normalised vector, zero-padded to d_p = 64 ceil(d_t
//                 / 64) and laid out for the kernels below (once per pass)
//   k_wide_mm     U = E P_in^T (the input projection per byte value)
//   k_wide_ln     x = U[byte], n = LN(x)   (the gain sits in the weights)
//   per block:    k_wide_mm gin = n A'      (gate inputs, units interleaved)
//                 k_rec_persist h           (recurrent weights pre-formed)
//                 k_wide_ln x += h, n = LN(x)
//                 k_wide_mm m = GELU(n U')
//                 k_wide_mm x += m V^T
//   k_wide_ln     n = LN(x)
//   k_wide_mm     u = n P_out'^T (the final gain folded into P_out)
//   k_wide_head   logits = u E^T, cross entropy
// Padded units have zero weights and zero gate inputs, so their cell state
// and h stay exactly 0 and every padded column of x stays 0.
#pragma once

#include "soma_kernels.hpp"
#include "soma_body.hpp"

namespace soma {

constexpr int kWideHeadWidth = 32;   // d_E of the GPU path (the paper's head width)
constexpr int kWidePad = 64;         // d_p: d_t rounded up to a multiple of this

__host__ __device__ constexpr int wide_padded(int dt) { return (dt + kWidePad - 1) / kWidePad * kWidePad; }

// Floats of one slot's pre-formed weights and their offsets.
struct WideForm {
  int64_t pin, blk0, blk_stride, pout, total;   // blk_stride: one block's four matrices
};

__host__ __device__ inline WideForm wide_form_layout(int dp, int D) {
  WideForm f{};
  const int64_t m = 4 * int64_t(dp) * dp;
  // Every matrix is stored output-major and split, [n][2][k] halves (a
  // row's hi parts, then its lo parts: the bytes of the fp32 matrix): the
  // rows of the gate matrices are interleaved (row 4 u + g is gate g of
  // unit u).
  f.pin = 0;                                   // P_in   [d_p][32]
  f.blk0 = int64_t(dp) * kWideHeadWidth;       // per block: A' [4 d_p][d_p], R [4 d_p][d_p],
  f.blk_stride = 4 * m;                        //   U' [4 d_p][d_p], V [d_p][4 d_p]
  f.pout = f.blk0 + int64_t(D) * f.blk_stride; // P_out' [32][d_p]
  f.total = f.pout + int64_t(dp) * kWideHeadWidth;
  return f;
}

struct WideArgs {
  const float* theta;     // [N][d]
  const uint64_t* seeds;  // [N]
  const uint8_t* bytes;   // [A][N][B][T]
  const float* E;         // tied matrices, expert e at E + e * e_stride, [256][32]
  int64_t e_stride;
  float* wform;           // pre-formed weights, [slots][WideForm::total]
  float* U;               // [slots][256][d_p]
  float* x;               // [slots][R][d_p] residual stream
  float* n;               // [slots][R][d_p] normalised x, split (also h of the recurrence, fp32)
  float* gin;             // [slots][R][4 d_p] gate inputs, then the MLP hidden layer
  double* part;           // [slots][row_tiles] cross-entropy sums
  float* fdec;            // evaluation: decoder inputs u [N][B][T-1][32] (position b (T-1) + t)
  float* lse;             // evaluation: log-sum-exps [N][B][T-1]
  int64_t d;              // parameters per expert
  uint64_t step;
  const float* eps_v;     // radius of expert e: eps_v[e * eps_stride]
  int eps_stride;
  unsigned* err;          // the step's sticky abort flag
  int probe;
  int ppb;                // directions per accumulation batch
  int64_t bstride;        // bytes per accumulation batch, N B T
  int N, D, dt, dp, B, T, PC, pcs, j0, NS;   // NS: signs per direction (2; 1 for an evaluation)
  int row_tiles;          // 64-row tiles of the head per slot
};

// Sum and max over the 64 lanes of a wave (butterfly; every lane gets the
// same value, each pair adding its two values in either order).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// Orders a wave's LDS writes before its later LDS reads of other lanes'
// words (a wave's LDS accesses execute in order; this keeps the compiler
// from moving them).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// One fp32 value -> its fp16 parts, as split2 does for a pair (hi rounded
// toward zero, lo the exact remainder rounded toward zero).
__device__ __forceinline__ void split1(float v, _Float16& hi, _Float16& lo) {
  const auto h = __builtin_amdgcn_cvt_pkrtz(v, 0.0f);
  hi = h[0];
  lo = __builtin_amdgcn_cvt_pkrtz(v - static_cast<float>(h[0]), 0.0f)[0];
}

// Slot s of the pass: (expert, direction in the pass, sign).
__device__ __forceinline__ void wide_slot(const WideArgs& a, int s, int& e, int& jl, int& sg) {
  sg = s % a.NS;
  const int pj = s / a.NS;
  jl = pj % a.pcs;
  e = pj / a.pcs;
}

__device__ __forceinline__ int64_t wide_slot_index(const WideArgs& a, int e, int jl, int sg) {
  return (int64_t(e) * a.PC + jl) * a.NS + sg;
}

// The perturbed value of canonical coordinate k of expert e (one probe quad
// drawn for it): theta_k + seps z_k.
__device__ __forceinline__ float wide_coord(const float* th, int64_t k, int64_t gain0, int law, uint2 key,
                                            uint32_t pair, uint32_t step_lo, float seps) {
  if (seps == 0.0f) return th[k];
  const int lw = (k >= gain0 && law == kProbeSparseRademacher) ? kProbeRademacher : law;
  const float4 z = probe_quad(lw, key, pair, step_lo, static_cast<uint64_t>(k & ~int64_t(3)));
  const float zz[4] = {z.x, z.y, z.z, z.w};
  return __builtin_fmaf(seps, zz[k & 3], th[k]);
}

// ---------------------------------------------------------------------------
// Pre-formed weights of every slot: one canonical probe quad per thread
// (grid: quads of the matrices, slots).  The gains are not stored: each
// matrix quad that reads a normalised vector multiplies by the perturbed gain
// of its row (one more probe quad).  Padded entries are zeroed beforehand
// (k_fill_f32).  A formed weight outside the split products' range, or NaN,
// sets the step's abort flag.
// ---------------------------------------------------------------------------
template <bool kPert>
__global__ __launch_bounds__(256) void k_wide_form(WideArgs a) {
  const int dt = a.dt, dp = a.dp, D = a.D;
  const int64_t dt4 = 4 * int64_t(dt), mat = dt4 * dt;
  const int64_t blk0 = int64_t(dt) * kWideHeadWidth, pout0 = blk0 + D * 4 * mat;
  const int64_t gain0 = pout0 + int64_t(dt) * kWideHeadWidth;
  const int64_t k = 4 * (blockIdx.x * int64_t(blockDim.x) + threadIdx.x);
  if (k >= gain0) return;
  int e, jl, sg;
  wide_slot(a, blockIdx.y, e, jl, sg);
  const int64_t slot = wide_slot_index(a, e, jl, sg);
  const float* th = a.theta + int64_t(e) * a.d;
  const uint2 key = kPert ? stream_key(a.seeds[e], a.step) : make_uint2(0u, 0u);
  const uint32_t pair = static_cast<uint32_t>(a.j0 + jl), step_lo = static_cast<uint32_t>(a.step);
  const float eps = kPert ? a.eps_v[int64_t(e) * a.eps_stride] : 0.0f;
  const float seps = sg == 0 ? eps : -eps;
  float w[4];
  if (kPert) {
    const int lw = a.probe;   // matrices follow the configured law
    const float4 z = probe_quad(lw, key, pair, step_lo, static_cast<uint64_t>(k));
    w[0] = __builtin_fmaf(seps, z.x, th[k]);
    w[1] = __builtin_fmaf(seps, z.y, th[k + 1]);
    w[2] = __builtin_fmaf(seps, z.z, th[k + 2]);
    w[3] = __builtin_fmaf(seps, z.w, th[k + 3]);
  } else {
    w[0] = th[k]; w[1] = th[k + 1]; w[2] = th[k + 2]; w[3] = th[k + 3];
  }
  const WideForm F = wide_form_layout(dp, D);
  _Float16* out = reinterpret_cast<_Float16*>(a.wform + slot * F.total);
  bool ok = true;
  // Element (row, col) of a matrix at float offset base with rows of K
  // values, stored split: row r is K hi parts then K lo parts.
  auto put = [&](int64_t base, int64_t row, int64_t col, int64_t K, float v) {
    ok = ok && __builtin_fabsf(v) <= kSplitMax;
    _Float16 h, l;
    split1(v, h, l);
    _Float16* p = out + 2 * base + row * 2 * K + col;
    p[0] = h;
    p[K] = l;
  };
  if (k < blk0) {                                     // P_in [c][q]
    const int64_t c = k / kWideHeadWidth, q = k % kWideHeadWidth;
    for (int i = 0; i < 4; ++i) put(F.pin, c, q + i, kWideHeadWidth, w[i]);
  } else if (k < pout0) {
    const int64_t r = k - blk0;
    const int l = static_cast<int>(r / (4 * mat));
    const int which = static_cast<int>((r / mat) % 4);
    const int64_t rr = r % mat, c = rr / dt4, j = rr % dt4;
    const int64_t mp = 4 * int64_t(dp) * dp, base = F.blk0 + l * F.blk_stride + which * mp;
    float g = 1.0f;
    if (which == 0 || which == 2)                     // A reads LN(x; g1), U reads LN(x; g2)
      g = wide_coord(th, gain0 + (2 * l + (which == 2 ? 1 : 0)) * int64_t(dt) + c, gain0, a.probe, key, pair,
                     step_lo, seps);
    for (int i = 0; i < 4; ++i) {
      const int64_t jj = j + i;
      if (which <= 1) {                               // gate column g dt + u -> row 4 u + g (A' and R)
        const int64_t gate = jj / dt, u = jj % dt;
        put(base, 4 * u + gate, c, dp, which == 0 ? w[i] * g : w[i]);
      } else if (which == 2) {                        // U'[j][c]
        put(base, jj, c, dp, w[i] * g);
      } else {                                        // V[c][j]: row = output feature
        put(base, c, jj, 4 * int64_t(dp), w[i]);
      }
    }
  } else {                                            // P_out'[q][c] = P_out[c][q] g_f[c]
    const int64_t r = k - pout0, c = r / kWideHeadWidth, q = r % kWideHeadWidth;
    const float g = wide_coord(th, gain0 + 2 * int64_t(D) * dt + c, gain0, a.probe, key, pair, step_lo, seps);
    for (int i = 0; i < 4; ++i) put(F.pout, q + i, c, dp, w[i] * g);
  }
  report_split_range(a.err, ok);
}

// out[i] = 0 for i < n (a fill kernel, so that callers may capture it).
__global__ void k_fill_f32(float* out, int64_t n) {
  for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x)
    out[i] = 0.0f;
}

// ---------------------------------------------------------------------------
// Batched products on the fp16 matrix cores from split fp32 operands:
//   C[s][m][n] (= | += | GELU of) sum_k A[s][m][k] W[s][n][k]
// W is stored split ([N][2][K] halves: per row its K hi parts, then its K lo
// parts), as the form kernel writes it.  A is either stored split the same
// way ([M][2][K], written so by LayerNorm and by the GELU epilogue) or fp32
// [M][K], split as it is staged (the tied matrix of the input projection);
// per slot, or per expert.  C is fp32 [M][N] (store, add), or split
// [M][2][N] (GELU: the next product's A).  Block tile 128 (n) x 128 (m),
// four waves of 64 x 64; K in 32-wide chunks (K % 32 == 0, N % 4 == 0)
// staged through two LDS buffers: chunk c + 1's global loads are in flight
// during chunk c's products and stored into the other buffer after them,
// one block barrier per chunk.  Tiles are dealt so that each XCD (blocks go to
// the 8 XCDs round-robin) works through a contiguous range of them: the n
// tiles of one m tile, and the m tiles of one slot, share its L2.
// ---------------------------------------------------------------------------
enum WideEpi { kEpiStore = 0, kEpiGelu = 1, kEpiAdd = 2 };

struct MmArgs {
  const void* A;
  int64_t a_slot;     // A elements (floats or split pairs) between consecutive A matrices (slots, or experts)
  int a_expert;       // A is per expert rather than per slot
  const void* W;      // split
  int64_t w_slot;     // floats (split pairs) between slots' matrices
  void* C;
  int64_t c_slot;     // elements between slots' outputs
  int M, N, K;
  int pcs, PC, NS;    // the pass's slots
  int ntn, ntm;       // n tiles, m tiles
  int64_t tiles;      // ntn * ntm * slots
  unsigned* err;
};

constexpr int kMmLd = 80;   // LDS row in halves: 32 hi, 32 lo, 16 spare (160 bytes, an odd multiple of 32)
constexpr int kXcds = 8;

template <bool kASplit, int kEpi>
__global__ __launch_bounds__(256) void k_wide_mm(MmArgs p) {
  __shared__ __attribute__((aligned(16))) _Float16 sa[2][128 * kMmLd];   // [buffer] activations, rows hi | lo
  __shared__ __attribute__((aligned(16))) _Float16 sw[2][128 * kMmLd];   // [buffer] weights, rows hi | lo
  const int64_t per_xcd = (p.tiles + kXcds - 1) / kXcds;
  const int64_t tile = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
  if (tile >= p.tiles) return;                          // block-uniform
  const int nt = static_cast<int>(tile % p.ntn);
  const int64_t rest = tile / p.ntn;
  const int mtile = static_cast<int>(rest % p.ntm), z = static_cast<int>(rest / p.ntm);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  const int wn = wave & 1, wm = wave >> 1;
  const int n0 = nt * 128, m0 = mtile * 128;
  const int sg = z % p.NS, jl = (z / p.NS) % p.pcs, e = z / (p.NS * p.pcs);
  const int64_t s = (int64_t(e) * p.PC + jl) * p.NS + sg;
  const int64_t a_off = (p.a_expert ? int64_t(e) : s) * p.a_slot;
  const int M = p.M, N = p.N, K = p.K;
  const _Float16* Wh = reinterpret_cast<const _Float16*>(p.W) + 2 * s * p.w_slot;
  bool ok = true;

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Staging: a split row chunk is 32 hi then 32 lo halves (4 uint4 each);
  // an fp32 row chunk is 8 float4.  Thread idx = t + 256 i covers row
  // idx >> 3 and piece idx & 7 of both operands.
  uint4 pa[4], pw[4];
  float4 pf[4];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = threadIdx.x + 256 * i;
      const int row = idx >> 3, pc = idx & 7, part = pc >> 2, q = pc & 3;
      const int m = m0 + row, n = n0 + row;
      if constexpr (kASplit) {
        const _Float16* A = reinterpret_cast<const _Float16*>(p.A) + 2 * a_off;
        pa[i] = m < M ? *reinterpret_cast<const uint4*>(A + int64_t(m) * 2 * K + part * K + k0 + 8 * q)
                      : make_uint4(0u, 0u, 0u, 0u);
      } else {
        const float* A = reinterpret_cast<const float*>(p.A) + a_off;
        pf[i] = m < M ? *reinterpret_cast<const float4*>(A + int64_t(m) * K + k0 + 4 * pc)
                      : make_float4(0.f, 0.f, 0.f, 0.f);
      }
      pw[i] = n < N ? *reinterpret_cast<const uint4*>(Wh + int64_t(n) * 2 * K + part * K + k0 + 8 * q)
                    : make_uint4(0u, 0u, 0u, 0u);
    }
  };
  auto sstore = [&](int b) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = threadIdx.x + 256 * i;
      const int row = idx >> 3, pc = idx & 7, part = pc >> 2, q = pc & 3;
      if constexpr (kASplit) {
        *reinterpret_cast<uint4*>(&sa[b][row * kMmLd + 32 * part + 8 * q]) = pa[i];
      } else {
        uint2 hi, lo;
        ok = ok && split_range_ok(pf[i]);
        split4(pf[i], hi, lo);
        *reinterpret_cast<uint2*>(&sa[b][row * kMmLd + 4 * pc]) = hi;
        *reinterpret_cast<uint2*>(&sa[b][row * kMmLd + 32 + 4 * pc]) = lo;
      }
      *reinterpret_cast<uint4*>(&sw[b][row * kMmLd + 32 * part + 8 * q]) = pw[i];
    }
  };

  gload(0);
  sstore(0);
  __syncthreads();
  const int nk = K / 32;
  for (int c = 0; c < nk; ++c) {
    const int b = c & 1;
    if (c + 1 < nk) gload(32 * (c + 1));
    uint4 bh[4], bl[4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      const int row = wm * 64 + 16 * mt + lr;
      bh[mt] = *reinterpret_cast<const uint4*>(&sa[b][row * kMmLd + 8 * lg]);
      bl[mt] = *reinterpret_cast<const uint4*>(&sa[b][row * kMmLd + 32 + 8 * lg]);
    }
#pragma unroll
    for (int ntl = 0; ntl < 4; ++ntl) {
      const int row = wn * 64 + 16 * ntl + lr;
      const uint4 wh = *reinterpret_cast<const uint4*>(&sw[b][row * kMmLd + 8 * lg]);
      const uint4 wl = *reinterpret_cast<const uint4*>(&sw[b][row * kMmLd + 32 + 8 * lg]);
      mfma3_batch<4>(wh, wl, bh, bl, acc[ntl]);
    }
    // The other buffer was last read in chunk c - 1, before the barrier
    // that ended it.
    if (c + 1 < nk) sstore(b ^ 1);
    __syncthreads();
  }

  // acc[ntl][mt][i] = C[m0 + 64 wm + 16 mt + lr][n0 + 64 wn + 16 ntl + 4 lg + i]
#pragma unroll
  for (int ntl = 0; ntl < 4; ++ntl) {
    const int n = n0 + wn * 64 + 16 * ntl + 4 * lg;
    if (n >= N) continue;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      const int m = m0 + wm * 64 + 16 * mt + lr;
      if (m >= M) continue;
      float4 v = make_float4(acc[ntl][mt][0], acc[ntl][mt][1], acc[ntl][mt][2], acc[ntl][mt][3]);
      if constexpr (kEpi == kEpiGelu) {
        v = make_float4(gelu_f(v.x), gelu_f(v.y), gelu_f(v.z), gelu_f(v.w));
        ok = ok && split_range_ok(v);
        uint2 hi, lo;
        split4(v, hi, lo);
        _Float16* C = reinterpret_cast<_Float16*>(p.C) + 2 * s * p.c_slot + int64_t(m) * 2 * N + n;
        *reinterpret_cast<uint2*>(C) = hi;
        *reinterpret_cast<uint2*>(C + N) = lo;
      } else {
        float4* c = reinterpret_cast<float4*>(reinterpret_cast<float*>(p.C) + s * p.c_slot + int64_t(m) * N + n);
        if constexpr (kEpi == kEpiAdd) {
          const float4 o = *c;
          v = make_float4(o.x + v.x, o.y + v.y, o.z + v.z, o.w + v.w);
        }
        *c = v;
      }
    }
  }
  report_split_range(p.err, ok);
}

// ---------------------------------------------------------------------------
// Gain-free LayerNorm of every row of x, one wave per row (four per block):
//   kMode 0: x = U[byte]          (the embedding's projection per byte value)
//   kMode 1: x += h               (the LSTM sublayer's residual; h in n)
//   kMode 2: x as it is
// then n = (x - mean) / sqrt(var + 1e-5) over the first d_t features (biased
// variance), 0 on the padded ones, written split (the row's hi parts, then
// its lo parts) over the fp32 row of h it replaces.  Rows are r = t B + b.
// ---------------------------------------------------------------------------
template <int kMode>
__global__ __launch_bounds__(256) void k_wide_ln(WideArgs a) {
  constexpr int kMaxC = 8;   // d_p <= 512
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t R = int64_t(a.T - 1) * a.B;
  const int64_t r = int64_t(blockIdx.x) * 4 + wave;
  if (r >= R) return;
  const int s = blockIdx.y;
  int e, jl, sg;
  wide_slot(a, s, e, jl, sg);
  const int64_t slot = wide_slot_index(a, e, jl, sg);
  const int dp = a.dp, dt = a.dt, nc = dp / 64;
  float* xr = a.x + (slot * R + r) * dp;
  float* nr = a.n + (slot * R + r) * dp;
  float v[kMaxC];
  if (kMode == 0) {
    const int64_t t = r / a.B, b = r % a.B;
    const uint8_t* by = a.bytes + int64_t((a.j0 + jl) / a.ppb) * a.bstride + (int64_t(e) * a.B + b) * a.T;
    const float* ur = a.U + (slot * kVocab + by[t]) * dp;
#pragma unroll
    for (int i = 0; i < kMaxC; ++i)
      if (i < nc) {
        v[i] = ur[64 * i + lane];
        xr[64 * i + lane] = v[i];
      }
  } else {
#pragma unroll
    for (int i = 0; i < kMaxC; ++i)
      if (i < nc) {
        v[i] = xr[64 * i + lane];
        if (kMode == 1) {
          v[i] += nr[64 * i + lane];
          xr[64 * i + lane] = v[i];
        }
      }
  }
  float sum = 0.0f;
#pragma unroll
  for (int i = 0; i < kMaxC; ++i)
    if (i < nc && 64 * i + lane < dt) sum += v[i];
  sum = wave_sum(sum);
  const float mean = sum / static_cast<float>(dt);
  float sq = 0.0f;
#pragma unroll
  for (int i = 0; i < kMaxC; ++i)
    if (i < nc && 64 * i + lane < dt) {
      const float c = v[i] - mean;
      sq = __builtin_fmaf(c, c, sq);
    }
  sq = wave_sum(sq);
  const float inv = 1.0f / __builtin_sqrtf(sq / static_cast<float>(dt) + 1e-5f);
  // n, split into its fp16 parts: the row's dp hi parts, then its dp lo
  // parts (the bytes of the fp32 row it replaces).
  _Float16* ns = reinterpret_cast<_Float16*>(nr);
#pragma unroll
  for (int i = 0; i < kMaxC; ++i)
    if (i < nc) {
      const float y = 64 * i + lane < dt ? (v[i] - mean) * inv : 0.0f;
      _Float16 h, l;
      split1(y, h, l);
      ns[64 * i + lane] = h;
      ns[dp + 64 * i + lane] = l;
    }
}

// ---------------------------------------------------------------------------
// The decoder: logits = u E^T over the 256 byte values and the cross entropy
// against the next byte, u = n P_out'^T from the products above ([R][32] per
// slot, row stride u_ld).  One wave per row; lane l keeps rows l, l + 64,
// l + 128, l + 192 of the expert's E in registers, and u is broadcast from
// the lanes that loaded it.  A block covers kWideHeadRows rows of a slot and
// writes their sum of cross entropies to part[slot][tile] (fp64, rows in
// order).  Evaluations also write u and the log-sum-exp per position
// b (T-1) + t for the delta rule.  fp32 products on the vector ALU.
// ---------------------------------------------------------------------------
constexpr int kWideHeadRows = 256;

template <bool kEval>
__global__ __launch_bounds__(256) void k_wide_head(WideArgs a, const float* u_base, int64_t u_slot, int u_ld) {
  constexpr int EW = kWideHeadWidth;
  constexpr int RPW = kWideHeadRows / 4;     // rows per wave
  __shared__ double ce_w[4];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int tile = blockIdx.x, s = blockIdx.y;
  int e, jl, sg;
  wide_slot(a, s, e, jl, sg);
  const int64_t slot = wide_slot_index(a, e, jl, sg);
  const int64_t R = int64_t(a.T - 1) * a.B;
  const float* Ee = a.E + int64_t(e) * a.e_stride;
  float ev[4][EW];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int k = 0; k < EW; k += 4) {
      const float4 v = *reinterpret_cast<const float4*>(Ee + (lane + 64 * j) * EW + k);
      ev[j][k] = v.x; ev[j][k + 1] = v.y; ev[j][k + 2] = v.z; ev[j][k + 3] = v.w;
    }
  const uint8_t* by = a.bytes + int64_t((a.j0 + jl) / a.ppb) * a.bstride + int64_t(e) * a.B * a.T;
  const float* ub = u_base + slot * u_slot;
  double ce_sum = 0.0;
  for (int i = 0; i < RPW; ++i) {
    const int64_t r = int64_t(tile) * kWideHeadRows + wave * RPW + i;
    if (r >= R) break;                                 // wave-uniform
    const float u = lane < EW ? ub[r * u_ld + lane] : 0.0f;
    float lg[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < EW; ++k) {
      const float uk = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(u), k));
#pragma unroll
      for (int j = 0; j < 4; ++j) lg[j] = __builtin_fmaf(ev[j][k], uk, lg[j]);
    }
    float mx = fmaxf(fmaxf(lg[0], lg[1]), fmaxf(lg[2], lg[3]));
    mx = wave_max(mx);
    float se = 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j) se += __expf(lg[j] - mx);
    se = wave_sum(se);
    const float lse = __logf(se) + mx;
    const int64_t t = r / a.B, b = r % a.B;
    const int y = by[b * a.T + t + 1];
    const float ly = __shfl(lg[y >> 6], y & 63);
    ce_sum += static_cast<double>(lse - ly);
    if (kEval) {
      const int64_t pos = int64_t(e) * R + b * (a.T - 1) + t;
      if (lane < EW) a.fdec[pos * EW + lane] = u;
      if (lane == 0) a.lse[pos] = lse;
    }
  }
  if (lane == 0) ce_w[wave] = ce_sum;
  __syncthreads();
  if (threadIdx.x == 0) a.part[slot * a.row_tiles + tile] = ((ce_w[0] + ce_w[1]) + ce_w[2]) + ce_w[3];
}

}  // namespace soma

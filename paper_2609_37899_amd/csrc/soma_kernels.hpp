// soma_kernels.hpp -- gfx950 kernels of the SOMA SPSA step.
//
// Data layout in HBM (fp32 unless noted; "slot" = (expert e, direction jl of
// the current chunk, sign s), slot = (e * PC + jl) * NS + s with NS = 2 signs
// in a step and 1 in evaluation):
//   theta [N][d]                 canonical parameter order (see soma.h)
//   bytes [N][B][T] uint8
//   U     [slot][256][4H]        layer-1 gate inputs per byte value:
//                                U[v] = Emb[v] W_1x^T (the embedding row times
//                                the input half of W_1, re-associated once per
//                                slot instead of once per token)
//   gin   [slot][T-1][B][4H]     gate inputs of layers >= 2 (x_t W_lx^T)
//   hseq  [slot][T-1][B][H]      hidden states of the current layer
//   cst   [slot][B][H]           cell state of the current layer
//   part  [slot][row tiles]      per-tile sums of cross entropy (fp64)
// The last axis of U and gin is gate-interleaved: column 4u + g holds gate g
// (i, f, g, o) of unit u, so that one MFMA output lane holds the four gates
// of one unit.
//
// Matrix cores: V_MFMA_F32_16X16X4_F32.  For A (16 x 4), B (4 x 16) and
// D (16 x 16), lane l supplies A[l % 16][l / 16] and B[l / 16][l % 16] and
// receives D[4 (l / 16) + r][l % 16] in accumulator register r.  Every
// contraction here is D = W x^T with the perturbed weight W in the A slot
// (rows = gate rows or vocabulary rows) and activations in the B slot
// (columns = batch rows).  A lane loads W[m][k .. k+3] and x[n][k .. k+3] as
// float4 along k and feeds component s to the s-th of four MFMAs, which
// permutes the order of k inside a 16-wide group identically on both
// operands.  The four consecutive k of one W row are exactly one Philox
// counter, so each lane draws its own probe quad in registers: the probe is
// generated where the weight tile is loaded and never stored.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "soma_rng.hpp"

namespace soma {

constexpr int kVocab = 256;
constexpr int kThreads = 256;  // 4 waves of 64

typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// acc += W(float4 along k) . X(float4 along k) over one 16-wide k group.
__device__ __forceinline__ f32x4 mfma_k16(const float4& w, const float4& x, f32x4 acc) {
  acc = mfma4(w.x, x.x, acc);
  acc = mfma4(w.y, x.y, acc);
  acc = mfma4(w.z, x.z, acc);
  acc = mfma4(w.w, x.w, acc);
  return acc;
}

// ---------------------------------------------------------------------------
// Split fp16 products.  gfx950's fp32 matrix instructions share their
// datapath with the vector ALU (one wave's or two waves' fp32 MFMAs and
// vector instructions take the sum of their times), while its fp16 matrix
// cores (V_MFMA_F32_16X16X32_F16) run alongside the vector ALU at 16 times
// the fp32 matrix rate.  The streaming and persistent kernels therefore form
// their fp32 products there: each fp32 operand is split into two fp16 parts,
// x = hi + lo (hi = x rounded toward zero to fp16; lo = the remainder, exact
// in fp32, rounded toward zero), and
//   A B = A_lo B_hi + A_hi B_lo + A_hi B_hi   (the lo * lo term dropped)
// is accumulated in fp32: about 21 significant bits per operand.  K runs in
// chunks of 32; lane group g = lane / 16 supplies the 8 consecutive K values
// 32 p + 8 g .. + 7 of chunk p for both operands, and its 16 lanes the rows
// (A) or columns (B); the result block is laid out as for the fp32 MFMA.
// ---------------------------------------------------------------------------
typedef _Float16 h8 __attribute__((ext_vector_type(8)));

// Two fp32 values -> their fp16 parts: hi = (h(x0), h(x1)), lo = (h(x0 -
// hi0), h(x1 - hi1)), both rounded toward zero; x - hi is exact in fp32.
__device__ __forceinline__ void split2(float x0, float x1, uint32_t& hi, uint32_t& lo) {
  const auto h = __builtin_amdgcn_cvt_pkrtz(x0, x1);
  const float r0 = x0 - static_cast<float>(h[0]), r1 = x1 - static_cast<float>(h[1]);
  hi = __builtin_bit_cast(uint32_t, h);
  lo = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(r0, r1));
}

// Range of the split.  hi saturates at 65504, the largest finite fp16 (the
// conversion rounds toward zero), so an operand is represented only for
// |x| <= kSplitMax; below 2^-3 lo, and below 2^-14 hi too, fall into fp16's
// subnormals, whose spacing 2^-24 bounds the absolute error there.  So the
// split keeps |x - (hi + lo)| <= 2^-21 |x| + 2^-24 for |x| <= kSplitMax: about
// 21 significant bits from |x| = 2^-3 up, fewer below.  Activations of the
// stacked LSTM are bounded by 1 (h = o tanh(c)); every kernel that forms a
// split weight checks it against kSplitMax (NaN included) and aborts the step
// through the sticky flag (bit kAbortRange) if one is outside.
constexpr float kSplitMax = 65504.0f;
constexpr unsigned kAbortRange = 2u;

__device__ __forceinline__ bool split_range_ok(const float4& v, float bound = kSplitMax) {
  // false for NaN as well
  return __builtin_fabsf(v.x) <= bound && __builtin_fabsf(v.y) <= bound && __builtin_fabsf(v.z) <= bound &&
         __builtin_fabsf(v.w) <= bound;
}

// Sets the step's abort flag if this lane formed a weight outside the range.
__device__ __forceinline__ void report_split_range(unsigned* err, bool ok) {
  if (!ok && err) __hip_atomic_fetch_or(err, kAbortRange, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Four consecutive fp32 values -> 8 bytes of hi parts and 8 bytes of lo parts.
__device__ __forceinline__ void split4(const float4& v, uint2& hi, uint2& lo) {
  split2(v.x, v.y, hi.x, lo.x);
  split2(v.z, v.w, hi.y, lo.y);
}

// Eight consecutive fp32 values (two float4) -> one 8-half fragment each.
__device__ __forceinline__ void split8v(const float4& a, const float4& b, uint4& hi, uint4& lo) {
  uint2 h0, l0, h1, l1;
  split4(a, h0, l0);
  split4(b, h1, l1);
  hi = make_uint4(h0.x, h0.y, h1.x, h1.y);
  lo = make_uint4(l0.x, l0.y, l1.x, l1.y);
}

// acc[nb] += A B_nb over one 32-wide K chunk from split fragments (8 halves
// per lane: A = A_hi + A_lo, B = B_hi + B_lo, the lo x lo product dropped)
// for NT row tiles that share the A fragments; the B fragments of every
// tile are read beforehand.  Each pass runs over the tiles, so neighbouring
// MFMAs use independent accumulators: one tile at a time would serialise
// the three passes behind each other and behind the tile's LDS reads.
template <int NT>
__device__ __forceinline__ void mfma3_batch(const uint4& ah, const uint4& al, const uint4 (&bh)[NT],
                                            const uint4 (&bl)[NT], f32x4 (&acc)[NT]) {
  const h8 AH = __builtin_bit_cast(h8, ah), AL = __builtin_bit_cast(h8, al);
#pragma unroll
  for (int nb = 0; nb < NT; ++nb)
    acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(AL, __builtin_bit_cast(h8, bh[nb]), acc[nb], 0, 0, 0);
#pragma unroll
  for (int nb = 0; nb < NT; ++nb)
    acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(AH, __builtin_bit_cast(h8, bl[nb]), acc[nb], 0, 0, 0);
#pragma unroll
  for (int nb = 0; nb < NT; ++nb)
    acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(AH, __builtin_bit_cast(h8, bh[nb]), acc[nb], 0, 0, 0);
}

// Pieces of K = 64 NCH staged per pass of the streaming and persistent
// kernels, each 64 or 128 wide (a whole number of 32-wide chunks).
__host__ __device__ constexpr int split_quarters(int nch) {
  return nch <= 4 ? nch : (nch % 4 == 0 ? 4 : (nch % 3 == 0 ? 3 : nch));
}

__device__ __forceinline__ float4 fma4(float a, const float4& z, const float4& t) {
  return make_float4(__builtin_fmaf(a, z.x, t.x), __builtin_fmaf(a, z.y, t.y),
                     __builtin_fmaf(a, z.z, t.z), __builtin_fmaf(a, z.w, t.w));
}

constexpr float kLog2e = 1.4426950408889634f;

// 2^x on the transcendental unit.
__device__ __forceinline__ float exp2_f(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float sigmoid_f(float x) {
  return __builtin_amdgcn_rcpf(1.0f + __expf(-x));
}

// Max and sum over the four lane groups (lanes l, l ^ 16, l ^ 32, l ^ 48),
// every lane receiving the result, on the vector ALU: with both operands
// holding x, permlane16_swap leaves x of the lane and of lane ^ 16 in the
// pair (odd 16-lane rows of one operand trade places with even rows of the
// other), permlane32_swap likewise for lane ^ 32.  Both lanes of a pair add
// the same two values in the same order, so every lane holds the same sum.
__device__ __forceinline__ float group4_max(float v) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float group4_sum(float v) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// One LSTM cell from its gate pre-activations (i, f, g, o):
//   c <- sigma(f) c + sigma(i) tanh(g),  h = sigma(o) tanh(c),
// with sigma(x) = 1 / (1 + e^{-x}) and tanh(x) = sgn(x) (1 - e^{-2|x|}) /
// (1 + e^{-2|x|}), each product of a sigmoid and a tanh over one common
// denominator: five exponentials and three reciprocals.  No exponent is
// positive except those of sigma, whose overflow to +inf gives 0 (a
// denominator of +inf), never NaN.
__device__ __forceinline__ void lstm_cell(float ai, float af, float ag, float ao, float& c, float& h) {
  const float ef = exp2_f(-kLog2e * af), ei = exp2_f(-kLog2e * ai), eo = exp2_f(-kLog2e * ao);
  const float eg = exp2_f(-2.0f * kLog2e * __builtin_fabsf(ag));
  const float sf = __builtin_amdgcn_rcpf(1.0f + ef);
  const float ig = __builtin_copysignf((1.0f - eg) * __builtin_amdgcn_rcpf((1.0f + ei) * (1.0f + eg)), ag);
  c = __builtin_fmaf(sf, c, ig);
  const float ec = exp2_f(-2.0f * kLog2e * __builtin_fabsf(c));
  h = __builtin_copysignf((1.0f - ec) * __builtin_amdgcn_rcpf((1.0f + eo) * (1.0f + ec)), c);
}

// The cell update from pre-activations already multiplied by gate_scale(g)
// (-log2 e for the gates i, f, o; 2 log2 e for the candidate g): the
// exponentials' arguments come straight from the products, |x| and the sign
// of the candidate being source modifiers.  Same formulas as lstm_cell.
__host__ __device__ constexpr float gate_scale(int g) { return g == 2 ? 2.0f * kLog2e : -kLog2e; }

__device__ __forceinline__ void lstm_cell_scaled(float pi, float pf, float pg, float po, float& c, float& h) {
  const float ef = exp2_f(pf), ei = exp2_f(pi), eo = exp2_f(po);
  const float eg = exp2_f(-__builtin_fabsf(pg));
  const float sf = __builtin_amdgcn_rcpf(1.0f + ef);
  const float ig = __builtin_copysignf((1.0f - eg) * __builtin_amdgcn_rcpf((1.0f + ei) * (1.0f + eg)), pg);
  c = __builtin_fmaf(sf, c, ig);
  const float ec = exp2_f(-2.0f * kLog2e * __builtin_fabsf(c));
  h = __builtin_copysignf((1.0f - ec) * __builtin_amdgcn_rcpf((1.0f + eo) * (1.0f + ec)), c);
}

__device__ __forceinline__ float tanh_f(float x) {
  // 1 - 2 / (e^{2x} + 1), saturating correctly for large |x|.
  return 1.0f - 2.0f * __builtin_amdgcn_rcpf(__expf(2.0f * x) + 1.0f);
}

// Shape and workspace pointers shared by the forward kernels.
struct FwdArgs {
  const float* theta;     // [N][d]
  const uint8_t* bytes;   // [N][B][T]
  const uint64_t* seeds;  // [N]
  float* U;
  float* gin;
  float* hseq;
  float* cst;
  double* part;
  int64_t d;        // parameters per expert
  int64_t off_l;    // canonical offset of W_l (current layer)
  int64_t off_head; // canonical offset of Whead
  uint64_t step;
  const float* eps_v;     // perturbation radius of expert e: eps_v[e * eps_stride]
  int eps_stride;
  unsigned pmask;         // perturbed parameter groups (kGroup* bits; all three when nothing is masked)
  unsigned* err;          // the step's sticky abort flag (a split weight out of range sets kAbortRange)
  int probe;              // probe law (kProbe*)
  int ppb;                // directions per accumulation batch (direction j reads batch j / ppb)
  int64_t bstride;        // bytes per accumulation batch, N B T
  int N, E, H, B, T, PC;  // PC = slot stride in directions
  int pcs;                // directions in this pass (grid extent)
  int j0;                 // first direction of the chunk
  int layer;              // current layer (0-based)
  int in_l;               // input width of the current layer
  int t;                  // time step (rec kernel)
  int row_tiles;          // head row tiles per slot
  // The persistent recurrence's pre-formed instantiation only: perturbed
  // recurrent weights formed beforehand, slot s's matrix at wpre + s *
  // wpre_slot, [4H][2][H] halves (each row's hi parts, then its lo parts)
  // with row 4 u + g = gate g of unit u; and the signs
  // per direction of the pass (1: one unperturbed job per expert, else both
  // signs).
  const float* wpre;
  int64_t wpre_slot;
  int ns;
};

// Parameter groups of the stacked LSTM that the perturbation mask names: the
// embedding, the LSTM layers and the head.  A masked group is formed with
// radius 0, i.e. theta itself (fma(0, z, theta) == theta for finite z).
constexpr unsigned kGroupEmb = 1, kGroupLstm = 2, kGroupHead = 4;

// The radius of expert e for the weights of parameter group `group`.
__device__ __forceinline__ float eps_of(const FwdArgs& a, int e, unsigned group) {
  return (a.pmask & group) ? a.eps_v[int64_t(e) * a.eps_stride] : 0.0f;
}

// Expert e's batch [B][T] for direction j0 + jl of the pass (its
// accumulation batch).
__device__ __forceinline__ const uint8_t* bytes_of(const FwdArgs& a, int e, int jl) {
  return a.bytes + int64_t((a.j0 + jl) / a.ppb) * a.bstride + int64_t(e) * a.B * a.T;
}

// ---------------------------------------------------------------------------
// Layer-1 gate inputs per byte value (the vocabulary fold).
//   U[slot][v][4u+g] = sum_{k<E} Emb+-[v][k] W_1+-[g H + u][k]
// Both operands are perturbed (same direction, same sign).  Grid:
// (4H/64 gate-row tiles, 4 vocabulary tiles, N * chunk).  Each wave owns 16
// gate rows; the 64 embedding rows of the tile are perturbed cooperatively
// into LDS, both signs from one probe quad.
// ---------------------------------------------------------------------------
template <bool kPert>
__global__ __launch_bounds__(kThreads) void k_fold(FwdArgs a) {
  constexpr int NS = kPert ? 2 : 1;
  constexpr int KC = 64, LDK = KC + 8;
  __shared__ float es[NS][64][LDK];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  const int mtile = blockIdx.x, v0 = blockIdx.y * 64;
  const int e = blockIdx.z / a.pcs, jl = blockIdx.z % a.pcs;
  const int E = a.E, H = a.H;
  const float* th = a.theta + static_cast<int64_t>(e) * a.d;
  const uint2 key = kPert ? stream_key(a.seeds[e], a.step) : make_uint2(0u, 0u);
  const float eps_e = kPert ? eps_of(a, e, kGroupEmb) : 0.0f;    // the embedding rows
  const float eps = kPert ? eps_of(a, e, kGroupLstm) : 0.0f;     // the input columns of W_1
  const uint32_t pair = static_cast<uint32_t>(a.j0 + jl), step_lo = static_cast<uint32_t>(a.step);
  const int prow = mtile * 64 + wave * 16 + lr;
  const int64_t wrow = a.off_l + static_cast<int64_t>((prow & 3) * H + (prow >> 2)) * (E + H);

  f32x4 acc[NS][4];
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) acc[s][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int k0 = 0; k0 < E; k0 += KC) {
    const int kc = min(KC, E - k0);
    __syncthreads();
    for (int idx = threadIdx.x; idx < 64 * (kc / 4); idx += kThreads) {
      const int n = idx / (kc / 4), c4 = idx % (kc / 4);
      const int64_t kk = static_cast<int64_t>(v0 + n) * E + k0 + 4 * c4;
      const float4 t4 = *reinterpret_cast<const float4*>(th + kk);
      if (kPert) {
        const float4 z = probe_quad(a.probe, key, pair, step_lo, static_cast<uint64_t>(kk));
        *reinterpret_cast<float4*>(&es[0][n][4 * c4]) = fma4(eps_e, z, t4);
        *reinterpret_cast<float4*>(&es[NS - 1][n][4 * c4]) = fma4(-eps_e, z, t4);
      } else {
        *reinterpret_cast<float4*>(&es[0][n][4 * c4]) = t4;
      }
    }
    __syncthreads();
    for (int g = 0; g < kc / 16; ++g) {
      const int64_t kw = wrow + k0 + 16 * g + 4 * lg;
      const float4 t4 = *reinterpret_cast<const float4*>(th + kw);
      float4 w[NS];
      if (kPert) {
        const float4 z = probe_quad(a.probe, key, pair, step_lo, static_cast<uint64_t>(kw));
        w[0] = fma4(eps, z, t4);
        w[NS - 1] = fma4(-eps, z, t4);
      } else {
        w[0] = t4;
      }
#pragma unroll
      for (int nb = 0; nb < 4; ++nb)
#pragma unroll
        for (int s = 0; s < NS; ++s) {
          const float4 x = *reinterpret_cast<const float4*>(&es[s][nb * 16 + lr][16 * g + 4 * lg]);
          acc[s][nb] = mfma_k16(w[s], x, acc[s][nb]);
        }
    }
  }
  const int p = mtile * 64 + wave * 16 + 4 * lg;
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const int64_t slot = (static_cast<int64_t>(e) * a.PC + jl) * NS + s;
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
      const int v = v0 + nb * 16 + lr;
      float* dst = a.U + (slot * kVocab + v) * (4 * static_cast<int64_t>(H)) + p;
      *reinterpret_cast<float4*>(dst) =
          make_float4(acc[s][nb][0], acc[s][nb][1], acc[s][nb][2], acc[s][nb][3]);
    }
  }
}

// ---------------------------------------------------------------------------
// Shared main loop of the contractions D = W x^T with a perturbed weight.
//
// Each wave owns MB blocks of 16 weight rows (canonical row starts wrow[mb]);
// a lane regenerates the probe quad of W[m][k .. k+3] for its row m = lane%16
// and k = 16 g + 4 (lane/16) and forms both signs in registers.  The
// activations (NS signs x NBR*16 rows x 32 k) are prefetched into registers
// one chunk ahead and staged through a double-buffered LDS tile (one barrier
// per chunk).  act(s, n, k) returns the float4 x[s][n][k .. k+3] or zeros.
// ---------------------------------------------------------------------------
constexpr int kChunk = 32;            // k per LDS chunk (two 16-wide groups)
constexpr int kLdk = kChunk + 8;      // padded LDS row (an odd multiple of 8 floats): conflict-free b128 reads

template <int NS, int NBR>
using StageTile = float[2][NS][NBR * 16][kLdk];

template <int NS, int MB, int NBR, bool kPert, class Act>
__device__ __forceinline__ void perturbed_mainloop(f32x4 (&acc)[MB][NS][NBR], StageTile<NS, NBR>& lds,
                                                   const float* __restrict__ th,
                                                   const int64_t (&wrow)[MB], int K, int law, uint2 key,
                                                   uint32_t pair, uint32_t step_lo, float eps,
                                                   const Act& act) {
  constexpr int ROWS = NBR * 16;
  constexpr int F4 = NS * ROWS * (kChunk / 4);
  constexpr int PT = (F4 + kThreads - 1) / kThreads;
  const int lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  const int nch = (K + kChunk - 1) / kChunk;
  float4 pre[PT];

  auto gload = [&](int c) {
#pragma unroll
    for (int i = 0; i < PT; ++i) {
      const int idx = threadIdx.x + i * kThreads;
      const int c4 = idx & 7, n = (idx >> 3) % ROWS, sg = idx / (8 * ROWS);
      const int k = c * kChunk + 4 * c4;
      pre[i] = (idx < F4 && k < K) ? act(sg, n, k) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < PT; ++i) {
      const int idx = threadIdx.x + i * kThreads;
      if (idx < F4) {
        const int c4 = idx & 7, n = (idx >> 3) % ROWS, sg = idx / (8 * ROWS);
        *reinterpret_cast<float4*>(&lds[buf][sg][n][4 * c4]) = pre[i];
      }
    }
  };

  gload(0);
  sstore(0);
  __syncthreads();
  for (int c = 0; c < nch; ++c) {
    if (c + 1 < nch) gload(c + 1);
    const int buf = c & 1;
#pragma unroll
    for (int g = 0; g < kChunk / 16; ++g) {
      const int k = c * kChunk + 16 * g;
      const bool valid = (g == 0) || (k < K);   // the second group of a tail chunk may be empty
      const int kk = (valid ? k : c * kChunk) + 4 * lg;
      float4 w[MB][NS];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const float4 t4 = *reinterpret_cast<const float4*>(th + wrow[mb] + kk);
        if (kPert) {
          const float4 z = probe_quad(law, key, pair, step_lo, static_cast<uint64_t>(wrow[mb] + kk));
          w[mb][0] = fma4(eps, z, t4);
          w[mb][NS - 1] = fma4(-eps, z, t4);
        } else {
          w[mb][0] = t4;
        }
        if (!valid) {
#pragma unroll
          for (int s = 0; s < NS; ++s) w[mb][s] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
#pragma unroll
      for (int nb = 0; nb < NBR; ++nb)
#pragma unroll
        for (int s = 0; s < NS; ++s) {
          const float4 x = *reinterpret_cast<const float4*>(&lds[buf][s][nb * 16 + lr][16 * g + 4 * lg]);
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) acc[mb][s][nb] = mfma_k16(w[mb][s], x, acc[mb][s][nb]);
        }
    }
    if (c + 1 < nch) sstore(buf ^ 1);
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Input projection of layer l >= 2, time-parallel over all B(T-1) rows:
//   gin[slot][row][4u+g] = sum_{k<H} W_l+-[g H + u][k] h_{l-1}[slot][row][k]
// Grid: (4H/64 gate-row tiles, ceil(R/128) row tiles, N * chunk).  One probe
// quad per lane and k group serves both signs and 128 rows per sign.
// ---------------------------------------------------------------------------
template <bool kPert>
__global__ __launch_bounds__(kThreads) void k_proj(FwdArgs a) {
  constexpr int NS = kPert ? 2 : 1;
  constexpr int NBP = 8;  // 16-row blocks per sign
  __shared__ StageTile<NS, NBP> xs;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  const int mtile = blockIdx.x;
  const int64_t r0 = static_cast<int64_t>(blockIdx.y) * NBP * 16;
  const int e = blockIdx.z / a.pcs, jl = blockIdx.z % a.pcs;
  const int H = a.H, in = a.in_l;
  const int64_t R = static_cast<int64_t>(a.T - 1) * a.B;
  const float* th = a.theta + static_cast<int64_t>(e) * a.d;
  const uint2 key = kPert ? stream_key(a.seeds[e], a.step) : make_uint2(0u, 0u);
  const uint32_t pair = static_cast<uint32_t>(a.j0 + jl), step_lo = static_cast<uint32_t>(a.step);
  const int prow = mtile * 64 + wave * 16 + lr;
  const int64_t wrow[1] = {a.off_l + static_cast<int64_t>((prow & 3) * H + (prow >> 2)) * (in + H)};
  const int64_t slot0 = (static_cast<int64_t>(e) * a.PC + jl) * NS;
  const float* hin = a.hseq;

  f32x4 acc[1][NS][NBP];
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int nb = 0; nb < NBP; ++nb) acc[0][s][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto act = [&](int s, int n, int k) {
    const int64_t row = r0 + n;
    return row < R ? *reinterpret_cast<const float4*>(hin + ((slot0 + s) * R + row) * H + k)
                   : make_float4(0.f, 0.f, 0.f, 0.f);
  };
  perturbed_mainloop<NS, 1, NBP, kPert>(acc, xs, th, wrow, in, a.probe, key, pair, step_lo,
        kPert ? eps_of(a, e, kGroupLstm) : 0.0f, act);

  const int p = mtile * 64 + wave * 16 + 4 * lg;
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int nb = 0; nb < NBP; ++nb) {
      const int64_t row = r0 + nb * 16 + lr;
      if (row < R) {
        float* dst = a.gin + ((slot0 + s) * R + row) * (4 * static_cast<int64_t>(H)) + p;
        *reinterpret_cast<float4*>(dst) =
            make_float4(acc[0][s][nb][0], acc[0][s][nb][1], acc[0][s][nb][2], acc[0][s][nb][3]);
      }
    }
}

// ---------------------------------------------------------------------------
// One time step t of the recurrence of one layer, all directions and signs:
//   a = gin_t + h_{t-1} W_lh+-^T;  i,f,o = sigma, g = tanh;
//   c_t = f c_{t-1} + i g;  h_t = o tanh(c_t)          (h_{-1} = c_{-1} = 0)
// Grid: (H/16 unit tiles * batch groups of 16 NB rows, chunk, N).  A block
// owns 16 units (64 gate rows, 16 per wave) for both signs and NB*16 batch
// rows; each lane ends with the four gates of one unit for one row and
// applies the cell update in registers.  The recurrent weights are
// re-perturbed from their probe counters every step.
// ---------------------------------------------------------------------------
template <int NB, bool kPert>
__global__ __launch_bounds__(kThreads) void k_rec_step(FwdArgs a) {
  constexpr int NS = kPert ? 2 : 1;
  __shared__ StageTile<NS, NB> hs;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  const int H = a.H, B = a.B, T = a.T, in = a.in_l, t = a.t;
  const int ntile = H / 16;
  const int utile = blockIdx.x % ntile, b0 = (blockIdx.x / ntile) * NB * 16;
  const int jl = blockIdx.y, e = blockIdx.z;
  const float* th = a.theta + static_cast<int64_t>(e) * a.d;
  const int64_t R = static_cast<int64_t>(T - 1) * B;
  const int64_t slot0 = (static_cast<int64_t>(e) * a.PC + jl) * NS;

  f32x4 acc[1][NS][NB];
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[0][s][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (t > 0) {
    const uint2 key = kPert ? stream_key(a.seeds[e], a.step) : make_uint2(0u, 0u);
    const uint32_t pair = static_cast<uint32_t>(a.j0 + jl), step_lo = static_cast<uint32_t>(a.step);
    const int prow = utile * 64 + wave * 16 + lr;
    const int64_t wrow[1] = {a.off_l + static_cast<int64_t>((prow & 3) * H + (prow >> 2)) * (in + H) + in};
    const float* hprev = a.hseq + static_cast<int64_t>(t - 1) * B * H;
    auto act = [&](int s, int n, int k) {
      const int b = b0 + n;
      return b < B ? *reinterpret_cast<const float4*>(hprev + ((slot0 + s) * R + b) * H + k)
                   : make_float4(0.f, 0.f, 0.f, 0.f);
    };
    perturbed_mainloop<NS, 1, NB, kPert>(acc, hs, th, wrow, H, a.probe, key, pair, step_lo,
        kPert ? eps_of(a, e, kGroupLstm) : 0.0f, act);
  }

  const int unit = utile * 16 + wave * 4 + lg;
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int b = b0 + nb * 16 + lr;
      if (b >= B) continue;
      const int64_t slot = slot0 + s;
      float4 gi;
      if (a.layer == 0) {
        const int v = bytes_of(a, e, jl)[static_cast<int64_t>(b) * T + t];
        gi = *reinterpret_cast<const float4*>(a.U + (slot * kVocab + v) * (4 * static_cast<int64_t>(H)) + 4 * unit);
      } else {
        gi = *reinterpret_cast<const float4*>(
            a.gin + (slot * R + static_cast<int64_t>(t) * B + b) * (4 * static_cast<int64_t>(H)) + 4 * unit);
      }
      const float ai = acc[0][s][nb][0] + gi.x, af = acc[0][s][nb][1] + gi.y;
      const float ag = acc[0][s][nb][2] + gi.z, ao = acc[0][s][nb][3] + gi.w;
      float* cp = a.cst + (slot * B + b) * static_cast<int64_t>(H) + unit;
      const float cprev = t > 0 ? *cp : 0.0f;
      const float c = sigmoid_f(af) * cprev + sigmoid_f(ai) * tanh_f(ag);
      *cp = c;
      a.hseq[(slot * R + static_cast<int64_t>(t) * B + b) * H + unit] = sigmoid_f(ao) * tanh_f(c);
    }
}

// ---------------------------------------------------------------------------
// One time step t, as k_rec_step (same grid, blocks, probes and cell update)
// but with the products of both signs on the fp16 matrix cores from split
// operands: h_{t-1} of both signs is split into its fp16 parts as it is
// staged (32 K per chunk), and each lane forms W+- for its gate row and 8 K
// values of a chunk from two probe quads, splits both signs and runs the
// three passes over the row tiles.  The fp32 products of k_rec_step share
// the vector ALU's datapath with the probe generation; these run beside it.
// Used where the shape rules out the persistent recurrence (H > 512 or
// H % 64 != 0, B > 64) and H % 32 == 0; SOMA_FLAG_PER_STEP_RECURRENCE keeps
// the fp32 k_rec_step.
// ---------------------------------------------------------------------------
constexpr int kStepSw = 32 + 16;   // staged row in halves (96 bytes: an odd multiple of 32)

template <int NB>
__global__ __launch_bounds__(kThreads) void k_rec_step_split(FwdArgs a) {
  constexpr int NS = 2, ROWS = NB * 16;
  constexpr int F4 = NS * ROWS * 8;                     // float4 of h per chunk (both signs)
  constexpr int PT = F4 / kThreads;
  static_assert(PT * kThreads == F4, "a chunk splits evenly over the threads");
  __shared__ __attribute__((aligned(16))) _Float16 hs[2][NS][2][ROWS][kStepSw];   // [buf][sign][hi, lo][row][k]
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  const int H = a.H, B = a.B, T = a.T, in = a.in_l, t = a.t;
  const int ntile = H / 16;
  const int utile = blockIdx.x % ntile, b0 = (blockIdx.x / ntile) * ROWS;
  const int jl = blockIdx.y, e = blockIdx.z;
  const float* th = a.theta + static_cast<int64_t>(e) * a.d;
  const int64_t R = static_cast<int64_t>(T - 1) * B;
  const int64_t slot0 = (static_cast<int64_t>(e) * a.PC + jl) * NS;

  f32x4 acc[NS][NB];
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[s][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (t > 0) {
    const uint2 key = stream_key(a.seeds[e], a.step);
    const uint32_t pair = static_cast<uint32_t>(a.j0 + jl), step_lo = static_cast<uint32_t>(a.step);
    const float eps = eps_of(a, e, kGroupLstm);
    const int prow = utile * 64 + wave * 16 + lr;
    const int64_t wrow = a.off_l + static_cast<int64_t>((prow & 3) * H + (prow >> 2)) * (in + H) + in;
    const float* hprev = a.hseq + static_cast<int64_t>(t - 1) * B * H;
    const int nch = H / 32;
    float4 pre[PT];
    // Thread load i of a chunk: float4 c4 = idx & 7 of row n = (idx >> 3) % ROWS
    // of sign s = idx / (8 ROWS); rows past the batch stage zeros.
    auto gload = [&](int c) {
#pragma unroll
      for (int i = 0; i < PT; ++i) {
        const int idx = threadIdx.x + i * kThreads;
        const int c4 = idx & 7, n = (idx >> 3) % ROWS, s = idx / (8 * ROWS);
        const int b = b0 + n;
        pre[i] = b < B ? *reinterpret_cast<const float4*>(hprev + ((slot0 + s) * R + b) * H + 32 * c + 4 * c4)
                       : make_float4(0.f, 0.f, 0.f, 0.f);
      }
    };
    auto sstore = [&](int buf) {
#pragma unroll
      for (int i = 0; i < PT; ++i) {
        const int idx = threadIdx.x + i * kThreads;
        const int c4 = idx & 7, n = (idx >> 3) % ROWS, s = idx / (8 * ROWS);
        uint2 hi, lo;
        split4(pre[i], hi, lo);
        *reinterpret_cast<uint2*>(&hs[buf][s][0][n][4 * c4]) = hi;
        *reinterpret_cast<uint2*>(&hs[buf][s][1][n][4 * c4]) = lo;
      }
    };
    bool in_range = true;
    gload(0);
    sstore(0);
    __syncthreads();
    for (int c = 0; c < nch; ++c) {
      if (c + 1 < nch) gload(c + 1);
      const int buf = c & 1;
      const int64_t kk = wrow + 32 * c + 8 * lg;
      const float4 t0 = *reinterpret_cast<const float4*>(th + kk);
      const float4 t1 = *reinterpret_cast<const float4*>(th + kk + 4);
      const float4 z0 = probe_quad(a.probe, key, pair, step_lo, static_cast<uint64_t>(kk));
      const float4 z1 = probe_quad(a.probe, key, pair, step_lo, static_cast<uint64_t>(kk + 4));
      uint4 wh[NS], wl[NS];
      const float4 wp0 = fma4(eps, z0, t0), wp1 = fma4(eps, z1, t1), wm0 = fma4(-eps, z0, t0), wm1 = fma4(-eps, z1, t1);
      in_range &= (split_range_ok(wp0) && split_range_ok(wp1)) && (split_range_ok(wm0) && split_range_ok(wm1));
      split8v(wp0, wp1, wh[0], wl[0]);
      split8v(wm0, wm1, wh[1], wl[1]);
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        uint4 bh[NB], bl[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          bh[nb] = *reinterpret_cast<const uint4*>(&hs[buf][s][0][nb * 16 + lr][8 * lg]);
          bl[nb] = *reinterpret_cast<const uint4*>(&hs[buf][s][1][nb * 16 + lr][8 * lg]);
        }
        mfma3_batch<NB>(wh[s], wl[s], bh, bl, acc[s]);
      }
      if (c + 1 < nch) sstore(buf ^ 1);
      __syncthreads();
    }
    report_split_range(a.err, in_range);
  }

  const int unit = utile * 16 + wave * 4 + lg;
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int b = b0 + nb * 16 + lr;
      if (b >= B) continue;
      const int64_t slot = slot0 + s;
      float4 gi;
      if (a.layer == 0) {
        const int v = bytes_of(a, e, jl)[static_cast<int64_t>(b) * T + t];
        gi = *reinterpret_cast<const float4*>(a.U + (slot * kVocab + v) * (4 * static_cast<int64_t>(H)) + 4 * unit);
      } else {
        gi = *reinterpret_cast<const float4*>(
            a.gin + (slot * R + static_cast<int64_t>(t) * B + b) * (4 * static_cast<int64_t>(H)) + 4 * unit);
      }
      float* cp = a.cst + (slot * B + b) * static_cast<int64_t>(H) + unit;
      float c = t > 0 ? *cp : 0.0f, h;
      lstm_cell(acc[s][nb][0] + gi.x, acc[s][nb][1] + gi.y, acc[s][nb][2] + gi.z, acc[s][nb][3] + gi.w, c, h);
      *cp = c;
      a.hseq[(slot * R + static_cast<int64_t>(t) * B + b) * H + unit] = h;
    }
}

// ---------------------------------------------------------------------------
// Head and fused softmax cross entropy over 256 byte values.
//   logits[row][v] = sum_k Whead+-[v][k] h[slot][row][k];
//   ce = log sum_v exp(logits - max) + max - logits[target]
// Grid: (ceil(R/64) row tiles, N * chunk).  Waves own 64 vocabulary rows
// each (four 16-row MFMA blocks); row maxima and sums meet across the four
// lane groups by shuffles and across waves through LDS in a fixed order.
// part[slot][tile] receives the tile's sum of ce in fp64 (deterministic order).
// ---------------------------------------------------------------------------
template <bool kPert>
__global__ __launch_bounds__(kThreads) void k_head_ce(FwdArgs a) {
  constexpr int NS = kPert ? 2 : 1;
  constexpr int NBH = 4;  // 64 rows per sign
  __shared__ StageTile<NS, NBH> xs;
  __shared__ float red[4][NS][NBH * 16];
  __shared__ float tgt[NS][NBH * 16];
  __shared__ float ces[NS][NBH * 16];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  const int H = a.H, B = a.B, T = a.T;
  const int64_t R = static_cast<int64_t>(T - 1) * B;
  const int tile = blockIdx.x;
  const int64_t r0 = static_cast<int64_t>(tile) * NBH * 16;
  const int e = blockIdx.y / a.pcs, jl = blockIdx.y % a.pcs;
  const float* th = a.theta + static_cast<int64_t>(e) * a.d;
  const uint2 key = kPert ? stream_key(a.seeds[e], a.step) : make_uint2(0u, 0u);
  const uint32_t pair = static_cast<uint32_t>(a.j0 + jl), step_lo = static_cast<uint32_t>(a.step);
  const int64_t slot0 = (static_cast<int64_t>(e) * a.PC + jl) * NS;

  f32x4 acc[4][NS][NBH];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int nb = 0; nb < NBH; ++nb) acc[mb][s][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  int64_t wrow[4];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) wrow[mb] = a.off_head + static_cast<int64_t>(wave * 64 + mb * 16 + lr) * H;
  const float* hin = a.hseq;
  auto act = [&](int s, int n, int k) {
    const int64_t row = r0 + n;
    return row < R ? *reinterpret_cast<const float4*>(hin + ((slot0 + s) * R + row) * H + k)
                   : make_float4(0.f, 0.f, 0.f, 0.f);
  };
  perturbed_mainloop<NS, 4, NBH, kPert>(acc, xs, th, wrow, H, a.probe, key, pair, step_lo,
        kPert ? eps_of(a, e, kGroupHead) : 0.0f, act);

  // Row maxima: lane-local over 16 logits, then across the 4 lane groups.
  float mx[NS][NBH];
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int nb = 0; nb < NBH; ++nb) {
      float m = acc[0][s][nb][0];
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r) m = fmaxf(m, acc[mb][s][nb][r]);
      m = fmaxf(m, __shfl_xor(m, 16));
      m = fmaxf(m, __shfl_xor(m, 32));
      mx[s][nb] = m;
    }
  if (lg == 0) {
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int nb = 0; nb < NBH; ++nb) red[wave][s][nb * 16 + lr] = mx[s][nb];
  }
  // target logits: the lane holding v = target writes it
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int nb = 0; nb < NBH; ++nb) {
      const int64_t row = r0 + nb * 16 + lr;
      if (row < R) {
        const int64_t tt = row / B, b = row % B;
        const int y = bytes_of(a, e, jl)[b * T + tt + 1];
        if ((y >> 6) == wave && ((y >> 2) & 3) == lg) {
          const int ymb = (y >> 4) & 3, yr = y & 3;
          float v = 0.0f;
#pragma unroll
          for (int mb = 0; mb < 4; ++mb)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (mb == ymb && r == yr) v = acc[mb][s][nb][r];
          tgt[s][nb * 16 + lr] = v;
        }
      }
    }
  __syncthreads();
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int nb = 0; nb < NBH; ++nb) {
      const int n = nb * 16 + lr;
      mx[s][nb] = fmaxf(fmaxf(red[0][s][n], red[1][s][n]), fmaxf(red[2][s][n], red[3][s][n]));
    }
  float se[NS][NBH];
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int nb = 0; nb < NBH; ++nb) {
      float sum = 0.0f;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r) sum += __expf(acc[mb][s][nb][r] - mx[s][nb]);
      sum += __shfl_xor(sum, 16);
      sum += __shfl_xor(sum, 32);
      se[s][nb] = sum;
    }
  __syncthreads();
  if (lg == 0) {
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int nb = 0; nb < NBH; ++nb) red[wave][s][nb * 16 + lr] = se[s][nb];
  }
  __syncthreads();
  // Every lane holds the row maxima (mx) of its rows; `red` holds the
  // per-wave sums.  Lane group 0 of wave 0 forms ce for the tile's rows.
  if (wave == 0 && lg == 0) {
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int nb = 0; nb < NBH; ++nb) {
        const int n = nb * 16 + lr;
        const int64_t row = r0 + n;
        float ce = 0.0f;
        if (row < R) {
          const float sum = ((red[0][s][n] + red[1][s][n]) + red[2][s][n]) + red[3][s][n];
          ce = __logf(sum) + mx[s][nb] - tgt[s][n];
        }
        ces[s][n] = ce;
      }
  }
  __syncthreads();
  if (threadIdx.x < NS) {
    const int s = threadIdx.x;
    double tot = 0.0;
    for (int n = 0; n < NBH * 16; ++n) tot += static_cast<double>(ces[s][n]);
    a.part[(slot0 + s) * a.row_tiles + tile] = tot;
  }
}

// ---------------------------------------------------------------------------
// Persistent recurrence of one layer (perturbed step only).
//
// A block of NW waves (8, or 12 where persist_waves says so) owns 4 NW units
// (16 NW gate rows) of one (expert, direction, sign): wave w keeps the
// perturbed recurrent weights of gate rows [16 w, +16) IN REGISTERS for the
// whole sequence -- the probes are drawn once per (expert, direction, sign)
// instead of once per time step.  A group of H / (4 NW) co-resident blocks
// carries one (expert, direction, sign) through time: after step t every
// block publishes its slice of h_t and arrives on the group's counter;
// before step t+1 it waits for all the group's arrivals, then streams h_{t-1}
// of its sign (B x H) through a ring of two LDS pieces of 128 (or 64) columns
// of K, splitting it into fp16 parts as it is stored and overlapping the next
// piece's loads with the current piece's MFMAs.  Groups take jobs
// round-robin; the cell state stays in registers.  One block per CU (two or
// three waves per SIMD).
//
// h is exchanged with device-coherent (sc1) stores and loads, so no cache
// writeback or invalidation is needed: a block's stores complete
// (s_waitcnt vmcnt(0)) before its arrival is counted, and readers load h
// only after observing every arrival.
//
// Every wait is bounded: a block that polls longer than spin_limit sets the
// sticky abort flag, and every block that sees the flag leaves, so the grid
// always drains; the update kernel then leaves theta untouched and the
// losses read NaN.
// ---------------------------------------------------------------------------
constexpr int kRecMaxH = 704;          // H <= 704: 176 VGPRs of split fragments per lane (K = H)
constexpr int kCoherent = 16;          // cache policy: device scope (sc1)
constexpr int kZpiece = 256;           // k per cooperatively drawn probe piece

struct PersistArgs {
  FwdArgs a;
  unsigned* bar;         // [groups] arrival counters, zero at launch
  unsigned* err;         // sticky abort flag, zero at the start of the step
  int groups;            // concurrent groups
  int jobs;              // N * directions in this pass * 2 signs
  unsigned spin_limit;   // polls before giving up
};

__device__ __forceinline__ void wait_vmem() {
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): every memory access of this wave has completed
}

__device__ __forceinline__ void group_arrive(unsigned* bar) {
  wait_vmem();
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_fetch_add(bar, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Returns true when the block must abort.
__device__ __forceinline__ bool group_wait(unsigned* bar, unsigned target, unsigned* err,
                                           unsigned spin_limit, unsigned* flag) {
  if (threadIdx.x == 0) {
    unsigned polls = 0, bad = 0;
    for (;;) {
      // Both words are read in one round trip.
      const unsigned arrived = __hip_atomic_load(bar, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const unsigned failed = __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (arrived >= target) break;
      if (failed != 0u) {
        bad = 1;
        break;
      }
      if (++polls > spin_limit) {
        __hip_atomic_fetch_or(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        bad = 1;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    *flag = bad;
  }
  __syncthreads();
  return *flag != 0u;
}

// Buffer resource over [base, base + bytes) (bytes < 2^31); reads past the
// end return zeros and writes past it are dropped.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_of(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes), 0x00020000);
}

// float4 load through a buffer resource (the builtin returns the bits as
// four 32-bit integers).
template <int kAux>
__device__ __forceinline__ float4 buffer_load_f4(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kAux);
  return make_float4(__uint_as_float(v[0]), __uint_as_float(v[1]), __uint_as_float(v[2]), __uint_as_float(v[3]));
}

// float4 load at a per-lane plus a wave-uniform (scalar) offset.
template <int kAux>
__device__ __forceinline__ float4 buffer_load_f4s(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, kAux);
  return make_float4(__uint_as_float(v[0]), __uint_as_float(v[1]), __uint_as_float(v[2]), __uint_as_float(v[3]));
}

// Perturbed weights of NR rows r0 .. r0 + NR - 1 (16 per wave) over columns
// col0 .. col0 + 32 KC of a matrix at canonical offset off_l with row length
// ld, one sign, as split fragments for the fp16 products:  w = theta + seps z
// is formed in fp32 and split.  With kGateRows the rows are a layer's gate
// rows in interleaved order (row 4u + g is gate g of unit u, canonical row
// g H + u); otherwise row r is canonical row r.  Lane (wave, lr, lg) keeps
// row r0 + 16 wave + lr, columns col0 + 32 c + 8 lg .. + 7 as (wh[c],
// wl[c]).  The block draws the probes cooperatively, ZW columns at a time,
// into the LDS scratch zs (NR x (ZW + 8) floats), which is free again on
// return.  The generator is fixed at compile time (kRad: a Rademacher law,
// `law` then telling sparse from dense; else Gaussian): a run-time choice
// between the two costs these register-resident kernels spills.  A weight
// outside the split's range sets the step's abort flag.
template <int KC, bool kGateRows, bool kRad, int ZW = kZpiece, int NR = 128>
__device__ __forceinline__ void resident_weights_split(uint4 (&wh)[KC], uint4 (&wl)[KC], float* zs, const float* th,
                                                       int64_t off_l, int ld, int col0, int H, int r0, int law,
                                                       uint2 key, uint32_t pair, uint32_t step_lo, float seps,
                                                       unsigned* err) {
  static_assert(ZW % 32 == 0 && ZW <= kZpiece, "probe pieces of whole chunks");
  constexpr int kPiece = ZW / 32;        // chunks per probe piece
  constexpr int ZLD = ZW + 8;            // scratch row in floats (an odd multiple of 32 bytes)
  bool in_range = true;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  auto canon = [&](int r) { return kGateRows ? (r & 3) * H + (r >> 2) : r; };
  const int prow = r0 + wave * 16 + lr;
  const int64_t wrow = off_l + static_cast<int64_t>(canon(prow)) * ld + col0;
#pragma unroll
  for (int piece = 0; piece < (KC + kPiece - 1) / kPiece; ++piece) {
    const int kc0 = piece * kPiece;
    const int nc = (KC - kc0 < kPiece ? KC - kc0 : kPiece);
    __syncthreads();
    for (int q = threadIdx.x; q < NR * nc * 8; q += blockDim.x) {
      const int m = q / (nc * 8), k4 = q % (nc * 8);
      const int pr = r0 + m;
      const uint64_t kk = static_cast<uint64_t>(off_l + static_cast<int64_t>(canon(pr)) * ld + col0 + 32 * kc0 + 4 * k4);
      *reinterpret_cast<float4*>(&zs[m * ZLD + 4 * k4]) =
          kRad ? rademacher_quad(key, pair, step_lo, kk, law == kProbeRademacher) : gauss_quad(key, pair, step_lo, kk >> 2);
    }
    __syncthreads();
#pragma unroll
    for (int c2 = 0; c2 < kPiece; ++c2) {
      const int c = kc0 + c2;
      if (c < KC) {
        const float* zr = &zs[(wave * 16 + lr) * ZLD + 32 * c2 + 8 * lg];
        const float* tr = th + wrow + 32 * c + 8 * lg;
        const float4 w0 = fma4(seps, *reinterpret_cast<const float4*>(zr), *reinterpret_cast<const float4*>(tr));
        const float4 w1 = fma4(seps, *reinterpret_cast<const float4*>(zr + 4), *reinterpret_cast<const float4*>(tr + 4));
        in_range = in_range && split_range_ok(w0) && split_range_ok(w1);
        split8v(w0, w1, wh[c], wl[c]);
      }
    }
  }
  report_split_range(err, in_range);
  __syncthreads();
}

// Waves per block of the persistent recurrence for hidden width H and batch
// B: 12 (192 gate rows, 48 units) where H is 192 or 384 and B <= 32, so that
// a group of H/48 blocks fits one XCD in groups of a multiple of 8 across all
// 256 compute units (at H = 384: 32 groups of 8 blocks instead of 16 groups
// of 12 blocks, a quarter of the chip idle); else 8 (128 gate rows, 32
// units).  With 12 waves (three per SIMD, 168 registers each) four row tiles
// do not fit.
__host__ __device__ constexpr int persist_waves(int H, int B) {
  return (H == 192 || H == 384) && B <= 32 ? 12 : 8;
}

// kPre: the recurrent weights come pre-formed (a.wpre) and a pass may run
// one sign per direction (a.ns == 1); a separate instantiation, so that the
// kernels that form their weights from the probes keep their registers.
template <int NB, int NCH, bool kRad, int NW, bool kPre = false>
__global__ __launch_bounds__(64 * NW, 1) void k_rec_persist(PersistArgs p) {
  constexpr int NU = 4 * NW;                            // units per block (16 NW gate rows, 16 per wave)
  constexpr int KC = 2 * NCH;                           // 32-wide k chunks: H = 64 NCH
  // Staging pieces of K, 128 wide where H allows, else 64: the first piece,
  // whose loads nothing hides, stays short, while a piece's products still
  // outlast the loads of the next (measured at H = 512: 256-wide pieces cost
  // 7% more time per step, 64-wide ones 8%).
  constexpr int KWQ = (64 * NCH) % 128 == 0 ? 128 : 64;   // k per piece
  constexpr int NQ = 64 * NCH / KWQ;
  constexpr int QC = KWQ / 32;                          // k chunks per piece
  constexpr int ROWS = NB * 16;
  constexpr int SW = KWQ + 16;                          // ring row in halves (an odd multiple of 32 bytes)
  constexpr int CW4 = KWQ / 4;                          // float4 per row of a piece: 16 or 32
  constexpr int RPW = 64 / CW4;                         // rows per wave load
  constexpr int WL = ROWS / RPW;                        // wave loads per piece
  constexpr int PT = (WL + NW - 1) / NW;                // of them per wave
  constexpr bool kAllWaves = WL % NW == 0;              // else the waves past the rows stage nothing
  constexpr int RING_BYTES = 2 * 2 * ROWS * SW * 2;     // [buffer][hi, lo][ROWS][SW] halves
  constexpr int ZW = NW > 8 ? 128 : kZpiece;            // probe piece: 16 NW rows x (ZW + 8) floats
  constexpr int ZS_BYTES = 16 * NW * (ZW + 8) * 4;
  constexpr int LDS_BYTES = RING_BYTES > ZS_BYTES ? RING_BYTES : ZS_BYTES;
  constexpr int HTLD = NU + 4;                          // LDS row of the transposed h_t tile
  static_assert(WL * RPW == ROWS, "a piece's rows split into whole wave loads");
  // Registers per lane: weights 8 KC, accumulators and gate inputs 8 NB, the
  // B fragments of a chunk 8 NB, staging 4 PT, about 40 more.  Where that
  // exceeds the 256 that two waves per SIMD leave each wave (H >= 576 with
  // four row tiles), the fragments are read one row tile at a time
  // (measured on the monolith workload: its recurrence 210 -> 192 ms per
  // step; with three waves per SIMD at H = 384 the serialised passes cost
  // more than the spills they avoid).
  constexpr bool kLeanFrag = NW == 8 && 8 * KC + 16 * NB + 4 * PT + 40 > 256;
  // a ring of two staged pieces of h_{t-1}, split into fp16 parts; the probe
  // piece at job start
  __shared__ __attribute__((aligned(16))) unsigned char lds[LDS_BYTES];
  __shared__ __attribute__((aligned(16))) float ht[ROWS * HTLD];   // h_t of the block's units, transposed for stores
  _Float16* ring = reinterpret_cast<_Float16*>(lds);    // buffer b: hi at ring + 2 b ROWS SW, lo one part later
  __shared__ unsigned abort_flag;
  const FwdArgs& a = p.a;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform (scalar) from here on
  const int lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  const int H = a.H, B = a.B, T = a.T, in = a.in_l;
  const int UT = H / NU;                                // blocks per group
  const int g = blockIdx.x % p.groups;
  const int utile = blockIdx.x / p.groups;              // < UT: the grid is groups * UT blocks
  const int64_t R = static_cast<int64_t>(T - 1) * B;
  const int64_t H4 = 4 * static_cast<int64_t>(H);
  const int unit = utile * NU + wave * 4 + lg;          // output unit of this lane
  const uint32_t slot_bytes = static_cast<uint32_t>(R * H * sizeof(float));   // < 2^31 (host check)
  unsigned* bar = p.bar + g;
  unsigned done = 0;                                    // steps this block has published

  const bool one_sign = kPre && a.ns == 1;
  for (int job = g; job < p.jobs; job += p.groups) {
    const int sg = one_sign ? 0 : job & 1, pj = one_sign ? job : job >> 1;
    const int e = pj / a.pcs, jl = pj % a.pcs;
    const float* th = a.theta + static_cast<int64_t>(e) * a.d;
    const uint2 key = kPre ? make_uint2(0u, 0u) : stream_key(a.seeds[e], a.step);   // no seeds for pre-formed weights
    const uint32_t pair = static_cast<uint32_t>(a.j0 + jl), step_lo = static_cast<uint32_t>(a.step);
    const int64_t slot = (static_cast<int64_t>(e) * a.PC + jl) * (one_sign ? 1 : 2) + sg;
    const float seps = kPre ? 0.0f : (sg == 0 ? eps_of(a, e, kGroupLstm) : -eps_of(a, e, kGroupLstm));
    const __amdgpu_buffer_rsrc_t hbuf = buffer_of(a.hseq + slot * R * H, slot_bytes);
    // Gate inputs of layer 1 (folded, per byte value) or of a later layer.
    const __amdgpu_buffer_rsrc_t gbuf =
        a.layer == 0 ? buffer_of(a.U + slot * kVocab * H4, static_cast<uint32_t>(kVocab * H4 * sizeof(float)))
                     : buffer_of(a.gin + slot * R * H4, static_cast<uint32_t>(R * H4 * sizeof(float)));
    const __amdgpu_buffer_rsrc_t bbuf =
        buffer_of(bytes_of(a, e, jl), static_cast<uint32_t>(B * T));

    // Perturbed recurrent weights of this lane, drawn once for the sequence
    // and held as split fragments.
    uint4 wh[KC], wl[KC];
    if constexpr (kPre) {
      // Rows of the pre-formed matrix, stored split (a row's H hi parts,
      // then its H lo parts): this lane's gate row, 8 consecutive k per
      // 32-wide chunk (the range was checked where the weights were formed).
      const _Float16* wr = reinterpret_cast<const _Float16*>(a.wpre + slot * a.wpre_slot) +
                           static_cast<int64_t>(utile * 16 * NW + wave * 16 + lr) * 2 * H + 8 * lg;
#pragma unroll
      for (int c = 0; c < KC; ++c) {
        wh[c] = *reinterpret_cast<const uint4*>(wr + 32 * c);
        wl[c] = *reinterpret_cast<const uint4*>(wr + H + 32 * c);
      }
    } else {
      resident_weights_split<KC, true, kRad, ZW, 16 * NW>(wh, wl, reinterpret_cast<float*>(lds), th, a.off_l, in + H,
                                                          in, H, utile * 16 * NW, a.probe, key, pair, step_lo, seps,
                                                          p.err);
    }
    // Rows past the batch compute on whatever follows in the same buffers
    // (finite inputs and h of later rows, possibly being rewritten, or zeros
    // past a buffer's end): a column of the product depends only on the same
    // column of h, so no stored output depends on them, and they are never
    // stored.  So the step has no divergent branches: its loads issue
    // together, and the stores of h, all at its end, are not waited on
    // before the arrival.
    // All addresses of the step loop are 32-bit offsets into the buffers
    // above (a few VGPRs instead of one 64-bit pointer per row).
    // Lane row lr of row tile nb is batch row 16 nb + lr: a per-lane offset
    // plus a scalar one.  Rows past the batch (B < 16 NB) read the data that
    // follows in the same buffer, or zeros past its end.
    float cs[NB];
    int vnext[NB];
    const uint32_t byte_lane = static_cast<uint32_t>(lr * T);
    const uint32_t gi_lane = static_cast<uint32_t>((lr * 4 * H + 4 * unit) * 4);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      cs[nb] = 0.0f;
      vnext[nb] = a.layer == 0
                      ? __builtin_amdgcn_raw_buffer_load_b8(bbuf, byte_lane, static_cast<uint32_t>(nb * 16 * T), 0)
                      : 0;
    }

    // Gate inputs of step tt; they seed the accumulators, which the
    // products then add to.  Layer 1 reads its folded inputs by byte value
    // (the byte of step tt + 1 is fetched along).  The inputs of step t + 1
    // are requested at the start of step t's last piece of products (the
    // staging registers are free by then), so their HBM latency is hidden
    // by the products and the cell updates; by the arrival only the stores
    // of h_t are outstanding, and the barrier polls, which return in order
    // behind earlier loads of the same wave, are not held up.
    float4 gi[NB];
    auto load_inputs = [&](int tt) {
      if (a.layer == 0) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          gi[nb] = buffer_load_f4<0>(gbuf, static_cast<uint32_t>((vnext[nb] * 4 * H + 4 * unit) * 4));
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          vnext[nb] = __builtin_amdgcn_raw_buffer_load_b8(bbuf, byte_lane,
                                                          static_cast<uint32_t>(nb * 16 * T + tt + 1), 0);
      } else {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          gi[nb] = buffer_load_f4s<0>(gbuf, gi_lane, static_cast<uint32_t>((tt * B + nb * 16) * 4 * H * 4));
      }
    };
    load_inputs(0);

    for (int t = 0; t + 1 < T; ++t) {
      f32x4 acc[NB];
      auto seed = [&]() {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{gi[nb].x, gi[nb].y, gi[nb].z, gi[nb].w};
      };
      // Cell update of row tile nb: c_t = f c_{t-1} + i g, h_t = o tanh(c_t),
      // written to the transposed tile that is published below.
      auto cell = [&](int nb) {
        float h;
        lstm_cell(acc[nb][0], acc[nb][1], acc[nb][2], acc[nb][3], cs[nb], h);
        ht[(nb * 16 + lr) * HTLD + wave * 4 + lg] = h;
      };

      if (t == 0) {
        wait_vmem();
        seed();
        if (t + 2 < T) load_inputs(t + 1);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) cell(nb);
      } else {
        if (group_wait(bar, static_cast<unsigned>(UT) * done, p.err, p.spin_limit, &abort_flag)) return;
        const int row0 = (t - 1) * B;                    // rows of h_{t-1} in the slot
        // Wave load i of a piece covers rows (wave + NW i) RPW + lane / CW4,
        // float4 lane % CW4 of the piece: a per-lane part and a scalar part.
        // Rows past the batch (B < 64) read whatever follows h_{t-1} (zeros
        // past the slot); their results are never stored.  Piece qq is staged
        // into ring buffer qq & 1: the products of piece qq - 1, the buffer's
        // previous contents, were finished before the block barrier that
        // ends their iteration.
        const int lrow = lane / CW4, lc4 = lane % CW4;
        const uint32_t lane_off = static_cast<uint32_t>((lrow * H + 4 * lc4) * 4);
        float4 pre[PT];
        auto gload = [&](int qq) {
#pragma unroll
          for (int i = 0; i < PT; ++i) {
            const int n0 = (wave + NW * i) * RPW;
            if (kAllWaves || n0 < ROWS) {                // wave-uniform
              const uint32_t soff = static_cast<uint32_t>(((row0 + n0) * H + qq * KWQ) * 4);
              typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
              const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(hbuf, lane_off, soff, kCoherent);
              pre[i] = make_float4(__uint_as_float(v[0]), __uint_as_float(v[1]), __uint_as_float(v[2]),
                                   __uint_as_float(v[3]));
            }
          }
        };
        // h_{t-1} is split into its fp16 parts as it is staged.
        auto sstore = [&](int qq) {
          _Float16* hi_part = ring + (2 * (qq & 1)) * ROWS * SW;
#pragma unroll
          for (int i = 0; i < PT; ++i) {
            if (!kAllWaves && (wave + NW * i) * RPW >= ROWS) continue;   // wave-uniform
            const int n = (wave + NW * i) * RPW + lrow;
            uint2 hi, lo;
            split4(pre[i], hi, lo);
            *reinterpret_cast<uint2*>(hi_part + n * SW + 4 * lc4) = hi;
            *reinterpret_cast<uint2*>(hi_part + ROWS * SW + n * SW + 4 * lc4) = lo;
          }
        };
        // Fragment (nb, chunk pq of piece qq) of this lane sits at a
        // compile-time offset from one per-lane base (within the 16-bit LDS
        // offset field).
        const _Float16* blane = ring + lr * SW + 8 * lg;
        auto mfma_chunk = [&](int qq, int pq) {
          const _Float16* bhi = blane + (2 * (qq & 1)) * ROWS * SW;
          if constexpr (kLeanFrag) {
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
              uint4 bh[1] = {*reinterpret_cast<const uint4*>(bhi + nb * 16 * SW + 32 * pq)};
              uint4 bl[1] = {*reinterpret_cast<const uint4*>(bhi + ROWS * SW + nb * 16 * SW + 32 * pq)};
              f32x4 a1[1] = {acc[nb]};
              mfma3_batch<1>(wh[qq * QC + pq], wl[qq * QC + pq], bh, bl, a1);
              acc[nb] = a1[0];
            }
          } else {
            uint4 bh[NB], bl[NB];
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
              bh[nb] = *reinterpret_cast<const uint4*>(bhi + nb * 16 * SW + 32 * pq);
              bl[nb] = *reinterpret_cast<const uint4*>(bhi + ROWS * SW + nb * 16 * SW + 32 * pq);
            }
            mfma3_batch<NB>(wh[qq * QC + pq], wl[qq * QC + pq], bh, bl, acc);
          }
        };
        gload(0);
        sstore(0);                                       // its wait covers the inputs too
        seed();
        __syncthreads();
#pragma unroll
        for (int qq = 0; qq < NQ; ++qq) {
          if (qq + 1 < NQ) {
            gload(qq + 1);
#pragma unroll
            for (int pq = 0; pq < QC; ++pq) mfma_chunk(qq, pq);
            sstore(qq + 1);
            __syncthreads();
          } else {
            if (t + 2 < T) load_inputs(t + 1);
#pragma unroll
            for (int pq = 0; pq < QC; ++pq) mfma_chunk(qq, pq);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) cell(nb);
          }
        }
      }

      // Publish h_t: the block's NU units of one row are 128 or 192
      // contiguous bytes; transposed through LDS (cell() wrote this lane's
      // words), each thread stores a float4, so the block writes whole lines
      // instead of scattered words.
      __syncthreads();
      if (threadIdx.x < ROWS * (NU / 4)) {
        const int n = threadIdx.x / (NU / 4), c4 = threadIdx.x % (NU / 4);
        if (n < B) {
          typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
          const float4 v = *reinterpret_cast<const float4*>(&ht[n * HTLD + 4 * c4]);
          __builtin_amdgcn_raw_buffer_store_b128(
              __builtin_bit_cast(u32x4, v), hbuf,
              static_cast<uint32_t>(((t * B + n) * H + utile * NU + 4 * c4) * 4), 0, kCoherent);
        }
      }
      // Every wave is done reading hs (its last piece) and ht before the
      // group moves on: group_arrive's barrier orders the next step's staging.
      group_arrive(bar);
      ++done;
    }
  }
}

// ---------------------------------------------------------------------------
// Persistent recurrence with a pipelined split exchange (k_rec_xchg): the
// per-step arithmetic of k_rec_persist -- G_t = G_in,t + h_{t-1} W_h+-^T on
// the fp16 matrix cores from split operands, the cell update in the lane
// that holds a unit's four gates -- organised so that the exchange of h
// between the blocks of a group overlaps the products.
//
//  * The batch's row tiles (16 sequences each) are independent recurrences
//    that share the block's resident weights.  A block runs sub-steps
//    s = (t, k) in the order t, then tile k: the products of tile k at step
//    t need only tile k's h_{t-1}, published NB sub-steps earlier, so its
//    exchange is hidden behind the products of the other tiles (NB >= 4).
//  * Each block publishes its 32 units of h_t of a tile (one 32-wide K
//    chunk) already split into fp16 hi and lo parts, in one of two layouts
//    of the chunk's 2 KiB.  Fragment order (H <= 512): per part (hi, lo) 64
//    lanes x 8 halves, lane (lr, lg) holding row lr, columns 8 lg .. + 7,
//    read by the products as they are; the block transposes h_t through
//    LDS (one more block barrier) and two waves store whole lines.  Words
//    (H >= 640): per wave and row one 16-byte word, the four hi parts then
//    the four lo parts, word (w, r) at index 64 (w & 1) + 16 (w >> 1) + r,
//    stored straight from the lanes of the cell update (a wave holds 4 units
//    of each row; three lane swaps bring them together); lane (lr, lg) reads
//    the words at indices lane and 64 + lane and takes its fragments from
//    them by register moves.  Either way every 128-byte line is written by
//    one wave: halves of one word stored by two waves (device coherent) now
//    and then left a half two steps old.  A group keeps two steps per tile
//    (parity t mod 2) in L2.  h_t is also written to the layer's hseq rows
//    for the kernels that read the whole sequence: in fp32, or (split_out:
//    fragment order, B = 64, where the next layer's projection is
//    k_proj_dma) as the same split words, in 1 KiB blocks [16-row tile][hi,
//    lo][32-wide k chunk], word 16 lg + lr holding row lr, k 8 lg .. + 7.
//  * The tile's h_{t-1} reaches LDS by DMA (buffer_load_dwordx4 ... lds):
//    each 1 KiB block lands unchanged -- no staging registers, vector
//    instructions or LDS stores.  The DMA of sub-step s + 2 is issued after
//    a block barrier of sub-step s, into the LDS buffer the products of
//    sub-step s have released (two buffers).
//  * Arrival is a per-(tile, block) flag word holding the steps published.
//    A sub-step's stores are acknowledged during the next sub-step's
//    products (one vmcnt(0) per sub-step, after the products: loads and
//    stores share the counter and may complete out of order, so only a full
//    wait is sound), and the flag is raised right behind the barrier that
//    follows; the flags needed for the DMA of sub-step s + 2 (raised a
//    sub-step earlier) are read with one load issued halfway through the
//    products of sub-step s and checked after them.
//  * The gate inputs of a tile's next step go out as early as the wait
//    allows: at layer 1 (rows of the folded table gathered by byte value,
//    often cache misses) right after the wait, for the next sub-step's
//    tile; at deeper layers (a stream of the time-parallel gate inputs)
//    right after the cell update, which measured faster there.
//
// Every wait is bounded: a wave that polls longer than the spin limit, or
// that sees the step's abort flag, sets the flag and stops waiting; every
// wave then runs to the end without waiting (on stale data), so the grid
// drains, and the losses read NaN.  A block of 8 waves owns 128 gate rows
// (32 units); a group of H / 32 blocks sits on one XCD; one block per
// compute unit, claimed at start from the compute unit it runs on.
//
// The LDS DMA is issued through inline assembly: the compiler assumes that a
// pending LDS DMA may alias every later LDS read and would wait for it
// before each fragment read.  Its completion is covered by the sub-step's
// vmcnt(0) and the block barrier that follows.
// ---------------------------------------------------------------------------
constexpr int kXchgMaxGroups = 256;    // groups of one launch (flags in the workspace)
constexpr int kXchgFlagWords = 256;    // flag words per group: [tile][block], H / 32 <= 64 blocks
constexpr int kXchgCuSlots = 8 * 64;   // blocks-per-compute-unit counters: (XCD, shader engine, CU)
constexpr int kXchgMaxPerCu = 4;
constexpr int kXchgTiles = 4;          // row tiles the pipeline needs: B > 48
constexpr unsigned kAbortPlace = 4u;   // a block found no (group, tile) to claim

struct XchgArgs {
  FwdArgs a;
  _Float16* xh;          // [groups][2][NB][H/32][wave & 1][wave >> 1][16 rows][4 hi + 4 lo] published h, split
  unsigned* flag;        // [groups][kXchgFlagWords] steps published per (tile, block), over all jobs
  unsigned* cu_count;    // [kXchgCuSlots] blocks started per compute unit (zero at launch)
  unsigned* rank_count;  // [8][kXchgMaxPerCu] blocks claimed per (XCD, rank on the CU) (zero at launch)
  unsigned* err;         // sticky abort flag
  int groups;            // 8 * groups per XCD
  int cus_per_xcd;       // compute units per XCD
  int per_cu;            // blocks per compute unit of the launch
  int jobs;              // N * directions in this pass * 2 signs
  unsigned spin_limit;   // polls per wait before giving up
  int split_out;         // store the layer's h to hseq split, in fragment-order blocks (for k_proj_dma)
};

typedef int i32x4 __attribute__((ext_vector_type(4)));

// Buffer descriptor over [base, base + bytes) as four scalar words.
__device__ __forceinline__ i32x4 buffer_words(const void* base, uint32_t bytes) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  return i32x4{static_cast<int>(static_cast<uint32_t>(b)), static_cast<int>(static_cast<uint32_t>(b >> 32)),
               static_cast<int>(bytes), 0x00020000};
}

// LDS byte address of a __shared__ location.
__device__ __forceinline__ uint32_t lds_address(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) void*)(p)));
}

// 16 bytes per lane from buffer offset voff + soff (device-coherent) into LDS
// at lds + 16 lane.
__device__ __forceinline__ void dma16(i32x4 rsrc, uint32_t voff, uint32_t soff, uint32_t lds) {
  asm volatile("buffer_load_dwordx4 %0, %1, %2 offen sc1 lds" : : "v"(voff), "s"(rsrc), "s"(soff), "{m0}"(lds)
               : "memory");
}

// kL1: the layer reads its inputs from the folded table by byte value (layer
// 1) rather than from the time-parallel gate inputs; a template parameter so
// that each instance loads its inputs on one path (the compiler would
// otherwise merge the two paths' pending loads and wait for all of them).
template <int NCH, bool kRad, bool kL1>
__global__ __launch_bounds__(512) void k_rec_xchg(XchgArgs p) {
  constexpr int NW = 8;                                 // waves: 128 gate rows, 32 units (one K chunk of h)
  constexpr int NU = 4 * NW;
  constexpr int NB = kXchgTiles;                        // row tiles of 16 sequences
  constexpr int KC = 2 * NCH;                           // 32-wide k chunks: H = 64 NCH
  constexpr int FRAG = 512;                             // halves per 1 KiB block (half a chunk of a tile)
  constexpr int TBUF = KC * 2 * FRAG;                   // halves of one tile's h in LDS
  constexpr int XTILE = KC * 2 * FRAG;                  // halves per published (step, tile)
  constexpr int XSLOT = 2 * NB * XTILE;                 // halves per group: parity x tile
  constexpr int ZW = 128;                               // probe piece: 128 rows x (ZW + 8) floats
  constexpr int ZS_BYTES = 16 * NW * (ZW + 8) * 4;
  constexpr int RING_BYTES = 2 * TBUF * 2;
  constexpr int LDS_BYTES = RING_BYTES > ZS_BYTES ? RING_BYTES : ZS_BYTES;
  // Layout of the published h: 16-byte words per (wave, row) at H >= 640,
  // published straight from the cell lanes (no LDS transpose, no second
  // block barrier; measured 12% faster at H = 704, where the compiler also
  // spills fewer registers: 13 against 25); else the MFMA fragment order,
  // transposed through LDS, whose fragments need no register moves between
  // the LDS reads and the products (faster at H = 512).
  constexpr bool kWords = NCH >= 10;
  constexpr int NBLK = 2 * KC;                          // 1 KiB blocks per tile: (chunk, half)
  constexpr int BPW = (NBLK + NW - 1) / NW;             // of them per wave (the last ones may be short)
  __shared__ __attribute__((aligned(16))) unsigned char lds[LDS_BYTES];
  constexpr int HTLD = NU + 4;                          // LDS row of the h_t tile (float4-aligned)
  __shared__ __attribute__((aligned(16))) float ht[kWords ? 4 : 16 * HTLD];
  __shared__ int role[2];
  _Float16* ring = reinterpret_cast<_Float16*>(lds);
  const FwdArgs& a = p.a;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  const int H = a.H, B = a.B, T = a.T, in = a.in_l;
  const int UT = H / NU;                                // blocks per group

  // Claim (group, unit tile): rank r = how many blocks started on this
  // compute unit before this one, i = how many blocks of rank r on this XCD
  // claimed before; position r * cus_per_xcd + i of the XCD's per_cu *
  // cus_per_xcd blocks, UT consecutive positions per group, positions past
  // the XCD's whole groups idle.
  if (threadIdx.x == 0) {
    const unsigned hw = __builtin_amdgcn_s_getreg((31 << 11) | 4);         // HW_ID
    const unsigned xcc = __builtin_amdgcn_s_getreg((31 << 11) | 20) & 15;  // XCC_ID
    const unsigned cu = ((hw >> 13) & 3) * 16 + ((hw >> 8) & 15);          // shader engine, compute unit
    int grp = -2, tile = 0;                             // -2: unplaced (an error), -1: idle
    if (xcc < 8) {
      const unsigned r = __hip_atomic_fetch_add(&p.cu_count[xcc * 64 + cu], 1u, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
      if (r < static_cast<unsigned>(p.per_cu)) {
        const unsigned i = __hip_atomic_fetch_add(&p.rank_count[xcc * kXchgMaxPerCu + r], 1u, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
        if (i < static_cast<unsigned>(p.cus_per_xcd)) {
          const int pos = static_cast<int>(r) * p.cus_per_xcd + static_cast<int>(i);
          grp = pos < (p.groups / 8) * UT ? (pos / UT) * 8 + static_cast<int>(xcc) : -1;
          tile = pos % UT;
        }
      }
    }
    if (grp == -2) __hip_atomic_fetch_or(p.err, kAbortPlace, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    role[0] = grp;
    role[1] = tile;
  }
  __syncthreads();
  const int grp = role[0], utile = role[1];
  if (grp < 0) return;
  unsigned* const flags = p.flag + grp * kXchgFlagWords;   // [tile][block]
  const uint32_t xbytes = static_cast<uint32_t>(p.groups) * XSLOT * 2u;
  const i32x4 xrs = buffer_words(p.xh, xbytes);            // the same buffer for the DMA (scalar words)
  const __amdgpu_buffer_rsrc_t xbuf = buffer_of(p.xh, xbytes);
  const int unit = utile * NU + wave * 4 + lg;          // output unit of this lane
  const int64_t R = static_cast<int64_t>(T - 1) * B;
  const int64_t H4 = 4 * static_cast<int64_t>(H);
  const uint32_t slot_bytes = static_cast<uint32_t>(R * H * sizeof(float));   // < 2^31 (host check)
  const int S = (T - 1) * NB;                           // sub-steps of a job
  bool failed = false;                                  // this wave stopped waiting (abort)

  // Poll until every block of the group has published `target` steps of
  // tile k (flag words [k][0 .. UT)), or give up.  Every wave polls for
  // itself; after an abort nothing waits any more.  One load per poll: lane
  // 63 reads the abort flag, the others their flag word, so no load of the
  // loop is left outstanding when it exits (the compiler would otherwise
  // wait for all memory accesses before the register is reused).
  auto ready = [&](unsigned target, unsigned v) { return __builtin_amdgcn_ballot_w64(lane < UT && v < target) == 0; };
  auto wait_flags = [&](int k, unsigned target) {
    unsigned polls = 0;
    const unsigned* addr = lane == 63 ? p.err : flags + k * 64 + lane;
    while (!failed) {
      const unsigned v = __hip_atomic_load(addr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const unsigned f = __builtin_amdgcn_readlane(v, 63);
      if (ready(target, v)) break;
      if (f != 0u || ++polls > p.spin_limit) {
        if (lane == 0) __hip_atomic_fetch_or(p.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        failed = true;
      } else {
        __builtin_amdgcn_s_sleep(1);
      }
    }
  };

  unsigned base = 0;                                    // steps of every tile published in earlier jobs
  for (int job = grp; job < p.jobs; job += p.groups, base += static_cast<unsigned>(T - 1)) {
    const int sg = job & 1, pj = job >> 1;
    const int e = pj / a.pcs, jl = pj % a.pcs;
    const float* th = a.theta + static_cast<int64_t>(e) * a.d;
    const uint2 key = stream_key(a.seeds[e], a.step);
    const uint32_t pair = static_cast<uint32_t>(a.j0 + jl), step_lo = static_cast<uint32_t>(a.step);
    const int64_t slot = (static_cast<int64_t>(e) * a.PC + jl) * 2 + sg;
    const float seps = sg == 0 ? eps_of(a, e, kGroupLstm) : -eps_of(a, e, kGroupLstm);
    const __amdgpu_buffer_rsrc_t hbuf = buffer_of(a.hseq + slot * R * H, slot_bytes);
    const __amdgpu_buffer_rsrc_t gbuf =
        kL1 ? buffer_of(a.U + slot * kVocab * H4, static_cast<uint32_t>(kVocab * H4 * sizeof(float)))
                     : buffer_of(a.gin + slot * R * H4, static_cast<uint32_t>(R * H4 * sizeof(float)));
    const __amdgpu_buffer_rsrc_t bbuf = buffer_of(bytes_of(a, e, jl), static_cast<uint32_t>(B * T));

    // The ring slots this job writes were read in the previous job: every
    // block must have finished it (its last publication of every tile).
    if (base > 0) {
      for (int k = 0; k < NB; ++k) wait_flags(k, base);
    }
    // Perturbed recurrent weights of this lane's gate row, split, for the
    // whole sequence (the probe scratch overlays the LDS ring; the barriers
    // inside order it after the previous job's last fragment reads).
    uint4 wh[KC], wl[KC];
    resident_weights_split<KC, true, kRad, ZW, 16 * NW>(wh, wl, reinterpret_cast<float*>(lds), th, a.off_l, in + H,
                                                        in, H, utile * 16 * NW, a.probe, key, pair, step_lo, seps,
                                                        p.err);
    float cs[NB];
    int vb[NB];                                         // layer 1: byte of the next step of each tile
    float4 gi[NB];                                      // gate inputs of each tile's next step
    const uint32_t byte_lane = static_cast<uint32_t>(lr * T);
    const uint32_t gi_lane = static_cast<uint32_t>((lr * 4 * H + 4 * unit) * 4);
    // Gate inputs of (step tt, tile k) into gi[k]; layer 1 reads its folded
    // inputs by byte value and fetches the byte of step tt + 1 along.
    auto load_inputs = [&](int tt, int k) {
      if constexpr (kL1) {
        gi[k] = buffer_load_f4<0>(gbuf, static_cast<uint32_t>((vb[k] * 4 * H + 4 * unit) * 4));
        vb[k] = __builtin_amdgcn_raw_buffer_load_b8(bbuf, byte_lane, static_cast<uint32_t>(k * 16 * T + tt + 1), 0);
      } else {
        gi[k] = buffer_load_f4s<0>(gbuf, gi_lane, static_cast<uint32_t>((tt * B + k * 16) * 4 * H * 4));
      }
    };
#pragma unroll
    for (int k = 0; k < NB; ++k) {
      cs[k] = 0.0f;
      vb[k] = kL1 ? __builtin_amdgcn_raw_buffer_load_b8(bbuf, byte_lane, static_cast<uint32_t>(k * 16 * T), 0)
                           : 0;
    }
    if constexpr (kL1) {
      load_inputs(0, 0);                                // the others go out one sub-step ahead
    } else {
#pragma unroll
      for (int k = 0; k < NB; ++k) load_inputs(0, k);
    }

    // Sub-step s = (t, k) reads tile k's h_{t-1} (published by every block
    // at sub-step s - NB) from LDS buffer s & 1, filled by DMA issued in
    // sub-step s - 2.
    auto issue = [&](int s) {
      const int t = s / NB, k = s % NB;
      const uint32_t src = static_cast<uint32_t>((grp * XSLOT + (((t - 1) & 1) * NB + k) * XTILE) * 2);
      const uint32_t dst = lds_address(ring + (s & 1) * TBUF);
#pragma unroll
      for (int i = 0; i < BPW; ++i) {
        const int b = wave + NW * i;                    // chunk b / 2, half b % 2
        if (NBLK % NW == 0 || b < NBLK)                 // wave-uniform
          dma16(xrs, static_cast<uint32_t>(lane * 16), src + static_cast<uint32_t>(b * FRAG * 2),
                dst + static_cast<uint32_t>(b * FRAG * 2));
      }
    };
    for (int t = 0; t + 1 < T; ++t) {
#pragma unroll
      for (int k = 0; k < NB; ++k) {
        const int s = t * NB + k;
        // DMA(s + 2) is issued after this sub-step's barrier; its flags, read
        // halfway through the products, are checked once they are done.
        const int s2 = s + 2, t2 = s2 / NB;
        const int k2 = (k + 2) % NB;
        const bool need2 = s2 < S && t2 >= 1;
        unsigned v2 = 0;
        f32x4 acc = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        if (t >= 1) {
          // buffer s & 1 (NB is even): each read is one contiguous KiB over
          // the wave's lanes
          const _Float16* bsrc = ring + (k & 1) * TBUF + lane * 8;
#pragma unroll
          for (int c = 0; c < KC; ++c) {
            if (c == KC / 2 && need2)
              v2 = __hip_atomic_load(flags + k2 * 64 + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            const uint4 w0 = *reinterpret_cast<const uint4*>(bsrc + c * 2 * FRAG);
            const uint4 w1 = *reinterpret_cast<const uint4*>(bsrc + c * 2 * FRAG + FRAG);
            // Words: lane (lr, lg) takes those of waves 2 lg and 2 lg + 1 for
            // its row (K 8 lg .. + 3 and 8 lg + 4 .. + 7); fragments: as read.
            const uint4 bh = kWords ? make_uint4(w0.x, w0.y, w1.x, w1.y) : w0;
            const uint4 bl = kWords ? make_uint4(w0.z, w0.w, w1.z, w1.w) : w1;
            const h8 AH = __builtin_bit_cast(h8, wh[c]), AL = __builtin_bit_cast(h8, wl[c]);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(AL, __builtin_bit_cast(h8, bh), acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(AH, __builtin_bit_cast(h8, bl), acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(AH, __builtin_bit_cast(h8, bh), acc, 0, 0, 0);
          }
        } else if (need2) {
          v2 = __hip_atomic_load(flags + k2 * 64 + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        // Every memory access of this wave has completed: the stores of
        // sub-step s - 1, the DMA of sub-step s + 1, the flag load, the inputs.
        // (Loads and stores share the counter and may complete out of order,
        // so only a full wait is sound here.)
        wait_vmem();
        // Layer 1: the inputs of the next sub-step's tile, as early as they
        // can go (the folded table's rows are gathered by byte value and often
        // miss the cache; the next wait covers them, a whole sub-step on).
        if constexpr (kL1) {
          if (s + 1 < S) load_inputs(k + 1 < NB ? t : t + 1, (k + 1) % NB);
        }
        __syncthreads();
        // Raise the flag of the previous publication (tile k - 1 at step t, or
        // the last tile at step t - 1): every wave's stores of it completed
        // before the barrier.
        if (threadIdx.x == 0 && s > 0) {
          const int kp = (k + NB - 1) % NB;
          const unsigned vp = base + static_cast<unsigned>(k == 0 ? t : t + 1);
          __hip_atomic_store(flags + kp * 64 + utile, vp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if (need2 && !ready(base + t2, v2)) wait_flags(k2, base + t2);
        // Every wave's products of this sub-step are done: its LDS buffer
        // takes the DMA of sub-step s + 2.
        if (kWords && need2) issue(s2);
        float h;
        {
          const float4 g = gi[k];
          lstm_cell(acc[0] + g.x, acc[1] + g.y, acc[2] + g.z, acc[3] + g.w, cs[k], h);
        }
        // Deeper layers: the tile's inputs of the next step, streamed from
        // the gate inputs (past the last step they read zeros past the
        // buffer); issued here they cost less than right after the wait.
        if constexpr (!kL1) load_inputs(t + 1, k);
        typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
        if constexpr (kWords) {
          // Publish h_t of tile k straight from the cell lanes.  Lane (lr, lg)
          // holds unit 4 wave + lg of row lr; the swaps give every lane of
          // the row all four units.  Lane group 0 stores the row's word (the
          // four hi parts, then the four lo parts), lane group 2 the four
          // fp32 values to the layer's sequence when the row is inside the
          // batch.  Every 128-byte line of the ring is written by one wave.
          const auto p16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(h), __float_as_uint(h), false, false);
          const auto qa = __builtin_amdgcn_permlane32_swap(p16[0], p16[0], false, false);   // units 0, 2
          const auto qb = __builtin_amdgcn_permlane32_swap(p16[1], p16[1], false, false);   // units 1, 3
          const float4 hv = make_float4(__uint_as_float(qa[0]), __uint_as_float(qb[0]), __uint_as_float(qa[1]),
                                        __uint_as_float(qb[1]));
          if (lg == 0) {
            uint2 hi, lo;
            split4(hv, hi, lo);
            const uint32_t off = static_cast<uint32_t>((grp * XSLOT + ((t & 1) * NB + k) * XTILE + utile * 2 * FRAG +
                                                        (wave & 1) * FRAG + (16 * (wave >> 1) + lr) * 8) * 2);
            __builtin_amdgcn_raw_buffer_store_b128(u32x4{hi.x, hi.y, lo.x, lo.y}, xbuf, off, 0, kCoherent);
          } else if (lg == 2 && k * 16 + lr < B) {
            const uint32_t off = static_cast<uint32_t>(((t * B + k * 16 + lr) * H + utile * NU + 4 * wave) * 4);
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, hv), hbuf, off, 0, 0);
          }
        } else {
          // Fragment order: h_t of the tile is transposed through LDS, then
          // threads 0..127 (part, word, row) split 8 units of one row into one
          // fragment word, each wave storing whole lines; threads 128..255
          // (row, quarter of 4 units) store the fp32 rows of the tile inside
          // the batch.  (Halves of one word stored by two waves, device
          // coherent, now and then left a half two steps old.)
          ht[lr * HTLD + wave * 4 + lg] = h;
          __syncthreads();
          if (need2) issue(s2);
          const int tid = threadIdx.x;
          if (tid < 128) {
            const int rr = tid & 15, hw = (tid >> 4) & 3, part = tid >> 6;
            const float* srcw = &ht[rr * HTLD + 8 * hw];
            uint4 hi, lo;
            split8v(*reinterpret_cast<const float4*>(srcw), *reinterpret_cast<const float4*>(srcw + 4), hi, lo);
            const uint4 v = part ? lo : hi;
            const uint32_t off = static_cast<uint32_t>(
                (grp * XSLOT + ((t & 1) * NB + k) * XTILE + (utile * 2 + part) * FRAG + (16 * hw + rr) * 8) * 2);
            __builtin_amdgcn_raw_buffer_store_b128(u32x4{v.x, v.y, v.z, v.w}, xbuf, off, 0, kCoherent);
          } else if (tid < 256) {
            if (p.split_out) {
              // The same words as the exchange's, into the sequence's
              // fragment-order layout: 1 KiB block (row tile, part, k chunk
              // = this block's units), word 16 hw + rr.  (B % 16 == 0, so a
              // tile of the batch is one row tile of the sequence.)  16-byte
              // stores: a version with two 8-byte stores per thread (whose
              // data registers the next instruction rewrote) left non-finite
              // values under the Rademacher laws at H = 128; its cause was
              // not established.
              const int u = tid - 128, rr = u & 15, hw = (u >> 4) & 3, part = u >> 6;
              const float* srcw = &ht[rr * HTLD + 8 * hw];
              uint4 hi, lo;
              split8v(*reinterpret_cast<const float4*>(srcw), *reinterpret_cast<const float4*>(srcw + 4), hi, lo);
              const uint4 v = part ? lo : hi;
              const int rt = (t * B) / 16 + k;
              __builtin_amdgcn_raw_buffer_store_b128(
                  u32x4{v.x, v.y, v.z, v.w}, hbuf,
                  static_cast<uint32_t>((((rt * 2 + part) * KC + utile) * FRAG + (16 * hw + rr) * 8) * 2), 0, 0);
            } else {
              const int n = (tid - 128) >> 3, c4 = tid & 7, row = k * 16 + n;
              if (row < B) {
                const float4 v = *reinterpret_cast<const float4*>(&ht[n * HTLD + 4 * c4]);
                __builtin_amdgcn_raw_buffer_store_b128(
                    __builtin_bit_cast(u32x4, v), hbuf,
                    static_cast<uint32_t>(((t * B + row) * H + utile * NU + 4 * c4) * 4), 0, 0);
              }
            }
          }
        }
      }
    }
    // The job's last publication (tile NB - 1 at step T - 2).
    wait_vmem();
    __syncthreads();
    if (threadIdx.x == 0)
      __hip_atomic_store(flags + (NB - 1) * 64 + utile, base + static_cast<unsigned>(T - 1), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
  }
}

// ---------------------------------------------------------------------------
// Recurrence of one layer for H = 64 (perturbed step only), one block per
// (expert, direction, sign) job.  All 4H = 256 gate rows of a job fit one
// block's registers (each of the 8 waves keeps 32 rows, two MFMA row tiles,
// as split fragments: 32 VGPRs at K = 64), so h never leaves the block
// between steps: the cell updates of step t write h_t, split into fp16
// parts, into one of two LDS buffers while the products of step t read
// h_{t-1} from the other, and one block barrier separates the steps -- no
// group counter, no cross-CU exchange, no cooperative launch; several jobs
// share a compute unit.  h_t is also stored to the slot's hseq rows for the
// next layer and the head.  Lane (wave, lr, lg) owns units 8 wave + 2 lg + m
// (m < 2: adjacent units, stored as pairs) of batch rows 16 nb + lr; rows
// past the batch compute on whatever follows in the input buffers and are
// never stored.  Probes and weights
// are those of k_rec_persist (same canonical indices, same order of
// operations), the products the same three split passes.
//
// Gate inputs.  KX = 0: read per step, from the slot's gin rows (layers
// >= 2) or gathered from the folded table U by byte value (layer 1).
// KX = E / 32 > 0 (layer 1 only, E = 32 or 64, B T <= kLocalBytes): the
// block forms them itself.  It keeps the input columns of W_1+- as split
// fragments beside the recurrent ones, and in LDS the whole perturbed
// embedding table Emb+- (256 x E, split into fp16 parts: E KiB) and the
// job's B x T bytes, and adds x_t W_1x+-^T with KX more chunks of the same
// three passes, x_t being the table row of byte b_t: the fold's 256-row
// table per slot and its per-step row gathers from HBM are never formed,
// and the loop issues no vector-memory load (a wait for one would also wait
// for the h stores before it: loads and stores share one counter).
// ---------------------------------------------------------------------------
constexpr int kLocalThreads = 512;
// Below this L1 norm of every perturbed head row, |logit| < 64 (|h| < 1), so
// e^logit neither overflows nor underflows in fp32 and the row maximum need
// not be subtracted before exponentiating.
constexpr float kNoShiftL1 = 64.0f;
constexpr int kLocalBytes = 16384;                      // largest B T kept in LDS (KX > 0)

template <int NB, bool kRad, int KX, bool kHead>
__global__ __launch_bounds__(kLocalThreads) __attribute__((amdgpu_waves_per_eu(kHead && NB == 1 ? 4 : 1)))
void k_rec_local(FwdArgs a, int jobs) {
  constexpr int H = 64, G = 4 * H;                      // gate rows of a job
  constexpr int KC = H / 32;                            // 32-wide k chunks
  constexpr int MT = G / (16 * 8);                      // row tiles per wave
  constexpr int ROWS = NB * 16;
  constexpr int EW = 32 * KX;                           // embedding width held in LDS (KX > 0)
  constexpr int HSW = H + 16;                           // LDS row of staged h in halves (160 B: an odd multiple of 32)
  constexpr int kZw = H + 8;                            // probe scratch row in floats (288 B)
  constexpr int PART = ROWS * HSW;                      // halves per fp16 part of one buffer
  constexpr int EMB_BYTES = 2 * kVocab * EW * 2;        // [hi, lo][256][EW] halves
  constexpr int BT_BYTES = KX > 0 ? kLocalBytes : 0;    // the job's bytes [B][T]
  constexpr int H_BYTES = 2 * 2 * PART * 2;            // [buffer][hi, lo][ROWS][HSW] halves
  // the fused head's per-wave partials (max, sum exp) and target logits of
  // each row, by step parity: [2][8][ROWS] float2, [2][ROWS] float
  constexpr int HEAD_BYTES = kHead ? 2 * 8 * ROWS * 8 + 2 * ROWS * 4 : 0;
  constexpr int ST_BYTES = EMB_BYTES + BT_BYTES + H_BYTES + HEAD_BYTES;
  constexpr int ZS_BYTES = 128 * kZw * 4;
  constexpr int LDS_BYTES = ST_BYTES > ZS_BYTES ? ST_BYTES : ZS_BYTES;
  static_assert(MT == 2 && KC == 2, "H = 64");
  static_assert(KX >= 0 && KX <= 2 && EW <= kZw, "E = 32 or 64");
  static_assert(!kHead || KX > 0, "the fused head reads the targets from the job's bytes in LDS");
  __shared__ __attribute__((aligned(16))) unsigned char lds[LDS_BYTES];
  _Float16* et = reinterpret_cast<_Float16*>(lds);     // Emb+- parts: hi at et, lo at et + 256 EW
  unsigned char* bts = lds + EMB_BYTES;                 // bytes of row n, step t at bts[n T + t]
  _Float16* hs = reinterpret_cast<_Float16*>(lds + EMB_BYTES + BT_BYTES);   // buffer b, part q at hs + (2 b + q) PART
  float2* red = reinterpret_cast<float2*>(lds + EMB_BYTES + BT_BYTES + H_BYTES);   // [parity][wave][row]
  float* tgl = reinterpret_cast<float*>(lds + EMB_BYTES + BT_BYTES + H_BYTES + 2 * 8 * ROWS * 8);   // [parity][row]
  __shared__ double dsum[ROWS];                         // the fused head's per-row cross-entropy sums
  __shared__ unsigned wide;                             // some head row has L1 norm >= kNoShiftL1
  float* zs = reinterpret_cast<float*>(lds);
  const int job = blockIdx.x;
  if (job >= jobs) return;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  const int B = a.B, T = a.T, in = a.in_l;
  const int64_t R = static_cast<int64_t>(T - 1) * B;
  const int sg = job & 1, pj = job >> 1;
  const int e = pj / a.pcs, jl = pj % a.pcs;
  const float* th = a.theta + static_cast<int64_t>(e) * a.d;
  const uint2 key = stream_key(a.seeds[e], a.step);
  const uint32_t pair = static_cast<uint32_t>(a.j0 + jl), step_lo = static_cast<uint32_t>(a.step);
  const int64_t slot = (static_cast<int64_t>(e) * a.PC + jl) * 2 + sg;
  const float seps = sg == 0 ? eps_of(a, e, kGroupLstm) : -eps_of(a, e, kGroupLstm);
  const float seps_emb = sg == 0 ? eps_of(a, e, kGroupEmb) : -eps_of(a, e, kGroupEmb);
  const __amdgpu_buffer_rsrc_t hbuf = buffer_of(a.hseq + slot * R * H, static_cast<uint32_t>(R * H * sizeof(float)));
  const __amdgpu_buffer_rsrc_t bbuf = buffer_of(bytes_of(a, e, jl), static_cast<uint32_t>(B * T));
  auto probe4 = [&](uint64_t kk) {
    return kRad ? rademacher_quad(key, pair, step_lo, kk, a.probe == kProbeRademacher)
                : gauss_quad(key, pair, step_lo, kk >> 2);
  };

  // Weights: MFMA row lr of row tile m is gate lr & 3 of unit 8 wave +
  // 2 (lr >> 2) + m, gate-interleaved row 32 wave + 8 (lr >> 2) + 4 m +
  // (lr & 3) (row 4u + g is gate g of unit u, canonical row g H + u), so the
  // result lane (lr, lg) holds all four gates of units 8 wave + 2 lg + m;
  // the recurrent columns [in, in + H) into wh/wl, with KX > 0 also the
  // input columns [0, E) into xh/xl.  The probes of 128 rows of one column
  // segment are drawn into the LDS scratch at a time.
  uint4 wh[MT][KC], wl[MT][KC];
  uint4 xh[MT][KX > 0 ? KX : 1], xl[MT][KX > 0 ? KX : 1];
  bool in_range = true;                                 // every split weight within the split's range
  auto canon = [&](int r) { return (r & 3) * H + (r >> 2); };
#pragma unroll
  for (int rg = 0; rg < G / 128; ++rg) {
#pragma unroll
    for (int seg = 0; seg < (KX > 0 ? 2 : 1); ++seg) {
      const int c0 = seg == 0 ? in : 0;                 // first column of the segment
      const int W4 = seg == 0 ? H / 4 : EW / 4;         // its width in quads
      __syncthreads();
      for (int q = threadIdx.x; q < 128 * W4; q += kLocalThreads) {
        const int m = q / W4, k4 = q % W4;
        const uint64_t kk = static_cast<uint64_t>(a.off_l + static_cast<int64_t>(canon(128 * rg + m)) * (in + H) +
                                                  c0 + 4 * k4);
        *reinterpret_cast<float4*>(&zs[m * kZw + 4 * k4]) = probe4(kk);
      }
      __syncthreads();
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        if ((32 * wave) / 128 != rg) continue;         // wave-uniform
        const int row = 32 * wave + 8 * (lr >> 2) + 4 * m + (lr & 3);
        const int64_t wrow = a.off_l + static_cast<int64_t>(canon(row)) * (in + H) + c0;
#pragma unroll
        for (int c = 0; c < (seg == 0 ? KC : KX); ++c) {
          const float* zr = &zs[(row - 128 * rg) * kZw + 32 * c + 8 * lg];
          const float* tr = th + wrow + 32 * c + 8 * lg;
          float4 w0 = fma4(seps, *reinterpret_cast<const float4*>(zr), *reinterpret_cast<const float4*>(tr));
          float4 w1 = fma4(seps, *reinterpret_cast<const float4*>(zr + 4), *reinterpret_cast<const float4*>(tr + 4));
          const float gs = gate_scale(lr & 3);
          w0 = make_float4(w0.x * gs, w0.y * gs, w0.z * gs, w0.w * gs);
          w1 = make_float4(w1.x * gs, w1.y * gs, w1.z * gs, w1.w * gs);
          in_range = in_range && split_range_ok(w0) && split_range_ok(w1);   // the scaled weight is split
          if (seg == 0)
            split8v(w0, w1, wh[m][c], wl[m][c]);
          else
            split8v(w0, w1, xh[m][c], xl[m][c]);
        }
      }
    }
  }
  // Head (kHead): wave w keeps vocabulary rows 32 w + 16 m + lr (m < 2) of
  // Whead+- over all 64 columns as split fragments, the same layout as the
  // recurrent rows, so the head's products take the same B fragments.  The
  // rows' L1 norms decide whether the row maxima must be subtracted before
  // exponentiating (as in k_head_fused: |h| < 1 bounds each logit by its
  // row's L1 norm).
  uint4 vh[kHead ? MT : 1][KC], vl[kHead ? MT : 1][KC];
  if constexpr (kHead) {
    const float seps_head = sg == 0 ? eps_of(a, e, kGroupHead) : -eps_of(a, e, kGroupHead);
    float l1[MT] = {0.0f, 0.0f};
    if (threadIdx.x == 0) wide = 0u;
#pragma unroll
    for (int rg = 0; rg < kVocab / 128; ++rg) {
      __syncthreads();
      for (int q = threadIdx.x; q < 128 * (H / 4); q += kLocalThreads) {
        const int m = q / (H / 4), k4 = q % (H / 4);
        *reinterpret_cast<float4*>(&zs[m * kZw + 4 * k4]) =
            probe4(static_cast<uint64_t>(a.off_head + static_cast<int64_t>(128 * rg + m) * H + 4 * k4));
      }
      __syncthreads();
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        const int row = 32 * wave + 16 * m + lr;
        if (row / 128 != rg) continue;                 // wave-uniform
#pragma unroll
        for (int c = 0; c < KC; ++c) {
          const float* zr = &zs[(row - 128 * rg) * kZw + 32 * c + 8 * lg];
          const float* tr = th + a.off_head + static_cast<int64_t>(row) * H + 32 * c + 8 * lg;
          const float4 w0 = fma4(seps_head, *reinterpret_cast<const float4*>(zr), *reinterpret_cast<const float4*>(tr));
          const float4 w1 =
              fma4(seps_head, *reinterpret_cast<const float4*>(zr + 4), *reinterpret_cast<const float4*>(tr + 4));
          in_range = in_range && split_range_ok(w0) && split_range_ok(w1);
          split8v(w0, w1, vh[m][c], vl[m][c]);
          l1[m] += ((fabsf(w0.x) + fabsf(w0.y)) + (fabsf(w0.z) + fabsf(w0.w))) +
                   ((fabsf(w1.x) + fabsf(w1.y)) + (fabsf(w1.z) + fabsf(w1.w)));
        }
      }
    }
#pragma unroll
    for (int m = 0; m < MT; ++m)
      if (group4_sum(l1[m]) >= kNoShiftL1) wide = 1u;
  }
  __syncthreads();                                      // the scratch becomes the embedding table and the h buffers
  const bool shift = !kHead || wide != 0u;              // block-uniform

  if constexpr (KX > 0) {
    // Emb+-[v][k] = theta[v E + k] +- eps z (canonical offset 0), split.
    for (int q = threadIdx.x; q < kVocab * EW / 4; q += kLocalThreads) {
      const int kk = 4 * q;                             // = v EW + 4 k4
      const float4 w = fma4(seps_emb, probe4(static_cast<uint64_t>(kk)), *reinterpret_cast<const float4*>(th + kk));
      in_range &= split_range_ok(w);
      uint2 hi, lo;
      split4(w, hi, lo);
      *reinterpret_cast<uint2*>(&et[kk]) = hi;
      *reinterpret_cast<uint2*>(&et[kVocab * EW + kk]) = lo;
    }
    // The job's bytes (B T <= kLocalBytes, checked by the host), eight
    // loads in flight per thread (past the end they read 0 and are dropped).
    for (int q0 = 0; q0 < B * T; q0 += 8 * kLocalThreads) {
      int v[8];
#pragma unroll
      for (int i = 0; i < 8; ++i)
        v[i] = __builtin_amdgcn_raw_buffer_load_b8(
            bbuf, static_cast<uint32_t>(q0 + i * kLocalThreads + threadIdx.x), 0, 0);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int q = q0 + i * kLocalThreads + threadIdx.x;
        if (q < B * T) bts[q] = static_cast<unsigned char>(v[i]);
      }
    }
    __syncthreads();
  }

  report_split_range(a.err, in_range);
  float cs[MT][NB];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) cs[m][nb] = 0.0f;
  const uint32_t byte_lane = static_cast<uint32_t>(lr * T);
  const int unit0 = 8 * wave + 2 * lg;                  // unit of row tile 0; row tile m: unit0 + m
  auto load_byte = [&](int nb, int tt) {
    return static_cast<int>(
        __builtin_amdgcn_raw_buffer_load_b8(bbuf, byte_lane, static_cast<uint32_t>(nb * 16 * T + tt), 0));
  };
  // acc += h_{t-1} W_h+-^T, h_{t-1} read from buffer b; with the fused head
  // also hacc = h_{t-1} Whead+-^T (the logits of step t - 1) from the same
  // fragments.  rec = false: the head's products alone (after the last step).
  f32x4 hacc[kHead ? MT : 1][NB];
  auto h_products = [&](f32x4 (&acc)[MT][NB], int b, bool rec) {
    const _Float16* bhi = hs + (2 * b) * PART + lr * HSW + 8 * lg;
    const _Float16* blo = bhi + PART;
    if constexpr (kHead) {
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) hacc[m][nb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    }
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
      uint4 bh[NB], bl[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        bh[nb] = *reinterpret_cast<const uint4*>(bhi + nb * 16 * HSW + 32 * kc);
        bl[nb] = *reinterpret_cast<const uint4*>(blo + nb * 16 * HSW + 32 * kc);
      }
      if (rec) {
#pragma unroll
        for (int m = 0; m < MT; ++m) mfma3_batch<NB>(wh[m][kc], wl[m][kc], bh, bl, acc[m]);
      }
      if constexpr (kHead) {
#pragma unroll
        for (int m = 0; m < MT; ++m) mfma3_batch<NB>(vh[m][kc], vl[m][kc], bh, bl, hacc[m]);
      }
    }
  };
  // Fused head, step tau's logits in hacc: this wave's (max, sum exp) over
  // its 32 vocabulary rows for each batch row, into red[parity][wave], and
  // the target logit of each row from the lane that holds it.
  auto head_partials = [&](int tau, int par) {
    if constexpr (kHead) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      float m = 0.0f;
      if (shift) {
        m = fmaxf(fmaxf(fmaxf(hacc[0][nb][0], hacc[0][nb][1]), fmaxf(hacc[0][nb][2], hacc[0][nb][3])),
                  fmaxf(fmaxf(hacc[1][nb][0], hacc[1][nb][1]), fmaxf(hacc[1][nb][2], hacc[1][nb][3])));
        m = group4_max(m);
      }
      const float ml = -m * kLog2e;
      float sum = 0.0f;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) sum += exp2_f(__builtin_fmaf(hacc[mt][nb][r], kLog2e, ml));
      sum = group4_sum(sum);
      const int n = nb * 16 + lr;
      if (lg == 0) red[(par * 8 + wave) * ROWS + n] = make_float2(m, sum);
      const int y = n < B ? bts[n * T + tau + 1] : 0;
      if (n < B && (y >> 5) == wave && ((y >> 2) & 3) == lg) {
        const int ym = (y >> 4) & 1, yr = y & 3;
        float v = 0.0f;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (mt == ym && r == yr) v = hacc[mt][nb][r];
        tgl[par * ROWS + n] = v;
      }
    }
    }
  };
  // The cross entropy of each batch row at one step from the 8 waves'
  // partials (threads 0 .. B-1, one row each), merged, logged and the target
  // subtracted in fp64, summed per row in fp64.
  double cacc = 0.0;
  auto head_combine = [&](int par) {
    const int n = threadIdx.x;
    if (kHead && n < B) {
      float M = 0.0f;
      double S = 0.0;
      if (shift) {
        M = red[par * 8 * ROWS + n].x;
#pragma unroll
        for (int w = 1; w < 8; ++w) M = fmaxf(M, red[(par * 8 + w) * ROWS + n].x);
        const float ML = -M * kLog2e;
#pragma unroll
        for (int w = 0; w < 8; ++w) {
          const float2 rw = red[(par * 8 + w) * ROWS + n];
          S += static_cast<double>(rw.y * exp2_f(__builtin_fmaf(rw.x, kLog2e, ML)));
        }
      } else {
#pragma unroll
        for (int w = 0; w < 8; ++w) S += static_cast<double>(red[(par * 8 + w) * ROWS + n].y);
      }
      cacc += (log(S) + static_cast<double>(M)) - static_cast<double>(tgl[par * ROWS + n]);
    }
  };
  // Cell updates of step t; h_t into buffer b (split) and to the slot's
  // rows, the lane's two adjacent units as one word per fp16 part and one
  // 8-byte store.
  auto cells = [&](const f32x4 (&acc)[MT][NB], int t, int b) {
    _Float16* dhi = hs + (2 * b) * PART;
    _Float16* dlo = dhi + PART;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      float h[MT];
#pragma unroll
      for (int m = 0; m < MT; ++m)
        lstm_cell_scaled(acc[m][nb][0], acc[m][nb][1], acc[m][nb][2], acc[m][nb][3], cs[m][nb], h[m]);
      const int n = nb * 16 + lr;
      uint32_t hi, lo;
      split2(h[0], h[1], hi, lo);
      *reinterpret_cast<uint32_t*>(dhi + n * HSW + unit0) = hi;
      *reinterpret_cast<uint32_t*>(dlo + n * HSW + unit0) = lo;
      if (!kHead && n < B) {                            // the fused head needs no h in HBM
        typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
        __builtin_amdgcn_raw_buffer_store_b64(u32x2{__float_as_uint(h[0]), __float_as_uint(h[1])}, hbuf,
                                              static_cast<uint32_t>(((t * B + n) * H + unit0) * 4), 0, 0);
      }
    }
  };

  if constexpr (KX == 0) {
    const __amdgpu_buffer_rsrc_t gbuf =
        a.layer == 0 ? buffer_of(a.U + slot * kVocab * G, static_cast<uint32_t>(kVocab * G * sizeof(float)))
                     : buffer_of(a.gin + slot * R * G, static_cast<uint32_t>(R * G * sizeof(float)));
    // The gate inputs of step t + 2 are requested at step t, into the ring
    // slot (t & 1) that step t's own inputs just left (a step here is well
    // under the latency of those loads).  Layer 1 gathers them by byte
    // value: the byte of step t + 2 was requested at step t - 2, right after
    // that step's gate inputs, so waiting for it waits for nothing the step
    // does not need anyway (one wave's loads complete in order).
    int vb[2][NB];                                      // bytes of steps t + 2 (slot t & 1)
    float4 gi[2][MT][NB];                               // gate inputs of steps t, t + 1 (slot t & 1)
    const uint32_t gi_lane = static_cast<uint32_t>((lr * G + 4 * unit0) * 4);
    auto load_inputs = [&](float4 (&g)[MT][NB], const int (&v)[NB], int tt) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int m = 0; m < MT; ++m)
          g[m][nb] = a.layer == 0
                         ? buffer_load_f4<0>(gbuf, static_cast<uint32_t>((v[nb] * G + 4 * (unit0 + m)) * 4))
                         : buffer_load_f4s<0>(gbuf, gi_lane + 16 * m,
                                              static_cast<uint32_t>((tt * B + nb * 16) * G * 4));
    };
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      vb[0][nb] = a.layer == 0 ? load_byte(nb, 0) : 0;
      vb[1][nb] = a.layer == 0 && T > 2 ? load_byte(nb, 1) : 0;
    }
    load_inputs(gi[0], vb[0], 0);
    if (T > 2) load_inputs(gi[1], vb[1], 1);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      vb[0][nb] = a.layer == 0 && T > 3 ? load_byte(nb, 2) : 0;
      vb[1][nb] = a.layer == 0 && T > 4 ? load_byte(nb, 3) : 0;
    }
    // One step; P = t & 1 selects the ring slots at compile time.
    auto step = [&](int t, auto Pc) {
      constexpr int P = decltype(Pc)::value;
      f32x4 acc[MT][NB];
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          acc[m][nb] = f32x4{gi[P][m][nb].x * gate_scale(0), gi[P][m][nb].y * gate_scale(1),
                             gi[P][m][nb].z * gate_scale(2), gi[P][m][nb].w * gate_scale(3)};
      if (t + 3 < T) {
        load_inputs(gi[P], vb[P], t + 2);
        if (a.layer == 0 && t + 5 < T) {
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) vb[P][nb] = load_byte(nb, t + 4);
        }
      }
      if (t > 0) h_products(acc, P ^ 1, true);          // h_{t-1}: buffer (t - 1) & 1
      cells(acc, t, P);
      __syncthreads();
    };
    for (int t = 0; t + 1 < T; t += 2) {
      step(t, std::integral_constant<int, 0>{});
      if (t + 2 < T) step(t + 1, std::integral_constant<int, 1>{});
    }
  } else {
    // acc = x_t W_1x+-^T for the byte v of each of the lane's rows: B
    // operand rows of the embedding table.
    auto x_products = [&](f32x4 (&acc)[MT][NB], const int (&v)[NB]) {
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[m][nb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int kx = 0; kx < KX; ++kx) {
        uint4 bh[NB], bl[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const _Float16* er = et + v[nb] * EW + 32 * kx + 8 * lg;
          bh[nb] = *reinterpret_cast<const uint4*>(er);
          bl[nb] = *reinterpret_cast<const uint4*>(er + kVocab * EW);
        }
#pragma unroll
        for (int m = 0; m < MT; ++m) mfma3_batch<NB>(xh[m][kx], xl[m][kx], bh, bl, acc[m]);
      }
    };
    // The input product of step t + 1 is formed at the end of step t, off
    // the path through the barrier.  Rows past the batch take byte 0.
    auto bytes_at = [&](int (&v)[NB], int tt) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int n = nb * 16 + lr;
        v[nb] = n < B ? bts[n * T + tt] : 0;
      }
    };
    int vb[NB];
    f32x4 acc[MT][NB];
    bytes_at(vb, 0);
    x_products(acc, vb);
    // With the fused head, step t also forms the logits of step t - 1 from
    // h_{t-1} (its partials into parity t & 1) and merges those of step t - 2
    // (parity (t - 1) & 1, written before the previous barrier).
    for (int t = 0; t + 1 < T; ++t) {
      if (t > 0) h_products(acc, (t & 1) ^ 1, true);    // h_{t-1}: buffer (t - 1) & 1
      if constexpr (kHead) {
        if (t > 1) head_combine((t - 1) & 1);
        if (t > 0) head_partials(t - 1, t & 1);
      }
      cells(acc, t, t & 1);
      if (t + 2 < T) {                                  // step t + 1 exists
        bytes_at(vb, t + 1);
        x_products(acc, vb);
      }
      __syncthreads();
    }
    if constexpr (kHead) {
      // The last step's logits (h_{T-2}, buffer (T - 2) & 1), then the
      // block's cross-entropy sum: part[slot][0], the other tiles 0.
      const int tl = T - 2;
      if (tl > 0) head_combine(tl & 1);
      h_products(acc, tl & 1, false);
      head_partials(tl, (tl + 1) & 1);
      __syncthreads();
      head_combine((tl + 1) & 1);
      if (threadIdx.x < ROWS) dsum[threadIdx.x] = cacc;
      __syncthreads();
      if (threadIdx.x == 0) {
        double tot = 0.0;
        for (int n = 0; n < ROWS; ++n) tot += dsum[n];
        a.part[slot * a.row_tiles] = tot;
      }
      for (int i = 1 + static_cast<int>(threadIdx.x); i < a.row_tiles; i += kLocalThreads) a.part[slot * a.row_tiles + i] = 0.0;
    }
  }
}

// ---------------------------------------------------------------------------
// Input projection of layer l >= 2 with register-resident weights:
//   gin[slot][row][4u+g] = sum_{k<H} W_l+-[g H + u][k] h_{l-1}[slot][row][k]
// A block owns one job, the 128 gate rows [128 mb, +128) of one (expert,
// direction, sign) slot: it forms their perturbed weights in registers once
// (the probes are drawn once per job instead of once per row tile) and
// streams all R = B (T-1) rows of the slot's h through a double-buffered LDS
// ring of 64-row chunks of 256 K values where H allows (else 128 or 64), one
// barrier per chunk; each lane stores the four gates of one unit for its rows
// after every 64-row tile.
// Grid: slots * mblocks blocks of 512 threads; where the slot count is a
// multiple of 8 the 16 row blocks of a slot run on one XCD (blocks are dealt
// to XCDs round-robin), so they share its L2 while streaming the same h.
// ---------------------------------------------------------------------------
constexpr int kProjThreads = 512;
constexpr int kStreamMaxH = 704;      // resident rows of K = 704: 176 VGPRs of split fragments per lane

template <int NCH, bool kRad>
__global__ __launch_bounds__(kProjThreads, NCH <= 2 ? 4 : 1) void k_proj_stream(FwdArgs a, int mblocks, int nslots) {
  constexpr int KC = 2 * NCH;                 // 32-wide k chunks: K = H = 64 NCH
  // ring chunks per row tile: 256 k each where possible, else 128 or 64
  constexpr int NQ = NCH % 4 == 0 ? NCH / 4 : (NCH > 8 ? (NCH % 2 == 0 ? NCH / 2 : NCH) : split_quarters(NCH));
  constexpr int QC = KC / NQ;                 // k chunks per ring chunk
  constexpr int KW = QC * 32;                 // k per ring chunk
  constexpr int SW = KW + 16;                 // padded LDS row in halves (an odd multiple of 32 bytes)
  constexpr int CF4 = 64 * KW / 4;            // float4 per ring chunk
  constexpr int PT = (CF4 + kProjThreads - 1) / kProjThreads;
  constexpr int RING_BYTES = 2 * 2 * 64 * SW * 2;
  constexpr int ZW = KC * 32 < kZpiece ? KC * 32 : kZpiece;   // probe piece width
  constexpr int ZS_BYTES = 128 * (ZW + 8) * 4;
  constexpr int LDS_BYTES = RING_BYTES > ZS_BYTES ? RING_BYTES : ZS_BYTES;
  // ring [buf][hi, lo][64][SW] halves; probe scratch while forming weights
  __shared__ __attribute__((aligned(16))) unsigned char lds[LDS_BYTES];
  _Float16* ring = reinterpret_cast<_Float16*>(lds);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform (scalar)
  const int lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  const int H = a.H, B = a.B, T = a.T;
  const int R = (T - 1) * B;
  const int H4 = 4 * H;

  int ps, mb;                                 // slot of this pass, row block
  {
    const int b = blockIdx.x;
    if (nslots % 8 == 0) {
      const int i = b / 8;
      mb = i % mblocks;
      ps = (i / mblocks) * 8 + b % 8;
    } else {
      ps = b / mblocks;
      mb = b % mblocks;
    }
  }
  const int sg = ps & 1, pj = ps >> 1;
  const int e = pj / a.pcs, jl = pj % a.pcs;
  const int64_t slot = (static_cast<int64_t>(e) * a.PC + jl) * 2 + sg;
  const float* th = a.theta + static_cast<int64_t>(e) * a.d;
  const uint2 key = stream_key(a.seeds[e], a.step);
  const uint32_t pair = static_cast<uint32_t>(a.j0 + jl), step_lo = static_cast<uint32_t>(a.step);
  const float seps = sg == 0 ? eps_of(a, e, kGroupLstm) : -eps_of(a, e, kGroupLstm);
  const int unit = mb * 32 + wave * 4 + lg;   // output unit of this lane
  // 32-bit offsets: R 4H floats < 2^31 bytes (host check).
  const __amdgpu_buffer_rsrc_t hbuf =
      buffer_of(a.hseq + slot * R * H, static_cast<uint32_t>(static_cast<int64_t>(R) * H * sizeof(float)));
  const __amdgpu_buffer_rsrc_t gbuf =
      buffer_of(a.gin + slot * R * H4, static_cast<uint32_t>(static_cast<int64_t>(R) * H4 * sizeof(float)));

  uint4 wh[KC], wl[KC];
  resident_weights_split<KC, true, kRad, ZW>(wh, wl, reinterpret_cast<float*>(lds), th, a.off_l, a.in_l + H, 0, H,
                                         mb * 128, a.probe, key, pair, step_lo, seps, a.err);

  // Ring chunk c covers rows [64 (c / NQ), +64) and k [KW (c % NQ), +KW);
  // rows past R read row R - 1 and are never stored.  h is split into its
  // fp16 parts as it is staged.
  const int nchunks = ((R + 63) / 64) * NQ;
  // Wave load i of a ring chunk covers rows (wave + 8 i) RPW + lane / CW4,
  // float4 lane % CW4 of the chunk: a per-lane part and a scalar part.
  // Rows past R read zeros (past the slot's buffer) and are never stored.
  constexpr int CW4 = KW / 4, RPW = 64 / CW4;
  static_assert(CW4 * RPW == 64 && PT * 8 * RPW == 64, "ring chunk rows must split evenly over the waves");
  const int lrow = lane / CW4, lc4 = lane % CW4;
  const uint32_t lane_off = static_cast<uint32_t>((lrow * H + 4 * lc4) * 4);
  float4 pre[PT];
  auto gload = [&](int c) {
    const int r0 = (c / NQ) * 64, k0 = (c % NQ) * KW;
#pragma unroll
    for (int i = 0; i < PT; ++i) {
      const uint32_t soff = static_cast<uint32_t>(((r0 + (wave + 8 * i) * RPW) * H + k0) * 4);
      typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
      const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(hbuf, lane_off, soff, 0);
      pre[i] = make_float4(__uint_as_float(v[0]), __uint_as_float(v[1]), __uint_as_float(v[2]), __uint_as_float(v[3]));
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < PT; ++i) {
      const int n = (wave + 8 * i) * RPW + lrow;
      uint2 hi, lo;
      split4(pre[i], hi, lo);
      *reinterpret_cast<uint2*>(ring + ((buf * 2) * 64 + n) * SW + 4 * lc4) = hi;
      *reinterpret_cast<uint2*>(ring + ((buf * 2 + 1) * 64 + n) * SW + 4 * lc4) = lo;
    }
  };

  const _Float16* blane = ring + lr * SW + 8 * lg;   // this lane's B fragments sit at constant offsets from here
  f32x4 acc[4];
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  gload(0);
  sstore(0);
  __syncthreads();
  for (int c = 0; c < nchunks; ++c) {
    if (c + 1 < nchunks) gload(c + 1);
    const int buf = c & 1, qq = c % NQ;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      if (q == qq) {                           // compile-time register index into wh, wl
#pragma unroll
        for (int pq = 0; pq < QC; ++pq) {
          uint4 bh[4], bl[4];
#pragma unroll
          for (int nb = 0; nb < 4; ++nb) {
            const int o = nb * 16 * SW + 32 * pq;
            bh[nb] = *reinterpret_cast<const uint4*>(blane + (buf * 2) * 64 * SW + o);
            bl[nb] = *reinterpret_cast<const uint4*>(blane + (buf * 2 + 1) * 64 * SW + o);
          }
          mfma3_batch<4>(wh[q * QC + pq], wl[q * QC + pq], bh, bl, acc);
        }
      }
    }
    if (qq == NQ - 1) {
      const int r0 = (c / NQ) * 64;
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        const int row = r0 + nb * 16 + lr;
        if (row < R) {
          typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc[nb]), gbuf,
                                                 static_cast<uint32_t>((row * H4 + 4 * unit) * 4), 0, 0);
        }
        acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
    if (c + 1 < nchunks) sstore(buf ^ 1);
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// The input projection of k_proj_stream from a pre-split sequence
// (k_proj_dma): where the previous layer's recurrence stored its h already
// split into fp16 parts, in MFMA fragment order -- hseq as 1 KiB blocks
// [16-row tile][hi, lo][32-wide k chunk], word 16 lg + lr holding row lr,
// k 8 lg .. + 7 (the same bytes as fp32) -- the ring is filled by LDS DMA
// (buffer_load_dwordx4 ... lds), one contiguous block per instruction, and
// the products read each fragment as one 16-byte word.  Staging
// then takes no registers, vector instructions, LDS stores or waits beside
// the products: the DMA of the next ring chunk is issued before the current
// chunk's products, and one wait and one barrier close each chunk.  The
// split is the one k_proj_stream applies while staging, so the products and
// results are the same.  The gate inputs of a finished 64-row tile are
// stored after the barrier, so the next wait finds them done.
// ---------------------------------------------------------------------------
template <int NCH, bool kRad>
__global__ __launch_bounds__(kProjThreads, NCH <= 2 ? 4 : 1) void k_proj_dma(FwdArgs a, int mblocks, int nslots) {
  constexpr int KC = 2 * NCH;                 // 32-wide k chunks: K = H = 64 NCH
  constexpr int NQ = NCH % 4 == 0 ? NCH / 4 : (NCH > 8 ? (NCH % 2 == 0 ? NCH / 2 : NCH) : split_quarters(NCH));
  constexpr int QC = KC / NQ;                 // k chunks per ring chunk
  constexpr int KW = QC * 32;                 // k per ring chunk
  constexpr int FRAG = 512;                   // halves per 1 KiB block
  constexpr int NBLK = 2 * 4 * QC;            // blocks per ring chunk: (part, row tile, k chunk)
  constexpr int BUF = NBLK * FRAG;            // halves per ring buffer
  constexpr int BPW = (NBLK + 7) / 8;         // blocks per wave
  constexpr int RING_BYTES = 2 * BUF * 2;
  constexpr int ZW = KC * 32 < kZpiece ? KC * 32 : kZpiece;   // probe piece width
  constexpr int ZS_BYTES = 128 * (ZW + 8) * 4;
  constexpr int LDS_BYTES = RING_BYTES > ZS_BYTES ? RING_BYTES : ZS_BYTES;
  __shared__ __attribute__((aligned(16))) unsigned char lds[LDS_BYTES];
  _Float16* ring = reinterpret_cast<_Float16*>(lds);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  const int H = a.H, B = a.B, T = a.T;
  const int R = (T - 1) * B;
  const int H4 = 4 * H;

  int ps, mb;                                 // slot of this pass, row block (as k_proj_stream)
  {
    const int b = blockIdx.x;
    if (nslots % 8 == 0) {
      const int i = b / 8;
      mb = i % mblocks;
      ps = (i / mblocks) * 8 + b % 8;
    } else {
      ps = b / mblocks;
      mb = b % mblocks;
    }
  }
  const int sg = ps & 1, pj = ps >> 1;
  const int e = pj / a.pcs, jl = pj % a.pcs;
  const int64_t slot = (static_cast<int64_t>(e) * a.PC + jl) * 2 + sg;
  const float* th = a.theta + static_cast<int64_t>(e) * a.d;
  const uint2 key = stream_key(a.seeds[e], a.step);
  const uint32_t pair = static_cast<uint32_t>(a.j0 + jl), step_lo = static_cast<uint32_t>(a.step);
  const float seps = sg == 0 ? eps_of(a, e, kGroupLstm) : -eps_of(a, e, kGroupLstm);
  const int unit = mb * 32 + wave * 4 + lg;   // output unit of this lane
  // 32-bit offsets: R 4H floats < 2^31 bytes (host check).  Every DMA offset
  // is per lane (bounds-checked): row tiles past R (B % 16 == 0) read zeros
  // and are never stored.
  const i32x4 hrs = buffer_words(a.hseq + slot * R * H, static_cast<uint32_t>(static_cast<int64_t>(R) * H * 4));
  const __amdgpu_buffer_rsrc_t gbuf =
      buffer_of(a.gin + slot * R * H4, static_cast<uint32_t>(static_cast<int64_t>(R) * H4 * sizeof(float)));

  uint4 wh[KC], wl[KC];
  resident_weights_split<KC, true, kRad, ZW>(wh, wl, reinterpret_cast<float*>(lds), th, a.off_l, a.in_l + H, 0, H,
                                         mb * 128, a.probe, key, pair, step_lo, seps, a.err);

  // Ring chunk c covers rows [64 (c / NQ), +64) and k [KW (c % NQ), +KW);
  // block b of it is (part b / (4 QC), row tile (b / QC) % 4, k chunk b % QC).
  const int nchunks = ((R + 63) / 64) * NQ;
  auto issue = [&](int c) {
    const int r0 = (c / NQ) * 64, k0 = (c % NQ) * KW;
    const uint32_t dst = lds_address(ring + (c & 1) * BUF);
#pragma unroll
    for (int i = 0; i < BPW; ++i) {
      const int b = wave + 8 * i;
      if (NBLK % 8 == 0 || b < NBLK) {            // wave-uniform
        const int part = b / (4 * QC), nb = (b / QC) % 4, pq = b % QC;
        const int rt = r0 / 16 + nb, kc = k0 / 32 + pq;
        const uint32_t voff = static_cast<uint32_t>((((rt * 2 + part) * KC + kc) * FRAG + lane * 8) * 2);
        dma16(hrs, voff, 0u, dst + static_cast<uint32_t>(b * FRAG * 2));
      }
    }
  };

  f32x4 acc[4];
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  // The weights' probe scratch overlays the ring: the barriers inside the
  // weight formation come before this first DMA.
  issue(0);
  wait_vmem();
  __syncthreads();
  for (int c = 0; c < nchunks; ++c) {
    if (c + 1 < nchunks) issue(c + 1);           // into the buffer chunk c - 1 read
    const int qq = c % NQ;
    const _Float16* bl0 = ring + (c & 1) * BUF + lane * 8;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      if (q == qq) {                           // compile-time register index into wh, wl
#pragma unroll
        for (int pq = 0; pq < QC; ++pq) {
          uint4 bh[4], bl[4];
#pragma unroll
          for (int nb = 0; nb < 4; ++nb) {
            bh[nb] = *reinterpret_cast<const uint4*>(bl0 + (nb * QC + pq) * FRAG);
            bl[nb] = *reinterpret_cast<const uint4*>(bl0 + ((4 + nb) * QC + pq) * FRAG);
          }
          mfma3_batch<4>(wh[q * QC + pq], wl[q * QC + pq], bh, bl, acc);
        }
      }
    }
    // The DMA of chunk c + 1 and the stores of the previous tile are done,
    // every wave's products of chunk c too (its buffer takes chunk c + 2).
    wait_vmem();
    __syncthreads();
    if (qq == NQ - 1) {
      const int r0 = (c / NQ) * 64;
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        const int row = r0 + nb * 16 + lr;
        if (row < R) {
          typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc[nb]), gbuf,
                                                 static_cast<uint32_t>((row * H4 + 4 * unit) * 4), 0, 0);
        }
        acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Output head and cross entropy with register-resident weights, in two
// passes.  k_head_stream: a block owns one job, one vocabulary half (128
// rows of Whead) of one (expert, direction, sign) slot: it forms the
// perturbed rows in registers once and streams all R rows of the slot's top
// layer h through the same double-buffered LDS ring as k_proj_stream.  After
// each 64-row tile it reduces the half's 128 logits of every row to
// (m, s) = (max, sum exp(logit - max)) and the lane holding the target byte
// stores its logit.  k_ce_combine merges the two halves of a row,
//   ce = M + ln(s_0 e^{m_0 - M} + s_1 e^{m_1 - M}) - logit_target,
// M = max(m_0, m_1), and sums each 64-row tile in fp64 (the per-tile sums
// that the loss reduction reads).
// Partials: hpart[slot][half][R] float2 (m, s); htgt[slot][R].
// ---------------------------------------------------------------------------
// The library launches it for H > 128 (k_head_fused covers H <= 128); at
// H <= 128 the probe scratch would be sized by K and the block would ask for
// four waves per SIMD, so that two blocks share a compute unit.
template <int NCH, bool kRad>
__global__ __launch_bounds__(kProjThreads, NCH <= 2 ? 4 : 1) void k_head_stream(FwdArgs a, int nslots,
                                                                             float2* hpart, float* htgt) {
  constexpr int KC = 2 * NCH;                 // 32-wide k chunks: K = H = 64 NCH
  constexpr int NQ = split_quarters(NCH);     // ring chunks per row tile
  constexpr int QC = KC / NQ;
  constexpr int KW = QC * 32;
  constexpr int SW = KW + 16;                 // padded LDS row in halves (an odd multiple of 32 bytes)
  constexpr int CF4 = 64 * KW / 4;
  constexpr int PT = (CF4 + kProjThreads - 1) / kProjThreads;
  constexpr int RING_BYTES = 2 * 2 * 64 * SW * 2;
  constexpr int ZW = KC * 32 < kZpiece ? KC * 32 : kZpiece;   // probe piece width
  constexpr int ZS_BYTES = 128 * (ZW + 8) * 4;
  constexpr int LDS_BYTES = RING_BYTES > ZS_BYTES ? RING_BYTES : ZS_BYTES;
  __shared__ __attribute__((aligned(16))) unsigned char lds[LDS_BYTES];   // ring [buf][hi, lo][64][SW]
  __shared__ float2 red[2][8][64];              // per-wave (m, s) of each row, by tile parity
  _Float16* ring = reinterpret_cast<_Float16*>(lds);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  const int H = a.H, B = a.B, T = a.T;
  const int R = (T - 1) * B;

  int ps, vh;                                   // slot of this pass, vocabulary half
  {
    const int b = blockIdx.x;
    if (nslots % 8 == 0) {
      const int i = b / 8;
      vh = i & 1;
      ps = (i >> 1) * 8 + b % 8;
    } else {
      ps = b >> 1;
      vh = b & 1;
    }
  }
  const int sg = ps & 1, pj = ps >> 1;
  const int e = pj / a.pcs, jl = pj % a.pcs;
  const int64_t slot = (static_cast<int64_t>(e) * a.PC + jl) * 2 + sg;
  const float* th = a.theta + static_cast<int64_t>(e) * a.d;
  const uint2 key = stream_key(a.seeds[e], a.step);
  const uint32_t pair = static_cast<uint32_t>(a.j0 + jl), step_lo = static_cast<uint32_t>(a.step);
  const float seps = sg == 0 ? eps_of(a, e, kGroupHead) : -eps_of(a, e, kGroupHead);
  const int vbase = vh * 128 + wave * 16 + 4 * lg;   // vocabulary rows vbase .. +3 of this lane
  // 32-bit offsets: R H floats < 2^31 bytes (host check).
  const __amdgpu_buffer_rsrc_t hbuf =
      buffer_of(a.hseq + slot * R * H, static_cast<uint32_t>(static_cast<int64_t>(R) * H * sizeof(float)));
  const __amdgpu_buffer_rsrc_t bbuf =
      buffer_of(bytes_of(a, e, jl), static_cast<uint32_t>(B * T));
  float2* hp = hpart + (slot * 2 + vh) * R;
  float* tg = htgt + slot * R;

  uint4 wh[KC], wl[KC];
  resident_weights_split<KC, false, kRad, ZW>(wh, wl, reinterpret_cast<float*>(lds), th, a.off_head, H, 0, H, vh * 128,
                                          a.probe, key, pair, step_lo, seps, a.err);

  const int nchunks = ((R + 63) / 64) * NQ;
  float4 pre[PT];
  auto gload = [&](int c) {
    const int r0 = (c / NQ) * 64, k0 = (c % NQ) * KW;
#pragma unroll
    for (int i = 0; i < PT; ++i) {
      const int idx = threadIdx.x + i * kProjThreads;
      if (idx < CF4) {
        const int c4 = idx % (KW / 4), n = idx / (KW / 4);
        const int row = r0 + n < R ? r0 + n : R - 1;
        pre[i] = buffer_load_f4<0>(hbuf, static_cast<uint32_t>((row * H + k0 + 4 * c4) * 4));
      }
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < PT; ++i) {
      const int idx = threadIdx.x + i * kProjThreads;
      if (idx < CF4) {
        const int c4 = idx % (KW / 4), n = idx / (KW / 4);
        uint2 hi, lo;
        split4(pre[i], hi, lo);
        *reinterpret_cast<uint2*>(ring + ((buf * 2) * 64 + n) * SW + 4 * c4) = hi;
        *reinterpret_cast<uint2*>(ring + ((buf * 2 + 1) * 64 + n) * SW + 4 * c4) = lo;
      }
    }
  };

  f32x4 acc[4];
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  int y[4];                                     // target bytes of this lane's rows in the current tile
  // Row r0 + lr = ytt B + yb of the tile, advanced by 64 rows a tile; rows
  // 16 nb further on add the wave-uniform quotient and remainder of 16 nb
  // by B (rows past R read past the batch: 0 from the buffer, never stored).
  int ytt = lr / B, yb = lr - (lr / B) * B;
  const int q64 = 64 / B, r64 = 64 % B;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int c = 0; c < nchunks; ++c) {
    if (c + 1 < nchunks) gload(c + 1);
    const int buf = c & 1, qq = c % NQ, r0 = (c / NQ) * 64;
    if (qq == NQ - 1) {
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        const int qn = (16 * nb) / B, rn = 16 * nb - qn * B;   // wave-uniform
        int bn = yb + rn, tn = ytt + qn;
        if (bn >= B) {
          bn -= B;
          ++tn;
        }
        y[nb] = __builtin_amdgcn_raw_buffer_load_b8(bbuf, static_cast<uint32_t>(bn * T + tn + 1), 0, 0);
      }
      yb += r64;
      ytt += q64;
      if (yb >= B) {
        yb -= B;
        ++ytt;
      }
    }
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      if (q == qq) {                            // compile-time register index into wh, wl
#pragma unroll
        for (int pq = 0; pq < QC; ++pq) {
          uint4 bh[4], bl[4];
#pragma unroll
          for (int nb = 0; nb < 4; ++nb) {
            const int o = (nb * 16 + lr) * SW + 32 * pq + 8 * lg;
            bh[nb] = *reinterpret_cast<const uint4*>(ring + (buf * 2) * 64 * SW + o);
            bl[nb] = *reinterpret_cast<const uint4*>(ring + (buf * 2 + 1) * 64 * SW + o);
          }
          mfma3_batch<4>(wh[q * QC + pq], wl[q * QC + pq], bh, bl, acc);
        }
      }
    }
    if (qq == NQ - 1) {
      // Lane (lr, lg) holds the logits of vocabulary rows vbase .. +3 for
      // tile rows nb*16 + lr: reduce over the 4 lane groups, then over the
      // 8 waves.
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        const float m = group4_max(fmaxf(fmaxf(acc[nb][0], acc[nb][1]), fmaxf(acc[nb][2], acc[nb][3])));
        // e^{x - m} = 2^{x log2 e - m log2 e}: one fma per logit.
        const float ml = -m * kLog2e;
        const float sum = group4_sum(
            ((exp2_f(__builtin_fmaf(acc[nb][0], kLog2e, ml)) + exp2_f(__builtin_fmaf(acc[nb][1], kLog2e, ml))) +
             exp2_f(__builtin_fmaf(acc[nb][2], kLog2e, ml))) +
            exp2_f(__builtin_fmaf(acc[nb][3], kLog2e, ml)));
        if (lg == 0) red[(c / NQ) & 1][wave][nb * 16 + lr] = make_float2(m, sum);
        const int row = r0 + nb * 16 + lr;
        const int yo = y[nb] - vbase;
        if (row < R && yo >= 0 && yo < 4) {
          float v = acc[nb][0];
#pragma unroll
          for (int r = 1; r < 4; ++r)
            if (yo == r) v = acc[nb][r];
          tg[row] = v;
        }
        acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
    if (c + 1 < nchunks) sstore(buf ^ 1);
    __syncthreads();
    if (qq == NQ - 1 && threadIdx.x < 64 && r0 + static_cast<int>(threadIdx.x) < R) {
      // This buffer is next written two tiles on, behind the next tile's
      // barrier, which these threads reach only after reading it.
      const int n = threadIdx.x;
      const float2 (&rd)[8][64] = red[(c / NQ) & 1];
      float M = rd[0][n].x;
#pragma unroll
      for (int wv = 1; wv < 8; ++wv) M = fmaxf(M, rd[wv][n].x);
      float S = 0.0f;
#pragma unroll
      for (int wv = 0; wv < 8; ++wv) S += rd[wv][n].y * __expf(rd[wv][n].x - M);
      hp[r0 + n] = make_float2(M, S);
    }
  }
}

// ---------------------------------------------------------------------------
// Output head and cross entropy in one pass for H <= 128: a block of 16
// waves owns one (expert, direction, sign) slot and all 256 rows of Whead
// (wave w keeps rows 16 w .. + 15 as split fragments: 16 or 32 VGPRs), so
// each row's cross entropy is finished in the block:
//   ce = M + ln(sum_w s_w e^{m_w - M}) - logit_target,  M = max_w m_w,
// from the 16 waves' (m_w, s_w) = (max, sum exp(logit - max)) over their 16
// vocabulary rows.  All R rows of the slot's top-layer h stream once through
// a double-buffered LDS ring of 64-row tiles (staged and split by all 1024
// threads); the next tile is requested at the start of a tile.  Waves 0..3
// (one per SIMD) combine a tile's partials, 16 rows each, while the next
// tile's products run, and keep fp64 sums per lane; the slot's total goes
// to the first of its per-tile loss partials at the end (the others are
// zeroed: the loss reduction sums them).  The loop issues no store, so
// waiting for the staged tile waits for nothing else.
// ---------------------------------------------------------------------------
constexpr int kHeadFusedThreads = 1024;

template <int NCH, bool kRad>
__global__ __launch_bounds__(kHeadFusedThreads) void k_head_fused(FwdArgs a) {
  constexpr int H = 64 * NCH;                 // 64 or 128
  constexpr int KC = 2 * NCH;                 // 32-wide k chunks
  constexpr int SW = H + 16;                  // ring row in halves (160 or 288 bytes: odd multiples of 32)
  constexpr int PT = 64 * H / 4 / kHeadFusedThreads;   // float4 per thread per tile: 1 or 2
  constexpr int ZLD = H + 8;                  // probe scratch row in floats
  constexpr int RING_BYTES = 2 * 2 * 64 * SW * 2;
  constexpr int ZS_BYTES = 128 * ZLD * 4;
  constexpr int LDS_BYTES = RING_BYTES > ZS_BYTES ? RING_BYTES : ZS_BYTES;
  static_assert(NCH == 1 || NCH == 2, "H = 64 or 128");
  static_assert(PT * kHeadFusedThreads * 4 == 64 * H, "a tile splits evenly over the threads");
  __shared__ __attribute__((aligned(16))) unsigned char lds[LDS_BYTES];   // ring [buf][hi, lo][64][SW]
  __shared__ float2 red[2][16][64];             // per-wave (m, s) of each row, by tile parity
  __shared__ float tgl[2][64];                  // target logit of each row, by tile parity
  __shared__ double dsum[64];
  __shared__ unsigned wide;                     // some row of Whead+- has L1 norm >= kNoShiftL1
  _Float16* ring = reinterpret_cast<_Float16*>(lds);
  float* zs = reinterpret_cast<float*>(lds);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  const int B = a.B, T = a.T;
  const int R = (T - 1) * B;
  const int ps = blockIdx.x;                  // slot of this pass
  const int sg = ps & 1, pj = ps >> 1;
  const int e = pj / a.pcs, jl = pj % a.pcs;
  const int64_t slot = (static_cast<int64_t>(e) * a.PC + jl) * 2 + sg;
  const float* th = a.theta + static_cast<int64_t>(e) * a.d;
  const uint2 key = stream_key(a.seeds[e], a.step);
  const uint32_t pair = static_cast<uint32_t>(a.j0 + jl), step_lo = static_cast<uint32_t>(a.step);
  const float seps = sg == 0 ? eps_of(a, e, kGroupHead) : -eps_of(a, e, kGroupHead);
  const int vbase = wave * 16 + 4 * lg;       // vocabulary rows vbase .. +3 of this lane
  // 32-bit offsets: R H floats < 2^31 bytes (host check).
  const __amdgpu_buffer_rsrc_t hbuf =
      buffer_of(a.hseq + slot * R * H, static_cast<uint32_t>(static_cast<int64_t>(R) * H * sizeof(float)));
  const __amdgpu_buffer_rsrc_t bbuf = buffer_of(bytes_of(a, e, jl), static_cast<uint32_t>(B * T));

  // Whead+- rows 16 wave + lr, drawn 128 rows (one vocabulary half) at a time.
  uint4 wh[KC], wl[KC];
  float l1 = 0.0f;                            // this lane's part of its row's L1 norm
  bool in_range = true;
  if (threadIdx.x == 0) wide = 0u;
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    __syncthreads();
    for (int q = threadIdx.x; q < 128 * (H / 4); q += kHeadFusedThreads) {
      const int m = q / (H / 4), k4 = q % (H / 4);
      const uint64_t kk = static_cast<uint64_t>(a.off_head + static_cast<int64_t>(128 * half + m) * H + 4 * k4);
      *reinterpret_cast<float4*>(&zs[m * ZLD + 4 * k4]) =
          kRad ? rademacher_quad(key, pair, step_lo, kk, a.probe == kProbeRademacher) : gauss_quad(key, pair, step_lo, kk >> 2);
    }
    __syncthreads();
    if ((wave >> 3) == half) {
      const int row = wave * 16 + lr;
      const float* tr = th + a.off_head + static_cast<int64_t>(row) * H;
#pragma unroll
      for (int c = 0; c < KC; ++c) {
        const float* zr = &zs[(row - 128 * half) * ZLD + 32 * c + 8 * lg];
        const float4 w0 = fma4(seps, *reinterpret_cast<const float4*>(zr), *reinterpret_cast<const float4*>(tr + 32 * c + 8 * lg));
        const float4 w1 = fma4(seps, *reinterpret_cast<const float4*>(zr + 4), *reinterpret_cast<const float4*>(tr + 32 * c + 8 * lg + 4));
        in_range = in_range && split_range_ok(w0) && split_range_ok(w1);
        split8v(w0, w1, wh[c], wl[c]);
        l1 += ((fabsf(w0.x) + fabsf(w0.y)) + (fabsf(w0.z) + fabsf(w0.w))) +
              ((fabsf(w1.x) + fabsf(w1.y)) + (fabsf(w1.z) + fabsf(w1.w)));
      }
    }
  }
  report_split_range(a.err, in_range);
  if (group4_sum(l1) >= kNoShiftL1) wide = 1u;
  __syncthreads();                            // the scratch becomes the ring
  // |h| <= 1, so |logit_v| <= ||Whead+-[v]||_1: below kNoShiftL1 for every v,
  // e^logit neither overflows nor underflows in fp32 (a row's sum stays in
  // [256 e^-64, 256 e^64]) and the maximum need not be subtracted.
  const bool shift = wide != 0u;              // block-uniform

  const int ntiles = (R + 63) / 64;
  // Thread load i of a tile covers float4 (threadIdx.x + 1024 i) of its 64 x H
  // block: row n = idx / (H / 4), quad idx % (H / 4).  Rows past R read zeros
  // (past the buffer) and are never used.
  float4 pre[PT];
  auto gload = [&](int c) {
#pragma unroll
    for (int i = 0; i < PT; ++i) {
      const int idx = threadIdx.x + i * kHeadFusedThreads;
      pre[i] = buffer_load_f4<0>(hbuf, static_cast<uint32_t>(((c * 64 + idx / (H / 4)) * H + 4 * (idx % (H / 4))) * 4));
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < PT; ++i) {
      const int idx = threadIdx.x + i * kHeadFusedThreads;
      const int n = idx / (H / 4), c4 = idx % (H / 4);
      uint2 hi, lo;
      split4(pre[i], hi, lo);
      *reinterpret_cast<uint2*>(ring + ((buf * 2) * 64 + n) * SW + 4 * c4) = hi;
      *reinterpret_cast<uint2*>(ring + ((buf * 2 + 1) * 64 + n) * SW + 4 * c4) = lo;
    }
  };

  // Row r0 + lr = ytt B + yb of the tile, advanced by 64 rows a tile; rows
  // 16 nb further on add the wave-uniform quotient and remainder of 16 nb
  // by B (rows past R read past the batch: 0 from the buffer, never used).
  int ytt = lr / B, yb = lr - (lr / B) * B;
  const int q64 = 64 / B, r64 = 64 % B;
  double cacc = 0.0;                          // this combining lane's ce sum (rows 16 wave + lane of every tile)
  f32x4 acc[4];
  // Rows of tile cc from the 16 waves' partials (waves 0..3, one per SIMD,
  // 16 rows each), summed, logged and the target subtracted in fp64: a loss
  // of one token then carries the rounding of the fp32 exponentials and
  // partial sums only.
  auto combine = [&](int cc) {
    const int cb = cc & 1;
    if (wave < 4 && lane < 16 && cc * 64 + wave * 16 + lane < R) {
      const int n = wave * 16 + lane;
      float M = 0.0f;
      double S = 0.0;
      if (shift) {
        M = red[cb][0][n].x;
#pragma unroll
        for (int w = 1; w < 16; ++w) M = fmaxf(M, red[cb][w][n].x);
        const float ML = -M * kLog2e;
#pragma unroll
        for (int w = 0; w < 16; ++w)
          S += static_cast<double>(red[cb][w][n].y * exp2_f(__builtin_fmaf(red[cb][w][n].x, kLog2e, ML)));
      } else {
#pragma unroll
        for (int w = 0; w < 16; ++w) S += static_cast<double>(red[cb][w][n].y);
      }
      cacc += (log(S) + static_cast<double>(M)) - static_cast<double>(tgl[cb][n]);
    }
  };
  gload(0);
  sstore(0);
  __syncthreads();
  for (int c = 0; c < ntiles; ++c) {
    const int buf = c & 1;
    if (c + 1 < ntiles) gload(c + 1);
    int y[4];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
      const int qn = (16 * nb) / B, rn = 16 * nb - qn * B;   // wave-uniform
      int bn = yb + rn, tn = ytt + qn;
      if (bn >= B) {
        bn -= B;
        ++tn;
      }
      y[nb] = __builtin_amdgcn_raw_buffer_load_b8(bbuf, static_cast<uint32_t>(bn * T + tn + 1), 0, 0);
    }
    yb += r64;
    ytt += q64;
    if (yb >= B) {
      yb -= B;
      ++ytt;
    }
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
      uint4 bh[4], bl[4];
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        const int o = (nb * 16 + lr) * SW + 32 * kc + 8 * lg;
        bh[nb] = *reinterpret_cast<const uint4*>(ring + (buf * 2) * 64 * SW + o);
        bl[nb] = *reinterpret_cast<const uint4*>(ring + (buf * 2 + 1) * 64 * SW + o);
      }
      mfma3_batch<4>(wh[kc], wl[kc], bh, bl, acc);
    }
    // The previous tile's rows, while the products run: its partials (the
    // other parity) were written before the last barrier and are next
    // written in tile c + 1, behind the next barrier.
    if (c > 0) combine(c - 1);
    // Lane (lr, lg) holds the logits of vocabulary rows vbase .. +3 for tile
    // rows nb*16 + lr: reduce over the 4 lane groups; the lane holding a
    // row's target logit records it.
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
      float m = 0.0f, sum;
      if (shift) {
        m = group4_max(fmaxf(fmaxf(acc[nb][0], acc[nb][1]), fmaxf(acc[nb][2], acc[nb][3])));
        const float ml = -m * kLog2e;
        sum = group4_sum(
            ((exp2_f(__builtin_fmaf(acc[nb][0], kLog2e, ml)) + exp2_f(__builtin_fmaf(acc[nb][1], kLog2e, ml))) +
             exp2_f(__builtin_fmaf(acc[nb][2], kLog2e, ml))) +
            exp2_f(__builtin_fmaf(acc[nb][3], kLog2e, ml)));
      } else {
        sum = group4_sum(((exp2_f(acc[nb][0] * kLog2e) + exp2_f(acc[nb][1] * kLog2e)) + exp2_f(acc[nb][2] * kLog2e)) +
                         exp2_f(acc[nb][3] * kLog2e));
      }
      if (lg == 0) red[buf][wave][nb * 16 + lr] = make_float2(m, sum);
      const int yo = y[nb] - vbase;
      if (yo >= 0 && yo < 4) {
        float v = acc[nb][0];
#pragma unroll
        for (int r = 1; r < 4; ++r)
          if (yo == r) v = acc[nb][r];
        tgl[buf][nb * 16 + lr] = v;
      }
    }
    if (c + 1 < ntiles) sstore(buf ^ 1);
    __syncthreads();
  }
  combine(ntiles - 1);
  // The slot's total into its first tile partial, zeros in the others.
  if (wave < 4 && lane < 16) dsum[wave * 16 + lane] = cacc;
  __syncthreads();
  double* part = a.part + slot * a.row_tiles;
  if (threadIdx.x == 0) {
    double tot = 0.0;
    for (int n = 0; n < 64; ++n) tot += dsum[n];
    part[0] = tot;
  }
  for (int k = 1 + static_cast<int>(threadIdx.x); k < a.row_tiles; k += kHeadFusedThreads) part[k] = 0.0;
}

// ce of every row from the two vocabulary halves, summed per 64-row tile in
// fp64.  Grid: (row tiles, slots of the pass); 64 threads.
__global__ void k_ce_combine(FwdArgs a, const float2* hpart, const float* htgt) {
  __shared__ float ces[64];
  const int tile = blockIdx.x, ps = blockIdx.y;
  const int sg = ps & 1, pj = ps >> 1;
  const int e = pj / a.pcs, jl = pj % a.pcs;
  const int64_t slot = (static_cast<int64_t>(e) * a.PC + jl) * 2 + sg;
  const int64_t R = static_cast<int64_t>(a.T - 1) * a.B;
  const int64_t row = static_cast<int64_t>(tile) * 64 + threadIdx.x;
  float ce = 0.0f;
  if (row < R) {
    const float2 p0 = hpart[(slot * 2) * R + row], p1 = hpart[(slot * 2 + 1) * R + row];
    const float M = fmaxf(p0.x, p1.x);
    ce = __logf(p0.y * __expf(p0.x - M) + p1.y * __expf(p1.x - M)) + M - htgt[slot * R + row];
  }
  ces[threadIdx.x] = ce;
  __syncthreads();
  if (threadIdx.x == 0) {
    double tot = 0.0;
    for (int n = 0; n < 64; ++n) tot += static_cast<double>(ces[n]);
    a.part[slot * a.row_tiles + tile] = tot;
  }
}

// Zero n words (barrier counters and the abort flag before a persistent launch).
__global__ void k_zero_u32(unsigned* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

}  // namespace soma

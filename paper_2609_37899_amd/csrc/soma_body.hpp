// soma_body.hpp -- the paper's expert body on gfx950 (Section 3; Appendix C,
// Fig. arch): D pre-norm residual blocks of width d = 16 DW, each a bias-free
// LSTM sublayer and a bias-free GELU MLP (hidden 4d) behind gain-only
// LayerNorms, a final gain-only LayerNorm, and the frozen tied matrix E
// [256][d] that embeds the input byte and decodes logits = f E^T.
//
// At the paper's width (d = 32, D = 2) one perturbed body is 32k weights
// (128 KB) and E is 32 KB: together they fill the 160 KB LDS of one compute
// unit exactly.  So one block carries 64 sequences of one (expert, direction,
// sign) through all T-1 steps with every weight on chip: the probe is drawn
// once per block while the weights are written to LDS, and HBM sees only the
// input bytes and one loss sum per block.
//
// Matrix products.  The fp32 matrix instructions of gfx950 share their
// datapath with the vector ALU, and this kernel's vector work (LayerNorm,
// gate nonlinearities, GELU, softmax) is of the same order as its products,
// so on fp32 matrix cores the two would run back to back.  The products run
// instead on the fp16 matrix cores (V_MFMA_F32_16X16X32_F16), which execute
// alongside the vector ALU, with every fp32 operand split into two fp16
// parts, x = hi + lo (hi = x rounded toward zero to fp16, lo = the remainder
// rounded toward zero), and each product formed as
//   A B = A_lo B_hi + A_hi B_lo + A_hi B_hi   (the lo * lo term dropped),
// accumulated in fp32: about 21 significant bits per operand.  The weights
// are split once per block (hi and lo take the 4 bytes of the fp32 weight);
// the activations are split each step.
//
// Register layout.  Each wave owns 16 sequences (the MFMA columns).  A
// length-n activation vector of sequence c lives in lanes c, c+16, c+32,
// c+48: lane group g = lane / 16 holds elements 16 m + 4 g + i in register i
// of f32x4 number m -- the layout of an MFMA result block (rows
// 16 m .. 16 m + 15).  An fp16 MFMA contracts 32 K values, 8 per lane; K
// chunk p takes, in lane group g, the elements 32 p + 16 (j / 4) + 4 g + j % 4
// (j = 0..7), i.e. registers 0..3 of result blocks 2p and 2p+1.  With the
// weights' columns laid out in the same order, each product consumes the
// previous one's accumulators in place.  LayerNorm and softmax statistics
// are summed over the four lane groups with the permlane swaps (no LDS).
//
// LDS layout ("fragment order"): for output block mb and K chunk p, lane l
// reads the 8 weights W[16 mb + l % 16][col(p, l / 16, j)] as one 16-byte hi
// fragment and one 16-byte lo fragment, slot (mb * KC + p), 2 KB per slot.
// Per block l: the gate matrix [4d][2d] (columns [LN input | recurrent]),
// W1 [4d][d], W2 [d][4d]; then E [256][d].  K is zero-padded to 32 where a
// matrix has only 16 columns (d = 16).  The LayerNorm gains g1 and g2 are
// folded into the columns of the matrix that reads the normalised vector,
// W diag(g) n = W (g * n); the final gain multiplies f in registers.
#pragma once

#include "soma_kernels.hpp"

namespace soma {

constexpr int kBodyThreads = 256;   // 4 waves x 16 sequences
constexpr int kBodySeqs = 64;       // sequences per block
constexpr float kLnEps = 1e-5f;     // LayerNorm's variance offset

struct BodyArgs {
  const float* theta;     // [N][d]
  const uint8_t* bytes;   // [A][N][B][T] (perturbed) or [N][B][T] (evaluation)
  const uint64_t* seeds;  // [N]
  const float* E;         // tied matrix of expert e at E + e * e_stride, [256][dm] row-major
  int64_t e_stride;
  double* part;           // [slot][btiles] cross-entropy sums of each block
  float* fdec;            // evaluation: decoder inputs f [N][B][T-1][dm]
  float* lse;             // evaluation: log-sum-exp of the logits [N][B][T-1]
  int64_t d;              // parameters per expert
  uint64_t step;
  const float* eps_v;     // perturbation radius of expert e at eps_v[e * eps_stride]
  int eps_stride;
  int probe;              // probe law of the weights (gains: body_gain_law)
  int ppb;                // directions per accumulation batch
  int64_t bstride;        // bytes per accumulation batch, N B T
  int N, B, T, PC, pcs, j0, btiles;
  unsigned* err;          // the step's sticky abort flag (a weight out of the split's range sets kAbortRange)
};

// Ranges the split products need (kSplitMax per operand).  The normalised
// vector has |n_i| <= sqrt(d - 1) (zero mean, sum of squares <= d), so with
// every folded matrix weight (gains and gate scales folded in) at most
// kBodyWeightMax, a GELU input is at most kBodyWeightMax d = 8192 at d = 32,
// and with |g_f| <= kBodyGainMax the decoder input f = g_f n stays below
// 4096 sqrt(31) < 23000; h is bounded by 1.  A block that forms a weight
// outside these bounds (or NaN) aborts the step.
constexpr float kBodyWeightMax = 256.0f;
constexpr float kBodyGainMax = 4096.0f;

// Under the paper's sparse law the normalisation gains draw dense +-1
// (Appendix E); under the other laws they follow the weights.
__host__ __device__ constexpr int body_gain_law(int law) {
  return law == kProbeSparseRademacher ? kProbeRademacher : law;
}

// Canonical offsets of block l (d_b = 16 d^2 + 2 d parameters per block):
//   g1 [d] | W [4d][2d] | g2 [d] | W1 [4d][d] | W2 [d][4d];  g_f [d] after D blocks.
__host__ __device__ constexpr int64_t body_block(int64_t dm) { return 16 * dm * dm + 2 * dm; }

// Fragment slots (2 KB each: hi then lo) of one block and of E.
template <int DW, int D>
struct BodyLds {
  static constexpr int kGateKC = DW;                 // K = 2d in chunks of 32
  static constexpr int kW1KC = 1;                    // K = d (padded to 32 when d = 16)
  static constexpr int kW2KC = 2 * DW;               // K = 4d
  static constexpr int kGate = 4 * DW * kGateKC;     // output blocks x chunks
  static constexpr int kW1 = 4 * DW * kW1KC;
  static constexpr int kW2 = DW * kW2KC;
  static constexpr int kLayer = kGate + kW1 + kW2;
  static constexpr int kE = 16;                      // 256 rows, one chunk
  static constexpr int kSlots = D * kLayer + kE;
  static constexpr int kUint4 = kSlots * 128;        // 64 lanes x (hi, lo)
};

// theta[k4 .. k4+3] +- eps z (one rounding, as every other perturbed weight).
template <bool kPert>
__device__ __forceinline__ float4 body_weight4(const float* th, int64_t k4, int law, uint2 key, uint32_t pair,
                                               uint32_t step_lo, float seps) {
  const float4 t = *reinterpret_cast<const float4*>(th + k4);
  if (!kPert) return t;
  return fma4(seps, probe_quad(law, key, pair, step_lo, static_cast<uint64_t>(k4)), t);
}

// Sum and maximum over the four lanes l, l ^ 16, l ^ 32, l ^ 48 (the lane
// groups of one sequence).  Each swap pairs two copies of v, and the two
// results hold the two halves of the reduction, so that every lane ends
// with the same bits: (r0 + r2) + (r1 + r3) for lane rows r0 .. r3.
__device__ __forceinline__ float xsum4(float v) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(p[0]) + __uint_as_float(p[1]);
  const auto q = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(q[0]) + __uint_as_float(q[1]);
}

__device__ __forceinline__ float xmax4(float v) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
  const auto q = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(q[0]), __uint_as_float(q[1]));
}

// n = (x - mean) / sqrt(var + 1e-5) over the d = 16 DW features of each
// sequence (biased variance, two passes), without the gain.
template <int DW>
__device__ __forceinline__ void layer_norm0(const f32x4 (&x)[DW], f32x4 (&n)[DW]) {
  constexpr float kInvD = 1.0f / (16 * DW);
  float s = 0.0f;
#pragma unroll
  for (int m = 0; m < DW; ++m)
#pragma unroll
    for (int i = 0; i < 4; ++i) s += x[m][i];
  const float mu = xsum4(s) * kInvD;
  float q = 0.0f;
#pragma unroll
  for (int m = 0; m < DW; ++m)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      n[m][i] = x[m][i] - mu;
      q = __builtin_fmaf(n[m][i], n[m][i], q);
    }
  const float inv = __builtin_amdgcn_rsqf(__builtin_fmaf(xsum4(q), kInvD, kLnEps));
#pragma unroll
  for (int m = 0; m < DW; ++m)
#pragma unroll
    for (int i = 0; i < 4; ++i) n[m][i] *= inv;
}

// GELU(u) = u Phi(u) = max(u, 0) - |u| erfc(|u| / sqrt 2) / 2 (u erf(u / sqrt 2)
// is even in u), with erfc from Abramowitz & Stegun 7.1.26 (|error| <= 1.5e-7):
//   erfc(a) = t (a1 + t (a2 + t (a3 + t (a4 + t a5)))) e^{-a^2},
//   t = 1 / (1 + p a), a = |u| / sqrt 2 >= 0;
// the halving is folded into the coefficients and 1 / sqrt 2 into p and the
// exponent.
__device__ __forceinline__ float gelu_f(float u) {
  constexpr float kP = 0.3275911f * 0.70710678118654752f;
  constexpr float a1 = 0.5f * 0.254829592f, a2 = 0.5f * -0.284496736f, a3 = 0.5f * 1.421413741f,
                  a4 = 0.5f * -1.453152027f, a5 = 0.5f * 1.061405429f;
  constexpr float kE = -0.5f * kLog2e;                  // e^{-u^2/2} = 2^{kE u^2}
  const float au = __builtin_fabsf(u);
  const float t = __builtin_amdgcn_rcpf(__builtin_fmaf(kP, au, 1.0f));
  float q = __builtin_fmaf(t, a5, a4);
  q = __builtin_fmaf(t, q, a3);
  q = __builtin_fmaf(t, q, a2);
  q = __builtin_fmaf(t, q, a1);
  const float tail = q * t * __builtin_amdgcn_exp2f((u * u) * kE);   // erfc(a) / 2
  return __builtin_fmaf(-au, tail, fmaxf(u, 0.0f));
}

// The gate rows are stored pre-scaled so that each nonlinearity needs one
// exp2: sigmoid(a) = 1 / (1 + 2^{-a log2 e}) for i, f, o and
// tanh(a) = 1 - 2 / (2^{2 a log2 e} + 1) for g.
constexpr float kGateScaleSig = -kLog2e;
constexpr float kGateScaleTanh = 2.0f * kLog2e;

__device__ __forceinline__ float sigmoid_pre(float a) { return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(a)); }
__device__ __forceinline__ float tanh_pre(float a) {
  return __builtin_fmaf(-2.0f, __builtin_amdgcn_rcpf(__builtin_amdgcn_exp2f(a) + 1.0f), 1.0f);
}

// An LDS offset the compiler cannot see through.  The weights do not change
// inside the time loop, so without this every LDS read of the loop
// (hundreds of registers' worth) would be hoisted out of it and spilled.
__device__ __forceinline__ int opaque_offset(int off) {
  asm volatile("" : "+s"(off));
  return off;
}

// The 8 K values of a lane for one chunk: registers 0..3 of blocks a and b.
__device__ __forceinline__ void split8(const f32x4& a, const f32x4& b, h8& hi, h8& lo) {
  uint4 H, L;
  split2(a[0], a[1], H.x, L.x);
  split2(a[2], a[3], H.y, L.y);
  split2(b[0], b[1], H.z, L.z);
  split2(b[2], b[3], H.w, L.w);
  hi = __builtin_bit_cast(h8, H);
  lo = __builtin_bit_cast(h8, L);
}

// acc += A B over one K chunk, A from LDS slot `slot` (hi, lo), B split.
__device__ __forceinline__ f32x4 mfma_split(const uint4* w16, int slot, int lane, const h8& bh, const h8& bl,
                                            f32x4 acc) {
  const h8 ah = __builtin_bit_cast(h8, w16[slot * 128 + lane]);
  const h8 al = __builtin_bit_cast(h8, w16[slot * 128 + 64 + lane]);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(al, bh, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, bl, acc, 0, 0, 0);
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, bh, acc, 0, 0, 0);
}

// Expert e's batch for direction j0 + jl (its accumulation batch).
__device__ __forceinline__ const uint8_t* bytes_of_body(const BodyArgs& a, int e, int jl) {
  return a.bytes + static_cast<int64_t>((a.j0 + jl) / a.ppb) * a.bstride + static_cast<int64_t>(e) * a.B * a.T;
}

// One residual block for one time step of a wave's 16 sequences:
//   x <- x + h,  h = LSTM(LN(x), h)    (the gains folded into the weights)
//   x <- x + W2 GELU(W1 LN(x)).
// W points at the block's first slot.  With act false the recurrent state
// is left as it was (the pipeline's fill steps, whose results are discarded).
template <int DW>
__device__ __forceinline__ void body_block_step(const uint4* w16, int s0, int lane, f32x4 (&x)[DW], f32x4 (&h)[DW],
                                                f32x4 (&c)[DW], bool act) {
  using Lds = BodyLds<DW, 1>;
  const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
  f32x4 n[DW];
  layer_norm0<DW>(x, n);
  // K of the gate matrix: [n | h], 2 DW blocks, chunk p = blocks 2p, 2p+1.
  f32x4 kin[2 * DW];
#pragma unroll
  for (int m = 0; m < DW; ++m) {
    kin[m] = n[m];
    kin[DW + m] = h[m];
  }
  f32x4 acc[4 * DW];
#pragma unroll
  for (int mb = 0; mb < 4 * DW; ++mb) acc[mb] = zero;
#pragma unroll
  for (int p = 0; p < Lds::kGateKC; ++p) {
    h8 bh, bl;
    split8(kin[2 * p], kin[2 * p + 1], bh, bl);
#pragma unroll
    for (int mb = 0; mb < 4 * DW; ++mb) acc[mb] = mfma_split(w16, s0 + mb * Lds::kGateKC + p, lane, bh, bl, acc[mb]);
  }
  // Unit 16 m + 4 g + i has gate q in block q DW + m, register i.
#pragma unroll
  for (int m = 0; m < DW; ++m)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float ig = sigmoid_pre(acc[m][i]), fg = sigmoid_pre(acc[DW + m][i]);
      const float gg = tanh_pre(acc[2 * DW + m][i]), og = sigmoid_pre(acc[3 * DW + m][i]);
      const float c1 = __builtin_fmaf(fg, c[m][i], ig * gg);
      const float h1 = og * tanh_pre(c1 * kGateScaleTanh);
      c[m][i] = act ? c1 : c[m][i];
      h[m][i] = act ? h1 : h[m][i];
      x[m][i] += h1;
    }
  layer_norm0<DW>(x, n);
  f32x4 u[4 * DW];
#pragma unroll
  for (int mb = 0; mb < 4 * DW; ++mb) u[mb] = zero;
  {
    h8 bh, bl;
    split8(n[0], DW > 1 ? n[DW - 1] : zero, bh, bl);
    const int s1 = s0 + Lds::kGate;
#pragma unroll
    for (int mb = 0; mb < 4 * DW; ++mb) u[mb] = mfma_split(w16, s1 + mb, lane, bh, bl, u[mb]);
  }
#pragma unroll
  for (int mb = 0; mb < 4 * DW; ++mb)
#pragma unroll
    for (int i = 0; i < 4; ++i) u[mb][i] = gelu_f(u[mb][i]);
  const int s2 = s0 + Lds::kGate + Lds::kW1;
#pragma unroll
  for (int p = 0; p < Lds::kW2KC; ++p) {
    h8 bh, bl;
    split8(u[2 * p], u[2 * p + 1], bh, bl);
#pragma unroll
    for (int mb = 0; mb < DW; ++mb) x[mb] = mfma_split(w16, s2 + mb * Lds::kW2KC + p, lane, bh, bl, x[mb]);
  }
}

// The decoder for one time step: f = g_f * LN(x), logits = E f; returns the
// cross entropy against the target whose E row (this lane's features) is
// ey, and the log-sum-exp and f for the delta rule.
template <int DW>
__device__ __forceinline__ float body_decode_step(const uint4* w16, int se0, int lane, const f32x4 (&x)[DW],
                                                  const f32x4 (&gf)[DW], const float4 (&ey)[DW], f32x4 (&f)[DW],
                                                  float& lse) {
  const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
  layer_norm0<DW>(x, f);
#pragma unroll
  for (int m = 0; m < DW; ++m)
#pragma unroll
    for (int i = 0; i < 4; ++i) f[m][i] *= gf[m][i];
  h8 bh, bl;
  split8(f[0], DW > 1 ? f[DW - 1] : zero, bh, bl);
  f32x4 lo[16];
#pragma unroll
  for (int mb = 0; mb < 16; ++mb) lo[mb] = mfma_split(w16, se0 + mb, lane, bh, bl, zero);
  float mx = lo[0][0];
#pragma unroll
  for (int mb = 0; mb < 16; ++mb)
#pragma unroll
    for (int i = 0; i < 4; ++i) mx = fmaxf(mx, lo[mb][i]);
  mx = xmax4(mx);
  const float ms = mx * kLog2e;
  float se = 0.0f;
#pragma unroll
  for (int mb = 0; mb < 16; ++mb)
#pragma unroll
    for (int i = 0; i < 4; ++i) se += __builtin_amdgcn_exp2f(__builtin_fmaf(lo[mb][i], kLog2e, -ms));
  lse = __logf(xsum4(se)) + mx;
  float yl = 0.0f;
#pragma unroll
  for (int m = 0; m < DW; ++m) {
    yl = __builtin_fmaf(ey[m].x, f[m][0], yl);
    yl = __builtin_fmaf(ey[m].y, f[m][1], yl);
    yl = __builtin_fmaf(ey[m].z, f[m][2], yl);
    yl = __builtin_fmaf(ey[m].w, f[m][3], yl);
  }
  return lse - xsum4(yl);
}

// One weight fragment: lane `ln` of slot (mb, p) of a matrix with row stride
// `ld` (floats) and `ncol` columns, starting at canonical offset `base`;
// columns col(p, g, j) = 32 p + 16 (j / 4) + 4 g + j % 4 beyond ncol are zero.
// Columns below `gcol` are multiplied by the gain at canonical offset kg +
// column; the row's scale is applied; the fp32 weight is then split into
// (hi, lo).
template <bool kPert>
__device__ __forceinline__ void body_fragment(const float* th, int64_t base, int ld, int ncol, int row, int p,
                                              int ln, int64_t kg, int gcol, float scale, int wlaw, int glaw,
                                              uint2 key, uint32_t pair, uint32_t step_lo, float seps, uint4& hi,
                                              uint4& lo, float bound, bool& in_range) {
  float w[8];
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    const int c0 = 32 * p + 16 * half + 4 * (ln >> 4);
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (c0 < ncol) {
      v = body_weight4<kPert>(th, base + static_cast<int64_t>(row) * ld + c0, wlaw, key, pair, step_lo, seps);
      if (c0 < gcol) {
        const float4 g = body_weight4<kPert>(th, kg + c0, glaw, key, pair, step_lo, seps);
        v = make_float4(v.x * g.x, v.y * g.y, v.z * g.z, v.w * g.w);
      }
      v = make_float4(v.x * scale, v.y * scale, v.z * scale, v.w * scale);
      in_range &= split_range_ok(v, bound);
    }
    w[4 * half] = v.x;
    w[4 * half + 1] = v.y;
    w[4 * half + 2] = v.z;
    w[4 * half + 3] = v.w;
  }
  split2(w[0], w[1], hi.x, lo.x);
  split2(w[2], w[3], hi.y, lo.y);
  split2(w[4], w[5], hi.z, lo.z);
  split2(w[6], w[7], hi.w, lo.w);
}

// ---------------------------------------------------------------------------
// The fused body: one block per (64-sequence tile, expert, direction, sign)
// (one per (tile, expert) in evaluation).  Each sequence's loss is the sum
// of its T-1 next-byte cross entropies; the block writes their fp64 sum to
// part[slot][tile].  Evaluation also writes the decoder inputs f and the
// log-sum-exp of every position (the inputs of the delta rule).
//
// The time loop is pipelined over the D + 1 stages (block 1, ..., block D,
// decoder): iteration i runs block l on step i - l and the decoder on step
// i - D, each on what the stage before it produced in iteration i - 1.  The
// stages of one iteration are independent, so the matrix products of one
// can run on the matrix cores while the vector ALU works on another.  The
// first D iterations fill the pipeline and the last D drain it; their extra
// results are discarded.
// ---------------------------------------------------------------------------
template <int DW, int D, bool kPert>
__global__ __launch_bounds__(kBodyThreads, 1) void k_body(BodyArgs a) {
  using Lds = BodyLds<DW, D>;
  constexpr int dm = 16 * DW;
  constexpr int NS = kPert ? 2 : 1;
  __shared__ uint4 w16[Lds::kUint4];

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, col = lane & 15, lg = lane >> 4;
  const int bt = blockIdx.x % a.btiles;
  const int sp = blockIdx.x / a.btiles;
  const int s = sp % NS, pj = sp / NS;
  const int e = pj / a.pcs, jl = pj % a.pcs;
  const float* th = a.theta + static_cast<int64_t>(e) * a.d;
  const float* Ee = a.E + static_cast<int64_t>(e) * a.e_stride;
  const uint2 key = kPert ? stream_key(a.seeds[e], a.step) : make_uint2(0u, 0u);
  const uint32_t pair = static_cast<uint32_t>(a.j0 + jl), step_lo = static_cast<uint32_t>(a.step);
  const float eps = kPert ? a.eps_v[static_cast<int64_t>(e) * a.eps_stride] : 0.0f;
  const float seps = s == 0 ? eps : -eps;
  const int wlaw = a.probe, glaw = body_gain_law(a.probe);
  constexpr int64_t blk = body_block(dm);

  // Perturbed weights into LDS as split fragments, gains folded in, gate
  // rows pre-scaled for their nonlinearity.  One (slot, lane) per iteration.
  bool in_range = true;
  for (int q = threadIdx.x; q < Lds::kSlots * 64; q += kBodyThreads) {
    const int slot = q >> 6, ln = q & 63, r16 = ln & 15;
    uint4 hi, lo;
    if (slot < D * Lds::kLayer) {
      const int l = slot / Lds::kLayer, r = slot % Lds::kLayer;
      const int64_t base = l * blk;
      if (r < Lds::kGate) {
        // columns [0, d) read LN(x) (gain g1), [d, 2d) the recurrent state
        const int mb = r / Lds::kGateKC, p = r % Lds::kGateKC, row = 16 * mb + r16;
        const float scale = row / dm == 2 ? kGateScaleTanh : kGateScaleSig;
        body_fragment<kPert>(th, base + dm, 2 * dm, 2 * dm, row, p, ln, base, dm, scale, wlaw, glaw, key, pair,
                             step_lo, seps, hi, lo, kBodyWeightMax, in_range);
      } else if (r < Lds::kGate + Lds::kW1) {
        const int mb = r - Lds::kGate, row = 16 * mb + r16;
        body_fragment<kPert>(th, base + 2 * dm + 8 * dm * dm, dm, dm, row, 0, ln, base + dm + 8 * dm * dm, dm, 1.0f,
                             wlaw, glaw, key, pair, step_lo, seps, hi, lo, kBodyWeightMax, in_range);
      } else {
        const int rr = r - Lds::kGate - Lds::kW1, mb = rr / Lds::kW2KC, p = rr % Lds::kW2KC, row = 16 * mb + r16;
        body_fragment<kPert>(th, base + 2 * dm + 12 * dm * dm, 4 * dm, 4 * dm, row, p, ln, 0, 0, 1.0f, wlaw, glaw,
                             key, pair, step_lo, seps, hi, lo, kBodyWeightMax, in_range);
      }
    } else {
      // E (frozen, not perturbed): rows 16 mb + r16, columns as above.
      const int mb = slot - D * Lds::kLayer, row = 16 * mb + r16;
      body_fragment<false>(Ee, 0, dm, dm, row, 0, ln, 0, 0, 1.0f, 0, 0, key, pair, step_lo, 0.0f, hi, lo, kSplitMax,
                           in_range);
    }
    w16[slot * 128 + ln] = hi;
    w16[slot * 128 + 64 + ln] = lo;
  }
  f32x4 gf[DW];
#pragma unroll
  for (int m = 0; m < DW; ++m) {
    const float4 g = body_weight4<kPert>(th, D * blk + 16 * m + 4 * lg, glaw, key, pair, step_lo, seps);
    in_range &= split_range_ok(g, kBodyGainMax);
    gf[m] = f32x4{g.x, g.y, g.z, g.w};
  }
  report_split_range(a.err, in_range);
  __syncthreads();

  const int B = a.B, T = a.T;
  const int b_raw = bt * kBodySeqs + wave * 16 + col;
  const bool live = bt * kBodySeqs + wave * 16 < B;   // wave-uniform
  const bool valid = b_raw < B;
  const int b = valid ? b_raw : B - 1;
  const uint8_t* seq = kPert ? bytes_of_body(a, e, jl) + static_cast<int64_t>(b) * T
                             : a.bytes + (static_cast<int64_t>(e) * B + b) * T;
  double ce_sum = 0.0;
  if (live) {
    f32x4 h[D][DW], cs[D][DW], xs[D + 1][DW];   // xs[l]: the input of stage l this iteration
#pragma unroll
    for (int l = 0; l < D; ++l)
#pragma unroll
      for (int m = 0; m < DW; ++m) h[l][m] = cs[l][m] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int l = 0; l <= D; ++l)
#pragma unroll
      for (int m = 0; m < DW; ++m) xs[l][m] = f32x4{0.f, 0.f, 0.f, 0.f};
    // rows[k] = E[byte_{i-k}] (this lane's features); the decoder's target at
    // iteration i is byte_{i-D+1}, i.e. rows[D-1].
    float4 rows[D][DW];
    {
      const int v0 = seq[0];
#pragma unroll
      for (int m = 0; m < DW; ++m) rows[0][m] = *reinterpret_cast<const float4*>(Ee + v0 * dm + 16 * m + 4 * lg);
#pragma unroll
      for (int k = 1; k < D; ++k)
#pragma unroll
        for (int m = 0; m < DW; ++m) rows[k][m] = rows[0][m];
    }
    int vnext = seq[1 < T - 1 ? 1 : T - 1];
    for (int i = 0; i < T - 1 + D; ++i) {
      // Prefetch: the byte after next, and the E row of the next byte.
      const int vnn = seq[i + 2 < T - 1 ? i + 2 : T - 1];
      float4 rnext[DW];
#pragma unroll
      for (int m = 0; m < DW; ++m) rnext[m] = *reinterpret_cast<const float4*>(Ee + vnext * dm + 16 * m + 4 * lg);
      const uint4* W = w16 + opaque_offset(0);
#pragma unroll
      for (int m = 0; m < DW; ++m) xs[0][m] = f32x4{rows[0][m].x, rows[0][m].y, rows[0][m].z, rows[0][m].w};

      f32x4 out[D][DW];
#pragma unroll
      for (int l = 0; l < D; ++l) {
#pragma unroll
        for (int m = 0; m < DW; ++m) out[l][m] = xs[l][m];
        body_block_step<DW>(W, l * Lds::kLayer, lane, out[l], h[l], cs[l], i >= l);
      }
      f32x4 f[DW];
      float lse;
      const float ce = body_decode_step<DW>(W, D * Lds::kLayer, lane, xs[D], gf, rows[D - 1], f, lse);
      const int td = i - D;                       // the decoder's time step
      const bool scored = td >= 0 && td + 1 < T;
      ce_sum += (scored && valid && lg == 0) ? static_cast<double>(ce) : 0.0;
      if (!kPert && scored && valid) {
        const int64_t pos = (static_cast<int64_t>(e) * B + b) * (T - 1) + td;
#pragma unroll
        for (int m = 0; m < DW; ++m)
          *reinterpret_cast<float4*>(a.fdec + pos * dm + 16 * m + 4 * lg) = make_float4(f[m][0], f[m][1], f[m][2], f[m][3]);
        if (lg == 0) a.lse[pos] = lse;
      }
#pragma unroll
      for (int l = 0; l < D; ++l)
#pragma unroll
        for (int m = 0; m < DW; ++m) xs[l + 1][m] = out[l][m];
#pragma unroll
      for (int k = D - 1; k > 0; --k)
#pragma unroll
        for (int m = 0; m < DW; ++m) rows[k][m] = rows[k - 1][m];
#pragma unroll
      for (int m = 0; m < DW; ++m) rows[0][m] = rnext[m];
      vnext = vnn;
    }
  }

  // Per-block sum of the 64 sequence losses in a fixed order.
  __syncthreads();   // every wave is past its loop: the weight region is free
  double* red = reinterpret_cast<double*>(w16);
  if (lg == 0) red[wave * 16 + col] = ce_sum;
  __syncthreads();
  if (threadIdx.x == 0) {
    double tot = 0.0;
    for (int i = 0; i < kBodySeqs; ++i) tot += red[i];
    a.part[((static_cast<int64_t>(e) * a.PC + jl) * NS + s) * a.btiles + bt] = tot;
  }
}

// ---------------------------------------------------------------------------
// The decoder-path delta rule (Appendix E, Eq. delta) from an evaluation
// pass's decoder inputs f and log-sum-exps:
//   G[v][k] = sum_r (exp(E_v . f_r - lse_r) - [y_r = v]) f_r[k],
// one partial per chunk of kDeltaChunk positions (r = b (T-1) + t): thread v
// keeps row v of E and of G in registers; f is staged through LDS.
// ---------------------------------------------------------------------------
constexpr int kDeltaChunk = 1024;
constexpr int kDeltaStage = 256;

template <int DW>
__global__ __launch_bounds__(256) void k_head_delta_part(const float* fdec, const float* lse, const uint8_t* bytes,
                                                         const float* E, int64_t e_stride, int B, int T,
                                                         int chunks, float* dpart) {
  constexpr int dm = 16 * DW;
  __shared__ float fs[kDeltaStage][dm];
  __shared__ float ls[kDeltaStage];
  __shared__ int ys[kDeltaStage];
  const int e = blockIdx.y, chunk = blockIdx.x, v = threadIdx.x;
  const int64_t R = static_cast<int64_t>(B) * (T - 1);
  const float* Ee = E + static_cast<int64_t>(e) * e_stride;
  float ev[dm], G[dm];
#pragma unroll
  for (int k = 0; k < dm; ++k) {
    ev[k] = Ee[v * dm + k];
    G[k] = 0.0f;
  }
  for (int s0 = 0; s0 < kDeltaChunk; s0 += kDeltaStage) {
    const int64_t r0 = static_cast<int64_t>(chunk) * kDeltaChunk + s0;
    if (r0 >= R) break;
    const int n = static_cast<int>(R - r0 < kDeltaStage ? R - r0 : kDeltaStage);
    __syncthreads();
    for (int i = threadIdx.x; i < n * dm; i += 256)
      fs[i / dm][i % dm] = fdec[(static_cast<int64_t>(e) * R + r0) * dm + i];
    if (static_cast<int>(threadIdx.x) < n) {
      const int64_t r = r0 + threadIdx.x;
      const int64_t bb = r / (T - 1), tt = r % (T - 1);
      ls[threadIdx.x] = lse[static_cast<int64_t>(e) * R + r];
      ys[threadIdx.x] = bytes[(static_cast<int64_t>(e) * B + bb) * T + tt + 1];
    }
    __syncthreads();
    for (int p = 0; p < n; ++p) {
      float lgt = 0.0f;
#pragma unroll
      for (int k = 0; k < dm; ++k) lgt = __builtin_fmaf(ev[k], fs[p][k], lgt);
      const float pv = __expf(lgt - ls[p]) - (ys[p] == v ? 1.0f : 0.0f);
#pragma unroll
      for (int k = 0; k < dm; ++k) G[k] = __builtin_fmaf(pv, fs[p][k], G[k]);
    }
  }
  float* out = dpart + ((static_cast<int64_t>(e) * chunks + chunk) * kVocab + v) * dm;
#pragma unroll
  for (int k = 0; k < dm; k += 4) *reinterpret_cast<float4*>(out + k) = make_float4(G[k], G[k + 1], G[k + 2], G[k + 3]);
}

// grad[e][i] = (sum over chunks in order, fp64) / (B (T-1)); with lr != 0
// also E[e][i] -= lr grad (the caller's tied matrix, one expert per e).
__global__ void k_head_delta_reduce(const float* dpart, int chunks, int64_t vd, double inv_rows, float* grad,
                                    float* E, int64_t e_stride, float lr) {
  const int e = blockIdx.y;
  const int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x;
  if (i >= vd) return;
  double acc = 0.0;
  for (int c = 0; c < chunks; ++c) acc += static_cast<double>(dpart[(static_cast<int64_t>(e) * chunks + c) * vd + i]);
  const float gr = static_cast<float>(acc * inv_rows);
  if (grad) grad[static_cast<int64_t>(e) * vd + i] = gr;
  if (lr != 0.0f) {
    float* p = E + static_cast<int64_t>(e) * e_stride + i;
    *p = __builtin_fmaf(-lr, gr, *p);
  }
}

}  // namespace soma

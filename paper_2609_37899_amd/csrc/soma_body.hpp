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
// Register layout.  Each wave owns 16 sequences (MFMA columns).  A length-n
// activation vector of sequence c lives in lanes c, c+16, c+32, c+48: lane
// group g = lane / 16 holds elements 16 m + 4 g + i in register i of f32x4
// number m.  That is exactly the layout of a V_MFMA_F32_16X16X4_F32 result
// block (rows 16 m .. 16 m + 15), and it is also a valid B operand when the
// K index of MFMA (m, i) is taken as 16 m + 4 g + i: every product below
// consumes the previous one's accumulators in place, with no data movement.
// LayerNorm and softmax statistics are summed over the four lane groups with
// the permlane swaps (no LDS).
//
// LDS layout ("fragment order"): the A operand of MFMA (mb, m, i) for lane l
// is W[16 mb + l % 16][16 m + 4 (l / 16) + i]; the four i of one (mb, m, l)
// are one float4 at slot (mb * KM + m) * 64 + l, KM = K / 16, so a wave
// reads one conflict-free b128 per four MFMAs.  Per block l:
//   gate matrix [4d][2d]  (columns [LN input | recurrent]), 512 DW^2 slots
//   W1 [4d][d]                                             , 256 DW^2 slots
//   W2 [d][4d]                                             , 256 DW^2 slots
// then E [256][d] (1024 DW slots).  The LayerNorm gains g1 and g2 are folded
// into the columns of the matrix that reads the normalised vector,
// W diag(g) n = W (g * n); the final gain multiplies f in registers.
#pragma once

#include "soma_kernels.hpp"

namespace soma {

constexpr int kBodyThreads = 256;   // 4 waves x 16 sequences
constexpr int kBodySeqs = 64;       // sequences per block
constexpr float kLnEps = 1e-5f;     // LayerNorm's variance offset
constexpr float kLog2e = 1.4426950408889634f;

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
};

// Under the paper's sparse law the normalisation gains draw dense +-1
// (Appendix E); under the other laws they follow the weights.
__host__ __device__ constexpr int body_gain_law(int law) {
  return law == kProbeSparseRademacher ? kProbeRademacher : law;
}

// Canonical offsets of block l (d_b = 16 d^2 + 2 d parameters per block):
//   g1 [d] | W [4d][2d] | g2 [d] | W1 [4d][d] | W2 [d][4d];  g_f [d] after D blocks.
__host__ __device__ constexpr int64_t body_block(int64_t dm) { return 16 * dm * dm + 2 * dm; }

template <int DW, int D>
struct BodyLds {
  static constexpr int kGate = 512 * DW * DW;
  static constexpr int kW1 = 256 * DW * DW;
  static constexpr int kW2 = 256 * DW * DW;
  static constexpr int kLayer = kGate + kW1 + kW2;
  static constexpr int kE = 1024 * DW;
  static constexpr int kTotal = D * kLayer + kE;   // float4 slots
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

// GELU(u) = u Phi(u), Phi(u) = (1 + erf(u / sqrt 2)) / 2, with erf from
// Abramowitz & Stegun 7.1.26 (|error| <= 1.5e-7 on erf):
//   1 - erf(a) = t (a1 + t (a2 + t (a3 + t (a4 + t a5)))) e^{-a^2},
//   t = 1 / (1 + p a), a >= 0.
__device__ __forceinline__ float gelu_f(float u) {
  constexpr float p = 0.3275911f, a1 = 0.254829592f, a2 = -0.284496736f, a3 = 1.421413741f,
                  a4 = -1.453152027f, a5 = 1.061405429f;
  const float a = __builtin_fabsf(u) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(__builtin_fmaf(p, a, 1.0f));
  float poly = __builtin_fmaf(t, a5, a4);
  poly = __builtin_fmaf(t, poly, a3);
  poly = __builtin_fmaf(t, poly, a2);
  poly = __builtin_fmaf(t, poly, a1);
  poly *= t;
  const float tail = 0.5f * poly * __builtin_amdgcn_exp2f(-(a * a) * kLog2e);   // (1 - erf(a)) / 2
  return u * (u >= 0.0f ? 1.0f - tail : tail);
}

// An LDS slot offset the compiler cannot see through.  The weights do not
// change inside the time loop, so without this every LDS read of the step
// (hundreds of registers' worth) would be hoisted out of the loop and
// spilled; laundering the offset once per sublayer keeps each read next to
// its MFMAs.
__device__ __forceinline__ int opaque_offset(int off) {
  asm volatile("" : "+s"(off));
  return off;
}

// acc += A(float4 along the four MFMAs of one (mb, m)) . B(f32x4).
__device__ __forceinline__ f32x4 mfma_frag(const float4& a, const f32x4& b, f32x4 acc) {
  acc = mfma4(a.x, b[0], acc);
  acc = mfma4(a.y, b[1], acc);
  acc = mfma4(a.z, b[2], acc);
  acc = mfma4(a.w, b[3], acc);
  return acc;
}

// Expert e's batch for direction j0 + jl (its accumulation batch).
__device__ __forceinline__ const uint8_t* bytes_of_body(const BodyArgs& a, int e, int jl) {
  return a.bytes + static_cast<int64_t>((a.j0 + jl) / a.ppb) * a.bstride + static_cast<int64_t>(e) * a.B * a.T;
}

// ---------------------------------------------------------------------------
// The fused body: one block per (64-sequence tile, expert, direction, sign)
// (one per (tile, expert) in evaluation).  Each sequence's loss is the sum
// of its T-1 next-byte cross entropies; the block writes their fp64 sum to
// part[slot][tile].  Evaluation also writes the decoder inputs f and the
// log-sum-exp of every position (the inputs of the delta rule).
// ---------------------------------------------------------------------------
template <int DW, int D, bool kPert>
__global__ __launch_bounds__(kBodyThreads, 1) void k_body(BodyArgs a) {
  using Lds = BodyLds<DW, D>;
  constexpr int dm = 16 * DW;
  constexpr int NS = kPert ? 2 : 1;
  __shared__ float4 w4[Lds::kTotal];

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

  // Perturbed weights into LDS in fragment order, gains folded in.
  for (int q = threadIdx.x; q < D * Lds::kLayer; q += kBodyThreads) {
    const int l = q / Lds::kLayer, r = q % Lds::kLayer, ln = r & 63;
    const int64_t base = l * blk;
    int64_t k, kg = -1;
    if (r < Lds::kGate) {
      const int mb = r / (128 * DW), m = (r >> 6) % (2 * DW);
      const int row = 16 * mb + (ln & 15), c0 = 16 * m + 4 * (ln >> 4);
      k = base + dm + static_cast<int64_t>(row) * 2 * dm + c0;
      if (m < DW) kg = base + c0;                                       // g1 on the LN input
    } else if (r < Lds::kGate + Lds::kW1) {
      const int rr = r - Lds::kGate, mb = rr / (64 * DW), m = (rr >> 6) % DW;
      const int row = 16 * mb + (ln & 15), c0 = 16 * m + 4 * (ln >> 4);
      k = base + 2 * dm + 8 * dm * dm + static_cast<int64_t>(row) * dm + c0;
      kg = base + dm + 8 * dm * dm + c0;                                 // g2
    } else {
      const int rr = r - Lds::kGate - Lds::kW1, mb = rr / (256 * DW), m = (rr >> 6) % (4 * DW);
      const int row = 16 * mb + (ln & 15), c0 = 16 * m + 4 * (ln >> 4);
      k = base + 2 * dm + 12 * dm * dm + static_cast<int64_t>(row) * 4 * dm + c0;
    }
    float4 w = body_weight4<kPert>(th, k, wlaw, key, pair, step_lo, seps);
    if (kg >= 0) {
      const float4 g = body_weight4<kPert>(th, kg, glaw, key, pair, step_lo, seps);
      w = make_float4(w.x * g.x, w.y * g.y, w.z * g.z, w.w * g.w);
    }
    w4[q] = w;
  }
  for (int q = threadIdx.x; q < Lds::kE; q += kBodyThreads) {
    const int ln = q & 63, m = (q >> 6) % DW, mb = q / (64 * DW);
    w4[D * Lds::kLayer + q] =
        *reinterpret_cast<const float4*>(Ee + (16 * mb + (ln & 15)) * dm + 16 * m + 4 * (ln >> 4));
  }
  f32x4 gf[DW];
#pragma unroll
  for (int m = 0; m < DW; ++m) {
    const float4 g = body_weight4<kPert>(th, D * blk + 16 * m + 4 * lg, glaw, key, pair, step_lo, seps);
    gf[m] = f32x4{g.x, g.y, g.z, g.w};
  }
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
    f32x4 h[D][DW], cs[D][DW];
#pragma unroll
    for (int l = 0; l < D; ++l)
#pragma unroll
      for (int m = 0; m < DW; ++m) h[l][m] = cs[l][m] = f32x4{0.f, 0.f, 0.f, 0.f};
    float4 er[DW];   // E row of the current input byte, this lane's features
    {
      const int v = seq[0];
#pragma unroll
      for (int m = 0; m < DW; ++m) er[m] = *reinterpret_cast<const float4*>(Ee + v * dm + 16 * m + 4 * lg);
    }
    for (int t = 0; t + 1 < T; ++t) {
      const int y = seq[t + 1];
      float4 ey[DW];   // E row of the target: its logit now, the next input's embedding after
#pragma unroll
      for (int m = 0; m < DW; ++m) ey[m] = *reinterpret_cast<const float4*>(Ee + y * dm + 16 * m + 4 * lg);
      f32x4 x[DW];
#pragma unroll
      for (int m = 0; m < DW; ++m) x[m] = f32x4{er[m].x, er[m].y, er[m].z, er[m].w};

#pragma unroll
      for (int l = 0; l < D; ++l) {
        const float4* Wg = w4 + opaque_offset(l * Lds::kLayer);
        f32x4 n[DW];
        layer_norm0<DW>(x, n);
        // LSTM sublayer: gate pre-activations W' [n; h] (rows i, f, g, o).
        f32x4 acc[4 * DW];
#pragma unroll
        for (int mb = 0; mb < 4 * DW; ++mb) acc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int m = 0; m < 2 * DW; ++m) {
          const f32x4 bv = m < DW ? n[m] : h[l][m - DW];
#pragma unroll
          for (int mb = 0; mb < 4 * DW; ++mb) acc[mb] = mfma_frag(Wg[(mb * 2 * DW + m) * 64 + lane], bv, acc[mb]);
        }
        // Unit 16 m + 4 g + i has gate q in block q DW + m, register i.
#pragma unroll
        for (int m = 0; m < DW; ++m)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float ig = sigmoid_f(acc[m][i]), fg = sigmoid_f(acc[DW + m][i]);
            const float gg = tanh_f(acc[2 * DW + m][i]), og = sigmoid_f(acc[3 * DW + m][i]);
            const float c1 = __builtin_fmaf(fg, cs[l][m][i], ig * gg);
            cs[l][m][i] = c1;
            h[l][m][i] = og * tanh_f(c1);
            x[m][i] += h[l][m][i];
          }
        // MLP sublayer: x += W2 GELU(W1' LN(x)), the residual as W2's accumulator.
        layer_norm0<DW>(x, n);
        const float4* W1 = w4 + opaque_offset(l * Lds::kLayer + Lds::kGate);
        const float4* W2 = W1 + Lds::kW1;
        f32x4 u[4 * DW];
#pragma unroll
        for (int mb = 0; mb < 4 * DW; ++mb) u[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int m = 0; m < DW; ++m)
#pragma unroll
          for (int mb = 0; mb < 4 * DW; ++mb) u[mb] = mfma_frag(W1[(mb * DW + m) * 64 + lane], n[m], u[mb]);
#pragma unroll
        for (int mb = 0; mb < 4 * DW; ++mb)
#pragma unroll
          for (int i = 0; i < 4; ++i) u[mb][i] = gelu_f(u[mb][i]);
#pragma unroll
        for (int m = 0; m < 4 * DW; ++m)
#pragma unroll
          for (int mb = 0; mb < DW; ++mb) x[mb] = mfma_frag(W2[(mb * 4 * DW + m) * 64 + lane], u[m], x[mb]);
      }

      // Decoder: f = g_f * LN(x), logits = E f, cross entropy against y.
      f32x4 f[DW];
      layer_norm0<DW>(x, f);
#pragma unroll
      for (int m = 0; m < DW; ++m)
#pragma unroll
        for (int i = 0; i < 4; ++i) f[m][i] *= gf[m][i];
      const float4* Ef = w4 + opaque_offset(D * Lds::kLayer);
      f32x4 lo[16];
#pragma unroll
      for (int mb = 0; mb < 16; ++mb) lo[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int m = 0; m < DW; ++m)
#pragma unroll
        for (int mb = 0; mb < 16; ++mb) lo[mb] = mfma_frag(Ef[(mb * DW + m) * 64 + lane], f[m], lo[mb]);
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
      const float lse = __logf(xsum4(se)) + mx;
      float yl = 0.0f;
#pragma unroll
      for (int m = 0; m < DW; ++m) {
        yl = __builtin_fmaf(ey[m].x, f[m][0], yl);
        yl = __builtin_fmaf(ey[m].y, f[m][1], yl);
        yl = __builtin_fmaf(ey[m].z, f[m][2], yl);
        yl = __builtin_fmaf(ey[m].w, f[m][3], yl);
      }
      yl = xsum4(yl);
      if (lg == 0 && valid) ce_sum += static_cast<double>(lse - yl);
      if (!kPert && valid) {
        const int64_t pos = (static_cast<int64_t>(e) * B + b) * (T - 1) + t;
#pragma unroll
        for (int m = 0; m < DW; ++m)
          *reinterpret_cast<float4*>(a.fdec + pos * dm + 16 * m + 4 * lg) = make_float4(f[m][0], f[m][1], f[m][2], f[m][3]);
        if (lg == 0) a.lse[pos] = lse;
      }
#pragma unroll
      for (int m = 0; m < DW; ++m) er[m] = ey[m];
    }
  }

  // Per-block sum of the 64 sequence losses in a fixed order.
  __syncthreads();   // every wave is past its loop: the weight region is free
  double* red = reinterpret_cast<double*>(w4);
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
    if (threadIdx.x < n) {
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

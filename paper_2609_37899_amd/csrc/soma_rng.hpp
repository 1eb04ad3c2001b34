// soma_rng.hpp -- counter-based probe generators for gfx950.
//
// z[k] for parameter k of direction j at step `step` of an expert with stream
// seed `seed` is element k & 3 of gauss_quad(stream_key(seed, step), j,
// lo32(step), k >> 2):
//   Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11) with
//     key = (lo32(seed), hi32(seed) ^ hi32(step)),
//     counter = (lo32(q), j, lo32(step), hi32(q));
//   Box-Muller on (w0, w1) and (w2, w3):
//     u1 = ((wa >> 8) + 1) 2^-24, u2 = (wb >> 8) 2^-24,
//     r = sqrt(-2 ln u1), (za, zb) = (r cos 2 pi u2, r sin 2 pi u2).
// ln, cos and sin are series evaluated with correctly rounded fp32 +, *, /,
// fma and sqrt in a fixed order (the file must be compiled with
// -ffp-contract=off), so every lane reproduces the same bits as any other
// conforming implementation of the same definition.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace soma {

__device__ __forceinline__ uint2 stream_key(uint64_t seed, uint64_t step) {
  return make_uint2(static_cast<uint32_t>(seed),
                    static_cast<uint32_t>(seed >> 32) ^ static_cast<uint32_t>(step >> 32));
}

// Ten rounds of the Philox4x32 S-P network; the key advances by the Weyl
// increments (golden ratio, sqrt(3) - 1) after every round.
__device__ __forceinline__ uint4 philox4x32_10(uint4 x, uint2 k) {
  constexpr uint32_t kM0 = 0xD2511F53u, kM1 = 0xCD9E8D57u;
  constexpr uint32_t kW0 = 0x9E3779B9u, kW1 = 0xBB67AE85u;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    // One 32x32->64 product per multiplier (a single v_mad_u64_u32).
    const uint64_t p0 = static_cast<uint64_t>(kM0) * x.x;
    const uint64_t p1 = static_cast<uint64_t>(kM1) * x.z;
    x = make_uint4(static_cast<uint32_t>(p1 >> 32) ^ x.y ^ k.x, static_cast<uint32_t>(p1),
                   static_cast<uint32_t>(p0 >> 32) ^ x.w ^ k.y, static_cast<uint32_t>(p0));
    k.x += kW0;
    k.y += kW1;
  }
  return x;
}

// ln(m 2^-24), m in [1, 2^24]: m 2^-24 = 2^n f, f in (1/sqrt2, sqrt2];
// ln f = 2 atanh(s) = 2s (1 + s^2/3 + s^4/5 + ... + s^10/11), s = (f-1)/(f+1);
// ln 2 = hi + lo with a 16-bit hi so that n * hi is exact.
__device__ __forceinline__ float ln_u24(uint32_t m) {
  // m <= 2^24 converts exactly; its exponent field is floor(log2 m) and its
  // mantissa field with a zero exponent is f = m 2^-floor(log2 m) in [1, 2).
  const uint32_t mb = __float_as_uint(static_cast<float>(m));
  int e = static_cast<int>(mb >> 23) - 127;
  float f = __uint_as_float((mb & 0x007FFFFFu) | 0x3F800000u);
  if (f > 0x1.6a09e6p+0f) {  // fp32 nearest to sqrt(2)
    f = f * 0.5f;
    e = e + 1;
  }
  const float n = static_cast<float>(e - 24);
  const float kLn2Hi = 0x1.62e4p-1f;           // 0.693145751953125
  const float kLn2Lo = 0x1.7f7d1cp-20f;        // fp32 nearest to ln 2 - kLn2Hi
  const float s = (f - 1.0f) / (f + 1.0f);
  const float s2 = s * s;
  float q = __builtin_fmaf(s2, 1.0f / 11.0f, 1.0f / 9.0f);
  q = __builtin_fmaf(s2, q, 1.0f / 7.0f);
  q = __builtin_fmaf(s2, q, 1.0f / 5.0f);
  q = __builtin_fmaf(s2, q, 1.0f / 3.0f);
  q = q * s2;
  const float two_s = s + s;
  const float lnf = __builtin_fmaf(two_s, q, two_s);
  return __builtin_fmaf(n, kLn2Hi, __builtin_fmaf(n, kLn2Lo, lnf));
}

// (cos, sin)(2 pi i 2^-24), i in [0, 2^24).  4 i 2^-24 = qd + r exactly, qd
// the nearest quarter turn (ties up), r in [-1/2, 1/2); sin and cos of
// (pi/2) r by their Taylor series to r^11 and r^12.  Coefficients: the fp32
// values nearest to (-1)^floor(n/2) (pi/2)^n / n!.
__device__ __forceinline__ void sincos_2pi_u24(uint32_t i, float& c_out, float& s_out) {
  const uint32_t qd = (i + (1u << 21)) >> 22;
  const int32_t rem = static_cast<int32_t>(i) - static_cast<int32_t>(qd << 22);
  const float r = static_cast<float>(rem) * 0x1p-22f;
  const float r2 = r * r;
  float sp = __builtin_fmaf(r2, -0x1.e3075p-19f, 0x1.507834p-13f);  // S11, S9
  sp = __builtin_fmaf(r2, sp, -0x1.32d2ccp-8f);                     // S7
  sp = __builtin_fmaf(r2, sp, 0x1.466bc6p-4f);                      // S5
  sp = __builtin_fmaf(r2, sp, -0x1.4abbcep-1f);                     // S3
  sp = __builtin_fmaf(r2, sp, 0x1.921fb6p+0f);                      // S1
  const float sn = sp * r;
  float cp = __builtin_fmaf(r2, 0x1.f9d38ap-22f, -0x1.a6d1f2p-16f);  // C12, C10
  cp = __builtin_fmaf(r2, cp, 0x1.e1f506p-11f);                      // C8
  cp = __builtin_fmaf(r2, cp, -0x1.55d3c8p-6f);                      // C6
  cp = __builtin_fmaf(r2, cp, 0x1.03c1fp-2f);                        // C4
  cp = __builtin_fmaf(r2, cp, -0x1.3bd3ccp+0f);                      // C2
  const float cs = __builtin_fmaf(r2, cp, 1.0f);                     // C0
  const uint32_t qm = qd & 3u;
  const bool odd = (qm & 1u) != 0u;
  const float cm = odd ? sn : cs;
  const float sm = odd ? cs : sn;
  c_out = (qm == 1u || qm == 2u) ? -cm : cm;
  s_out = (qm >= 2u) ? -sm : sm;
}

// Correctly rounded sqrt for y = +-0 or a positive normal fp32 number: the
// hardware estimate s (within 1 ulp) is replaced by its neighbour when the
// exact residual y - s'^2 of a neighbour s' shows it to be the rounded root.
// (The general lowering adds a rescale for tiny inputs and a special-value
// path; y = -2 ln u1 is never tiny, infinite or NaN.)
__device__ __forceinline__ float sqrt_rn_normal(float y) {
  const float s = __builtin_amdgcn_sqrtf(y);
  const float sm = __uint_as_float(__float_as_uint(s) - 1u);
  const float sp = __uint_as_float(__float_as_uint(s) + 1u);
  const float rm = __builtin_fmaf(-sm, s, y);
  const float rp = __builtin_fmaf(-sp, s, y);
  float r = (rm <= 0.0f) ? sm : s;
  r = (rp > 0.0f) ? sp : r;
  return r;
}

__device__ __forceinline__ float2 box_muller(uint32_t wa, uint32_t wb) {
  const float lnu = ln_u24((wa >> 8) + 1u);
  const float r = sqrt_rn_normal(-2.0f * lnu);
  float c, s;
  sincos_2pi_u24(wb >> 8, c, s);
  return make_float2(r * c, r * s);
}

// z[4q .. 4q+3] of direction `pair`.
__device__ __forceinline__ float4 gauss_quad(uint2 key, uint32_t pair, uint32_t step_lo,
                                             uint64_t q) {
  const uint4 w = philox4x32_10(
      make_uint4(static_cast<uint32_t>(q), pair, step_lo, static_cast<uint32_t>(q >> 32)), key);
  const float2 a = box_muller(w.x, w.y);
  const float2 b = box_muller(w.z, w.w);
  return make_float4(a.x, a.y, b.x, b.y);
}

// Probe laws.  Gaussian; sparse Rademacher, the paper's training law (each
// coordinate 0 w.p. 1/2, -1 or +1 w.p. 1/4, Appendix E); dense Rademacher,
// the law of its variance theory (Section 4; Appendix F).
enum : int { kProbeGaussian = 0, kProbeSparseRademacher = 1, kProbeRademacher = 2 };

// z[k4 .. k4+3] (k4 a multiple of 4) under a Rademacher law.  Coordinate k
// reads the 2-bit field at bits 2 (k & 15) of word (k >> 4) & 3 of Philox
// block k >> 6, counter (lo32(k >> 6), pair, lo32(step), hi32(k >> 6)): the
// high bit makes a sparse coordinate active, the low bit is the sign (1: -1);
// the dense law uses the sign bit alone.
__device__ __forceinline__ float4 rademacher_quad(uint2 key, uint32_t pair, uint32_t step_lo, uint64_t k4,
                                                  bool dense) {
  const uint64_t b = k4 >> 6;
  const uint4 w = philox4x32_10(
      make_uint4(static_cast<uint32_t>(b), pair, step_lo, static_cast<uint32_t>(b >> 32)), key);
  const uint32_t wi = static_cast<uint32_t>(k4 >> 4) & 3u;
  const uint32_t word = wi == 0u ? w.x : (wi == 1u ? w.y : (wi == 2u ? w.z : w.w));
  const uint32_t f8 = word >> (2u * (static_cast<uint32_t>(k4) & 15u));   // four 2-bit fields
  float z[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t f = (f8 >> (2 * i)) & 3u;
    const float sgn = (f & 1u) ? -1.0f : 1.0f;
    z[i] = (dense || (f >> 1) != 0u) ? sgn : 0.0f;
  }
  return make_float4(z[0], z[1], z[2], z[3]);
}

// z[k4 .. k4+3] of direction `pair` under probe law `law` (k4 a multiple of 4).
__device__ __forceinline__ float4 probe_quad(int law, uint2 key, uint32_t pair, uint32_t step_lo, uint64_t k4) {
  if (law == kProbeGaussian) return gauss_quad(key, pair, step_lo, k4 >> 2);
  return rademacher_quad(key, pair, step_lo, k4, law == kProbeRademacher);
}

}  // namespace soma

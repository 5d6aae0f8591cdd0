// Counter-based Gaussian perturbation Z(seed, step, query, arena index).
//
// ZO-Act samples Z ~ N(0, I) in each layer's coefficient space (Section 3) and
// draws a fresh Z per step and query (Algorithm 2).  Here Z is a pure function of
// its coordinates, regenerated wherever it is needed and never stored:
//   * Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): key (lo32 seed, hi32 seed),
//     counter (lo32(e >> 2), hi32(e >> 2), step, query); arena index e is lane e & 3.
//   * Box-Muller with the angle in quarter turns: words (w0, w1) -> lanes 0, 1 as
//     (R cos, R sin), words (w2, w3) -> lanes 2, 3.  u1 = ((w0 >> 8) + 1) 2^-24,
//     ln u1 = (E - 24) ln2 + ln m with m in [sqrt(1/2), sqrt(2)) and
//     ln m = 2s(1 + s^2/3 + s^4/5 + s^6/7 + s^8/9), s = (m - 1)/(m + 1);
//     R = sqrt(-2 ln u1); quadrant w1 >> 30 and 22 fraction bits f, with
//     sin(pi f/2), cos(pi f/2) from Maclaurin series of degree 13 and 14.
// Every step is one fp32 operation in the written order: no contraction into
// fused multiply-adds, IEEE correctly rounded division and square root, so the
// values are reproducible bit for bit by any IEEE fp32 implementation.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace zoact {
namespace rng {

struct Words {
  uint32_t w0, w1, w2, w3;
};

__device__ __forceinline__ Words philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0,
                                               uint32_t k1) {
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    if (round) {
      k0 += 0x9E3779B9u;  // Weyl increments of the key schedule
      k1 += 0xBB67AE85u;
    }
    const uint32_t hi0 = __umulhi(0xD2511F53u, c0), lo0 = 0xD2511F53u * c0;
    const uint32_t hi1 = __umulhi(0xCD9E8D57u, c2), lo1 = 0xCD9E8D57u * c2;
    const uint32_t n0 = hi1 ^ c1 ^ k0;
    const uint32_t n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  return Words{c0, c1, c2, c3};
}

__device__ __forceinline__ float f32_bits(uint32_t b) { return __uint_as_float(b); }

// ln(((w >> 8) + 1) * 2^-24) via exponent split and the atanh series.
__device__ __forceinline__ float log_uniform(uint32_t w) {
#pragma clang fp contract(off)
  const uint32_t n = (w >> 8) + 1u;  // 1 .. 2^24, exact as fp32
  const uint32_t bits = __float_as_uint((float)n);
  int e = (int)(bits >> 23) - 127;
  float m = f32_bits((bits & 0x007FFFFFu) | 0x3F800000u);
  if (m >= f32_bits(0x3FB504F3u)) {  // sqrt(2)
    m = m * 0.5f;
    e += 1;
  }
  const float s = (m - 1.0f) / (m + 1.0f);
  const float s2 = s * s;
  float p = f32_bits(0x3DE38E39u);   // 1/9
  p = p * s2 + f32_bits(0x3E124925u);  // 1/7
  p = p * s2 + f32_bits(0x3E4CCCCDu);  // 1/5
  p = p * s2 + f32_bits(0x3EAAAAABu);  // 1/3
  p = p * s2 + 1.0f;
  const float lnm = (s + s) * p;
  return (float)(e - 24) * f32_bits(0x3F317218u) + lnm;  // ln 2
}

// (cos, sin) of the quarter-turn angle (w >> 30) + f, f = ((w >> 8) & 0x3FFFFF) 2^-22.
__device__ __forceinline__ void quarter_turn_sincos(uint32_t w, float& c_out, float& s_out) {
#pragma clang fp contract(off)
  const uint32_t q = w >> 30;
  const float f = (float)((w >> 8) & 0x3FFFFFu) * 0x1p-22f;
  const float f2 = f * f;
  // (pi/2)^n / n! with alternating signs, rounded to fp32
  float sp = f32_bits(0x33747A1Au);   // + x^13
  sp = sp * f2 + f32_bits(0xB67183A8u);  // - x^11
  sp = sp * f2 + f32_bits(0x39283C1Au);  // + x^9
  sp = sp * f2 + f32_bits(0xBB996966u);  // - x^7
  sp = sp * f2 + f32_bits(0x3DA335E3u);  // + x^5
  sp = sp * f2 + f32_bits(0xBF255DE7u);  // - x^3
  sp = sp * f2 + f32_bits(0x3FC90FDBu);  // + x
  const float sn = f * sp;
  float cp = f32_bits(0xB1DB7128u);   // - x^14
  cp = cp * f2 + f32_bits(0x34FCE9C5u);  // + x^12
  cp = cp * f2 + f32_bits(0xB7D368F9u);  // - x^10
  cp = cp * f2 + f32_bits(0x3A70FA83u);  // + x^8
  cp = cp * f2 + f32_bits(0xBCAAE9E4u);  // - x^6
  cp = cp * f2 + f32_bits(0x3E81E0F8u);  // + x^4
  cp = cp * f2 + f32_bits(0xBF9DE9E6u);  // - x^2
  cp = cp * f2 + 1.0f;
  const float cs = cp;
  c_out = (q == 0) ? cs : (q == 1) ? -sn : (q == 2) ? -cs : sn;
  s_out = (q == 0) ? sn : (q == 1) ? cs : (q == 2) ? -sn : -cs;
}

__device__ __forceinline__ void box_muller(uint32_t wa, uint32_t wb, float& z0, float& z1) {
#pragma clang fp contract(off)
  const float rad = __builtin_sqrtf(-2.0f * log_uniform(wa));
  float c, s;
  quarter_turn_sincos(wb, c, s);
  z0 = rad * c;
  z1 = rad * s;
}

// The four Z values of counter block `blk` (arena indices 4 blk .. 4 blk + 3).
__device__ __forceinline__ float4 gauss_block(uint64_t seed, uint32_t step, uint32_t query, uint64_t blk) {
  const Words w = philox4x32_10((uint32_t)blk, (uint32_t)(blk >> 32), step, query, (uint32_t)seed,
                                (uint32_t)(seed >> 32));
  float4 z;
  box_muller(w.w0, w.w1, z.x, z.y);
  box_muller(w.w2, w.w3, z.z, z.w);
  return z;
}

__device__ __forceinline__ float lane_of(const float4& z, int lane) {
  return lane == 0 ? z.x : lane == 1 ? z.y : lane == 2 ? z.z : z.w;
}

// Z at a single arena index.
__device__ __forceinline__ float gauss_at(uint64_t seed, uint32_t step, uint32_t query, uint64_t e) {
  return lane_of(gauss_block(seed, step, query, e >> 2), (int)(e & 3));
}

}  // namespace rng
}  // namespace zoact

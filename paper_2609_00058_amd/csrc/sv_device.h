// sv_device.h -- device building blocks of libsynthverify (gfx950).
//
// Counter-based generation and the distribution transforms behind sv_synth
// and sv_perturb.  Every floating-point step is one IEEE-754 fp32 operation
// rounded to nearest-even: the library is compiled with -ffp-contract=off, no
// fast-math, fp32 denormals kept, and correctly rounded fp32 division and
// square root, so a value depends only on (seed, stream, index) and is the same
// bits on any machine that performs the same operation sequence.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sv {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11).  Ten rounds of two
// 32x32->64 multiplications by the round multipliers; the high halves are
// XOR-ed with the untouched words and the round key, the low halves move
// across.  The key advances by the Weyl increments 2^32/phi and
// 2^32 (sqrt(3) - 1) between rounds.  Key = 64-bit seed; counter =
// (block index, substream id), each as (low, high) words.  The key words
// and the substream words are uniform across a launch, so the compiler keeps
// the key schedule and the first round's second product in scalar registers.
// ---------------------------------------------------------------------------
struct Key {
  uint32_t k0, k1;   // seed words
  uint32_t s0, s1;   // substream words
};

// a ^ b ^ k in one VALU instruction: CDNA4's three-input bitwise operation
// with truth table 0x96 (odd parity).  k is wave-uniform (a round key).
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t k) {
  uint32_t r;
  asm("v_bitop3_b32 %0, %1, %2, %3 bitop3:0x96" : "=v"(r) : "v"(a), "v"(b), "s"(k));
  return r;
}

__device__ __forceinline__ u32x4 philox_block(const Key &key, uint64_t block) {
  uint32_t x0 = (uint32_t)block, x1 = (uint32_t)(block >> 32), x2 = key.s0, x3 = key.s1;
  uint32_t k0 = key.k0, k1 = key.k1;
  {
    // first round: words 2 and 3 are the (uniform) substream, left to the compiler
    const uint64_t a = (uint64_t)0xD2511F53u * x0;
    const uint64_t b = (uint64_t)0xCD9E8D57u * x2;
    const uint32_t n0 = (uint32_t)(b >> 32) ^ x1 ^ k0;
    const uint32_t n2 = (uint32_t)(a >> 32) ^ x3 ^ k1;
    x1 = (uint32_t)b;
    x3 = (uint32_t)a;
    x0 = n0;
    x2 = n2;
  }
#pragma unroll
  for (int r = 1; r < 10; ++r) {
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
    const uint64_t a = (uint64_t)0xD2511F53u * x0;
    const uint64_t b = (uint64_t)0xCD9E8D57u * x2;
    const uint32_t n0 = xor3((uint32_t)(b >> 32), x1, k0);
    const uint32_t n2 = xor3((uint32_t)(a >> 32), x3, k1);
    x1 = (uint32_t)b;
    x3 = (uint32_t)a;
    x0 = n0;
    x2 = n2;
  }
  return u32x4{x0, x1, x2, x3};
}

// ---------------------------------------------------------------------------
// Bit views
// ---------------------------------------------------------------------------
__device__ __forceinline__ float as_f32(uint32_t u) { return __uint_as_float(u); }
__device__ __forceinline__ uint32_t as_u32(float f) { return __float_as_uint(f); }

// fp32 -> bf16 bits, round to nearest even; NaN keeps its top half with the
// quiet bit set.
__device__ __forceinline__ uint32_t bf16_rne(uint32_t x) {
  const bool nan = (x & 0x7FFFFFFFu) > 0x7F800000u;
  const uint32_t r = (x + 0x7FFFu + ((x >> 16) & 1u)) >> 16;
  return nan ? ((x >> 16) | 0x40u) : r;
}

// 24-bit uniform: top 24 bits of a word scaled by 2^-24 (exact).
__device__ __forceinline__ float unit24(uint32_t w) { return (float)(w >> 8) * 0x1p-24f; }

// ---------------------------------------------------------------------------
// ln of a positive normal fp32 value.  Write x = 2^e m, m in [1, 2), and
// halve m (raising e) when it exceeds sqrt(2), so m lies in [sqrt(1/2),
// sqrt(2)).  Then ln m = 2 atanh(s) with s = (m - 1)/(m + 1), |s| < 0.172,
// summed as s (2 + s^2 (2/3 + s^2 (2/5 + s^2 (2/7 + s^2 2/9)))), and
// ln x = e ln2_hi + (ln m + e ln2_lo) where ln2_hi = 45426/2^16 (so e ln2_hi
// is exact) and ln2_lo is the fp32 rounding of ln 2 - ln2_hi.  Constants are
// the fp32 roundings of the stated exact values.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float ln_f32(float x) {
  const uint32_t bits = as_u32(x);
  int e = (int)(bits >> 23) - 127;                      // x > 0
  float m = as_f32((bits & 0x007FFFFFu) | 0x3F800000u);
  if (m > 0x1.6a09e6p+0f) {                            // sqrt(2)
    m = m * 0.5f;
    e = e + 1;
  }
  const float f = m - 1.0f;
  const float s = f / (2.0f + f);
  const float z = s * s;
  float p = 0x1.c71c72p-3f;                              // 2/9
  p = 0x1.24924ap-2f + z * p;                            // 2/7
  p = 0x1.99999ap-2f + z * p;                            // 2/5
  p = 0x1.555556p-1f + z * p;                            // 2/3
  p = 2.0f + z * p;
  const float lnm = s * p;
  const float ef = (float)e;
  return ef * 0x1.62e4p-1f + (lnm + ef * 0x1.7f7d1cp-20f);   // ln2 hi, lo
}

// sin(pi f / 2) and cos(pi f / 2) for f in [0, 1/2], Taylor series in f whose
// coefficients are (-1)^k (pi/2)^n / n! rounded to fp32.
__device__ __forceinline__ float sin_q(float f) {
  const float f2 = f * f;
  float p = 0x1.507834p-13f;           //  (pi/2)^9 / 9!
  p = -0x1.32d2ccp-8f + f2 * p;        // -(pi/2)^7 / 7!
  p = 0x1.466bc6p-4f + f2 * p;         //  (pi/2)^5 / 5!
  p = -0x1.4abbcep-1f + f2 * p;        // -(pi/2)^3 / 3!
  p = 0x1.921fb6p+0f + f2 * p;         //  pi/2
  return f * p;
}

__device__ __forceinline__ float cos_q(float f) {
  const float f2 = f * f;
  float p = -0x1.a6d1f2p-16f;          // -(pi/2)^10 / 10!
  p = 0x1.e1f506p-11f + f2 * p;        //  (pi/2)^8 / 8!
  p = -0x1.55d3c8p-6f + f2 * p;        // -(pi/2)^6 / 6!
  p = 0x1.03c1f0p-2f + f2 * p;         //  (pi/2)^4 / 4!
  p = -0x1.3bd3ccp+0f + f2 * p;        // -(pi/2)^2 / 2!
  return 1.0f + f2 * p;
}

// sin and cos of 2 pi j / 2^24 for j < 2^24: quadrant q = j >> 22, fraction
// f = (j mod 2^22) / 2^22; above f = 1/2 the series run on the exact
// complement 1 - f with sine and cosine exchanged; the quadrant rotates the
// pair (negation is exact).
__device__ __forceinline__ void sincos_2pi(uint32_t j, float &s, float &c) {
  const uint32_t q = j >> 22;
  const uint32_t fj = j & 0x003FFFFFu;
  const bool lower = fj <= 0x00200000u;
  const float f = (float)(lower ? fj : 0x00400000u - fj) * 0x1p-22f;
  const float a = sin_q(f), b = cos_q(f);
  const float S = lower ? a : b;       // sin(pi fj / 2^23)
  const float C = lower ? b : a;       // cos(pi fj / 2^23)
  const float sq = (q & 1u) ? C : S;
  const float cq = (q & 1u) ? -S : C;
  s = (q & 2u) ? -sq : sq;
  c = (q & 2u) ? -cq : cq;
}

// Box-Muller pair from two words: u1 = ((wa >> 8) + 1) 2^-24 in (0, 1],
// u2 = (wb >> 8) 2^-24; r = sqrt(-2 ln u1); (r cos 2 pi u2, r sin 2 pi u2).
__device__ __forceinline__ void box_muller(uint32_t wa, uint32_t wb, float &zc, float &zs) {
  const float u1 = (float)((wa >> 8) + 1u) * 0x1p-24f;
  const float r = sqrtf(-2.0f * ln_f32(u1));
  float s, c;
  sincos_2pi(wb >> 8, s, c);
  zc = r * c;
  zs = r * s;
}

// ---------------------------------------------------------------------------
// Next representable value up or down (IEEE nextafter toward +-Inf); NaN is
// returned unchanged, a step from +-0 lands on the smallest denormal of the
// direction's sign, Inf stays Inf in its own direction.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t next_f32(uint32_t x, bool up) {
  const uint32_t mag = x & 0x7FFFFFFFu;
  if (mag > 0x7F800000u) return x;
  if (mag == 0u) return up ? 0x00000001u : 0x80000001u;
  if ((x == 0x7F800000u && up) || (x == 0xFF800000u && !up)) return x;
  const bool neg = (x >> 31) != 0u;
  return (up != neg) ? x + 1u : x - 1u;
}

__device__ __forceinline__ uint32_t next_bf16(uint32_t x, bool up) {
  const uint32_t mag = x & 0x7FFFu;
  if (mag > 0x7F80u) return x;
  if (mag == 0u) return up ? 0x0001u : 0x8001u;
  if ((x == 0x7F80u && up) || (x == 0xFF80u && !up)) return x;
  const bool neg = (x >> 15) != 0u;
  return ((up != neg) ? x + 1u : x - 1u) & 0xFFFFu;
}

}  // namespace sv

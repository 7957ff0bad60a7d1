// sv_device.h -- device building blocks of libsynthverify (gfx950).
//
// Counter-based generation and the distribution transforms behind sv_synth
// and sv_perturb.  Every floating-point step is one IEEE-754 fp32 operation
// rounded to nearest-even (a fused multiply-add where written as one): the
// library is compiled with -ffp-contract=off, no fast-math, fp32 denormals
// kept, and correctly rounded fp32 division and square root, so a value
// depends only on (seed, stream, index) and is the same bits on any machine
// that performs the same operation sequence.
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
  {
    // second round: word 1 is the low half of the first round's uniform
    // product, so (word 1 ^ key) is one scalar and a plain XOR leaves the
    // compiler free to keep uniform operands scalar
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
    const uint64_t a = (uint64_t)0xD2511F53u * x0;
    const uint64_t b = (uint64_t)0xCD9E8D57u * x2;
    const uint32_t n0 = (uint32_t)(b >> 32) ^ (x1 ^ k0);
    const uint32_t n2 = ((uint32_t)(a >> 32) ^ k1) ^ x3;
    x1 = (uint32_t)b;
    x3 = (uint32_t)a;
    x0 = n0;
    x2 = n2;
  }
  {
    // third round: in a launch whose block indices stay below 2^32, word 3
    // (the low half of the second round's product of a uniform word) is
    // uniform too; a plain XOR costs no more when it is not
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
    const uint64_t a = (uint64_t)0xD2511F53u * x0;
    const uint64_t b = (uint64_t)0xCD9E8D57u * x2;
    const uint32_t n0 = xor3((uint32_t)(b >> 32), x1, k0);
    const uint32_t n2 = (uint32_t)(a >> 32) ^ (x3 ^ k1);
    x1 = (uint32_t)b;
    x3 = (uint32_t)a;
    x0 = n0;
    x2 = n2;
  }
#pragma unroll
  for (int r = 3; r < 10; ++r) {
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

// A wave-uniform value copied once into a vector register: for an operand
// that a loop would otherwise move there again on every iteration (a VOP3
// instruction reads at most one scalar register).
__device__ __forceinline__ float in_vgpr(float x) {
  float r;
  asm("v_mov_b32 %0, %1" : "=v"(r) : "s"(x));
  return r;
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

// Two fp32 values, neither a NaN, to two bf16 in one word (the first in the
// low half) by the hardware conversion (v_cvt_pk_bf16_f32): round to nearest
// even, Inf stays Inf, denormals are kept -- bf16_rne's result for every fp32
// bit pattern that is not a NaN (checked on all of them).  For values that
// cannot be NaN: uniform and normal synthesis.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t bf16x2_rne_not_nan(uint32_t lo, uint32_t hi) {
  // the empty asm keeps the fp32 rounding of the values: no fusion of the
  // arithmetic that produced them with this conversion
  asm("" : "+v"(lo), "+v"(hi));
  const bf16x2_t h = __builtin_convertvector((f32x2_t{as_f32(lo), as_f32(hi)}), bf16x2_t);
  return __builtin_bit_cast(uint32_t, h);
}

// 24-bit uniform: top 24 bits of a word scaled by 2^-24 (exact).
__device__ __forceinline__ float unit24(uint32_t w) { return (float)(w >> 8) * 0x1p-24f; }

// ---------------------------------------------------------------------------
// ln of a positive normal fp32 value.  x = 2^e 1.M; when 1.M >= fp32(sqrt 2)
// the mantissa is halved and e raised, so m lies in [sqrt(1/2), sqrt(2)) and
// f = m - 1 is exact.  Both follow from one integer offset: subtracting the
// bits of fp32(sqrt(1/2)) = 0x3F3504F3 leaves e in the bits above the
// mantissa field (arithmetic shift) and m - fp32(sqrt(1/2)) below it.
// ln m = f P(f), P the degree-9 Chebyshev interpolant of ln(1 + f) / f on
// [sqrt(1/2) - 1, sqrt(2) - 1] with coefficients rounded to fp32, by fused
// multiply-add Horner steps; then ln x = e ln2_hi + (ln m + e ln2_lo),
// ln2_hi = 45426/2^16 (e ln2_hi exact), ln2_lo the fp32 rounding of
// ln 2 - ln2_hi, both sums fused with their products.  No division.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float ln_f32(float x) {
  const int32_t ix = (int32_t)as_u32(x) - 0x3F3504F3;
  const float ef = (float)(ix >> 23);
  const float m = as_f32((uint32_t)(ix & 0x007FFFFF) + 0x3F3504F3u);
  const float f = m - 1.0f;
  float p = -0x1.31335ap-4f;                             // degree 9
  p = __builtin_fmaf(p, f, 0x1.064786p-3f);
  p = __builtin_fmaf(p, f, -0x1.0fb036p-3f);
  p = __builtin_fmaf(p, f, 0x1.22cf10p-3f);
  p = __builtin_fmaf(p, f, -0x1.5423b0p-3f);
  p = __builtin_fmaf(p, f, 0x1.999e86p-3f);
  p = __builtin_fmaf(p, f, -0x1.000424p-2f);
  p = __builtin_fmaf(p, f, 0x1.55555ep-2f);
  p = __builtin_fmaf(p, f, -0x1.fffff8p-2f);
  p = __builtin_fmaf(p, f, 1.0f);                        // degree 0
  const float lnm = f * p;
  return __builtin_fmaf(ef, 0x1.62e4p-1f, __builtin_fmaf(ef, 0x1.7f7d1cp-20f, lnm));   // ln2 hi, lo
}

// IEEE (correctly rounded) square root of v in {0} and [2^-126, 2^126]: the
// hardware square root is within one ulp (and not always rounded correctly on
// the Box-Muller radicands), and of it and its two neighbours the one whose
// fused residual v - s' s has the right sign is the rounded root (no input
// here is denormal, infinite or negative, so no scaling).
__device__ __forceinline__ float sqrt_rn(float v) {
  float s = __builtin_amdgcn_sqrtf(v);
  const float sd = as_f32(as_u32(s) - 1u), su = as_f32(as_u32(s) + 1u);
  const float rd = __builtin_fmaf(-sd, s, v), ru = __builtin_fmaf(-su, s, v);
  s = (rd <= 0.0f) ? sd : s;
  s = (ru > 0.0f) ? su : s;
  return s;
}

// ---------------------------------------------------------------------------
// sin and cos of 2 pi j / 2^24 for j < 2^24: j = 2^16 k + r at the nearest of
// 256 table angles (k = round(j / 2^16) mod 256, r in [-2^15, 2^15) the low
// half of j as a signed 16-bit number), b = fp32(r) fp32(2 pi / 2^24),
// sin b = b + b (b^2 fp32(-1/6)), cos b = 1 - b^2 / 2 (within 2^-30 of the
// true values for |b| <= pi / 256), then the angle-sum formulas, one fused
// multiply-add each.  The table holds sin and cos of 2 pi k / 256 rounded to
// nearest fp32 (exact zeros positive); it lives in LDS, filled at the start of
// every kernel that draws normal values (load_sincos_table).
// ---------------------------------------------------------------------------
static __shared__ f32x2_t sincos_tab[256];

// sin x and cos x for 0 <= x <= pi / 4 in fp64: Taylor series through x^19
// and x^20 (the first omitted terms are below 2^-60 relative).
__device__ inline double sin_series_f64(double x) {
  const double x2 = x * x;
  double p = 1.0 / 121645100408832000.0;                 // 1 / 19!
  p = __builtin_fma(p, -x2, 1.0 / 355687428096000.0);    // 1 / 17!
  p = __builtin_fma(p, -x2, 1.0 / 1307674368000.0);      // 1 / 15!
  p = __builtin_fma(p, -x2, 1.0 / 6227020800.0);         // 1 / 13!
  p = __builtin_fma(p, -x2, 1.0 / 39916800.0);           // 1 / 11!
  p = __builtin_fma(p, -x2, 1.0 / 362880.0);             // 1 / 9!
  p = __builtin_fma(p, -x2, 1.0 / 5040.0);               // 1 / 7!
  p = __builtin_fma(p, -x2, 1.0 / 120.0);                // 1 / 5!
  p = __builtin_fma(p, -x2, 1.0 / 6.0);                  // 1 / 3!
  p = __builtin_fma(p, -x2, 1.0);
  return x * p;
}

__device__ inline double cos_series_f64(double x) {
  const double x2 = x * x;
  double p = 1.0 / 2432902008176640000.0;                // 1 / 20!
  p = __builtin_fma(p, -x2, 1.0 / 6402373705728000.0);   // 1 / 18!
  p = __builtin_fma(p, -x2, 1.0 / 20922789888000.0);     // 1 / 16!
  p = __builtin_fma(p, -x2, 1.0 / 87178291200.0);        // 1 / 14!
  p = __builtin_fma(p, -x2, 1.0 / 479001600.0);          // 1 / 12!
  p = __builtin_fma(p, -x2, 1.0 / 3628800.0);            // 1 / 10!
  p = __builtin_fma(p, -x2, 1.0 / 40320.0);              // 1 / 8!
  p = __builtin_fma(p, -x2, 1.0 / 720.0);                // 1 / 6!
  p = __builtin_fma(p, -x2, 1.0 / 24.0);                 // 1 / 4!
  p = __builtin_fma(p, -x2, 1.0 / 2.0);                  // 1 / 2!
  return __builtin_fma(p, -x2, 1.0);
}

// Entry k of the table: the first octant (m in 0..32 of the 64 steps of a
// quadrant) from the series, the rest by the exact symmetries of the octant
// and the quadrant; fp64 rounded to nearest fp32.
__device__ inline f32x2_t sincos_entry(uint32_t k) {
  const uint32_t q = k >> 6, m = k & 63u;
  double sm = 0.0, cm = 1.0;
  if (m != 0u) {
    const double x = (double)(m <= 32u ? m : 64u - m) * (3.141592653589793 / 128.0);
    const double sx = sin_series_f64(x), cx = cos_series_f64(x);
    sm = m <= 32u ? sx : cx;
    cm = m <= 32u ? cx : sx;
  }
  const double sv = q == 0 ? sm : q == 1 ? cm : q == 2 ? -sm : -cm;
  const double cv = q == 0 ? cm : q == 1 ? -sm : q == 2 ? -cm : sm;
  return f32x2_t{sv == 0.0 ? 0.0f : (float)sv, cv == 0.0 ? 0.0f : (float)cv};
}

// Fills the table; reached by every thread of the workgroup, before any use.
__device__ inline void load_sincos_table() {
  for (uint32_t k = threadIdx.x; k < 256u; k += blockDim.x) sincos_tab[k] = sincos_entry(k);
  __syncthreads();
}

// j = w >> 8 for a 32-bit word w: k = ((j + 2^15) >> 16) mod 256 is the top
// byte of w + 2^23 (the carry out of bit 31 is the mod 256), and r is bits
// 8..23 of w as a signed number.
__device__ __forceinline__ void sincos_2pi_word(uint32_t w, float &s, float &c) {
  const uint32_t k = (w + 0x800000u) >> 24;
  const int32_t r = (int32_t)(int16_t)(uint16_t)(w >> 8);
  const float b = (float)r * 0x1.921fb6p-22f;          // fp32(2 pi / 2^24)
  const float b2 = b * b;
  const float sb = __builtin_fmaf(b, b2 * -0x1.555556p-3f, b);   // fp32(-1/6)
  const float cb = __builtin_fmaf(b2, -0.5f, 1.0f);
  const f32x2_t t = sincos_tab[k];
  s = __builtin_fmaf(t.x, cb, t.y * sb);
  c = __builtin_fmaf(t.y, cb, -(t.x * sb));
}

__device__ __forceinline__ void sincos_2pi(uint32_t j, float &s, float &c) {   // j < 2^24
  sincos_2pi_word(j << 8, s, c);
}

// Box-Muller pair from two words: u1 = ((wa >> 8) + 1) 2^-24 in (0, 1],
// u2 = (wb >> 8) 2^-24; r = sqrt(-2 ln u1); (r cos 2 pi u2, r sin 2 pi u2).
//
// The radius takes ln_f32's steps with two exact rescalings folded in:
// u1's bits are those of the integer k24 + 1 (converted exactly) less 24 in
// the exponent field, so the offset subtracted from them absorbs the 2^-24;
// and -2 ln u1 is ln_f32 with every Horner coefficient and both ln 2 parts
// times -2 -- scaling by a power of two commutes with each rounding here (no
// intermediate is denormal or overflows), so the bits equal
// sqrt_rn(-2 * ln_f32(u1)) for every k24 (compared on all 2^24 of them).
__device__ __forceinline__ float bm_radicand(uint32_t k24) {
  const int32_t ix = (int32_t)as_u32((float)(k24 + 1u)) - (0x3F3504F3 + (24 << 23));
  const float ef = (float)(ix >> 23);
  const float m = as_f32((uint32_t)(ix & 0x007FFFFF) + 0x3F3504F3u);
  const float f = m - 1.0f;
  float p = 0x1.31335ap-3f;                              // -2 x the coefficients of ln_f32
  p = __builtin_fmaf(p, f, -0x1.064786p-2f);
  p = __builtin_fmaf(p, f, 0x1.0fb036p-2f);
  p = __builtin_fmaf(p, f, -0x1.22cf10p-2f);
  p = __builtin_fmaf(p, f, 0x1.5423b0p-2f);
  p = __builtin_fmaf(p, f, -0x1.999e86p-2f);
  p = __builtin_fmaf(p, f, 0x1.000424p-1f);
  p = __builtin_fmaf(p, f, -0x1.55555ep-1f);
  p = __builtin_fmaf(p, f, 0x1.fffff8p-1f);
  p = __builtin_fmaf(p, f, -2.0f);
  const float lnm = f * p;
  return __builtin_fmaf(ef, -0x1.62e4p+0f, __builtin_fmaf(ef, -0x1.7f7d1cp-19f, lnm));
}

__device__ __forceinline__ float bm_radius(uint32_t k24) {   // u1 = (k24 + 1) 2^-24
  return sqrt_rn(bm_radicand(k24));
}

__device__ __forceinline__ void box_muller(uint32_t wa, uint32_t wb, float &zc, float &zs) {
  const float r = bm_radius(wa >> 8);
  float s, c;
  sincos_2pi_word(wb, s, c);
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

__device__ __forceinline__ uint32_t next_f16(uint32_t x, bool up) {
  const uint32_t mag = x & 0x7FFFu;
  if (mag > 0x7C00u) return x;
  if (mag == 0u) return up ? 0x0001u : 0x8001u;
  if ((x == 0x7C00u && up) || (x == 0xFC00u && !up)) return x;
  const bool neg = (x >> 15) != 0u;
  return ((up != neg) ? x + 1u : x - 1u) & 0xFFFFu;
}

__device__ __forceinline__ uint64_t next_f64(uint64_t x, bool up) {
  const uint64_t mag = x & 0x7FFFFFFFFFFFFFFFull;
  if (mag > 0x7FF0000000000000ull) return x;
  if (mag == 0u) return up ? 1ull : 0x8000000000000001ull;
  if ((x == 0x7FF0000000000000ull && up) || (x == 0xFFF0000000000000ull && !up)) return x;
  const bool neg = (x >> 63) != 0u;
  return (up != neg) ? x + 1u : x - 1u;
}

// ---------------------------------------------------------------------------
// fp16 and fp64 outputs of fp32 values.  fp16: round to nearest even through
// the hardware conversion (IEEE, subnormals kept, overflow to Inf); a NaN
// keeps its sign and the top 10 fraction bits, bit 0 set if those are zero.
// fp64: exact widening; Inf stays Inf and a NaN keeps its sign and fraction,
// moved to the top of the fp64 fraction.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t f16_rne(uint32_t x) {
  if ((x & 0x7FFFFFFFu) > 0x7F800000u) {
    const uint32_t frac = (x & 0x7FFFFFu) >> 13;
    return ((x >> 16) & 0x8000u) | 0x7C00u | (frac ? frac : 1u);
  }
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)as_f32(x));
}

__device__ __forceinline__ float f16_widen(uint32_t h) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
}

__device__ __forceinline__ uint64_t widen_f32_bits(uint32_t b) {
  if ((b & 0x7F800000u) == 0x7F800000u)
    return ((uint64_t)(b >> 31) << 63) | 0x7FF0000000000000ull | ((uint64_t)(b & 0x7FFFFFu) << 29);
  return (uint64_t)__double_as_longlong((double)as_f32(b));
}

__device__ __forceinline__ uint64_t f64_bits(double d) { return (uint64_t)__double_as_longlong(d); }
__device__ __forceinline__ double bits_f64(uint64_t u) { return __longlong_as_double((long long)u); }

}  // namespace sv

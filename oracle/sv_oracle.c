/*
 * sv_oracle.c -- CPU test oracle: seeded synthesis, candidate derivation and
 * the elementwise check of Eq. (1) with its report.
 *
 * TEST INFRASTRUCTURE ONLY (see sv_oracle.h).  Plain serial C, one element at
 * a time, no vectorisation, no blocking, no threads.  Built with
 * -O2 -ffp-contract=off so that every float operation written below is one
 * IEEE-754 operation rounded to nearest-even, exactly as written; fmaf() is
 * the IEEE fused multiply-add (one rounding).
 *
 * What the paper fixes and what this file adds:
 *  - Sec. 4.2.1, Eq. (1): V = I[ |K(x) - y| <= atol + rtol*|y| ], rtol scaling
 *    the magnitude of the reference y.  or_compare() evaluates it per element.
 *  - Sec. 4.2.1 asks for test inputs drawn from a broad numeric range (a
 *    Gaussian with mean 5 and standard deviation 10 is its example); that is
 *    the normal distribution with explicit mean and std below.
 *  - The generator, the word-to-element mapping and the transforms are not in
 *    the paper (it only points to general-purpose numerical libraries).  They
 *    follow these conventions: Philox4x32-10 (Salmon, Moraes,
 *    Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC'11) keyed
 *    by the seed with counter (block, stream); uniform from the top 24 bits
 *    of a word (from a 16-bit half-word for bf16 outputs);
 *    Box-Muller (1958) with ln, sin and cos written as fixed sequences of fp32
 *    operations (a Chebyshev polynomial for ln, Horner steps fused
 *    multiply-adds; sin and cos from a table of 256 correctly rounded values
 *    and short series of the remaining angle); Lemire's multiply-shift for integer
 *    ranges; a class-threshold mix for special values.
 */
#include "sv_oracle.h"

#include <math.h>
#include <string.h>

/* ------------------------------------------------------------------------- */
/* Bit views                                                                  */
/* ------------------------------------------------------------------------- */
static uint32_t f2u(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
static float u2f(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

/* ------------------------------------------------------------------------- */
/* Philox4x32-10 (Salmon et al., SC'11).                                      */
/* One round multiplies counter words 0 and 2 by the two round multipliers;   */
/* the high halves are mixed with the other two words and the round key, the  */
/* low halves pass through.  The key is bumped by the two Weyl constants      */
/* (golden ratio and sqrt(3)-1, scaled by 2^32) between rounds.               */
/* ------------------------------------------------------------------------- */
#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

void or_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; round++) {
    if (round > 0) {
      k0 += PHILOX_W0;
      k1 += PHILOX_W1;
    }
    uint64_t p0 = (uint64_t)PHILOX_M0 * (uint64_t)x0;
    uint64_t p1 = (uint64_t)PHILOX_M1 * (uint64_t)x2;
    uint32_t y0 = (uint32_t)(p1 >> 32) ^ x1 ^ k0;
    uint32_t y1 = (uint32_t)p1;
    uint32_t y2 = (uint32_t)(p0 >> 32) ^ x3 ^ k1;
    uint32_t y3 = (uint32_t)p0;
    x0 = y0; x1 = y1; x2 = y2; x3 = y3;
  }
  out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* key = (low, high) words of the seed; counter = (low, high) words of the
 * block index c followed by (low, high) words of the substream id. */
void or_philox_block(uint64_t seed, uint64_t stream, uint64_t c, uint32_t out[4]) {
  uint32_t ctr[4] = {(uint32_t)c, (uint32_t)(c >> 32), (uint32_t)stream, (uint32_t)(stream >> 32)};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  or_philox4x32_10(ctr, key, out);
}

/* ------------------------------------------------------------------------- */
/* Natural logarithm for positive normal fp32 x.                              */
/* x = 2^e * m with m in [sqrt(1/2), sqrt(2)): m is x's mantissa as 1.M,      */
/* halved (and e raised) when 1.M >= fp32(sqrt 2); with f = m - 1 (exact),    */
/* ln m = f * P(f) where P is the degree-9 Chebyshev approximation of         */
/* ln(1 + f) / f on [sqrt(1/2) - 1, sqrt(2) - 1] (interpolation at the 10     */
/* Chebyshev nodes of that interval, coefficients rounded to fp32), evaluated */
/* by Horner steps that are each one fused multiply-add.                      */
/* ln x = e*ln2_hi + (ln m + e*ln2_lo), with ln2_hi = ln 2 rounded to 16 bits */
/* (so e*ln2_hi is exact for |e| < 2^8) and ln2_lo = fp32(ln 2 - ln2_hi),     */
/* both additions fused with their products.                                  */
/* ------------------------------------------------------------------------- */
static const float LN_SQRT2 = 0x1.6a09e6p+0f;      /* fp32(sqrt 2)                */
static const float LN_P1 = -0x1.fffff8p-2f;        /* Chebyshev fit, degree 1     */
static const float LN_P2 = 0x1.55555ep-2f;
static const float LN_P3 = -0x1.000424p-2f;
static const float LN_P4 = 0x1.999e86p-3f;
static const float LN_P5 = -0x1.5423b0p-3f;
static const float LN_P6 = 0x1.22cf10p-3f;
static const float LN_P7 = -0x1.0fb036p-3f;
static const float LN_P8 = 0x1.064786p-3f;
static const float LN_P9 = -0x1.31335ap-4f;        /* Chebyshev fit, degree 9     */
static const float LN2_HI = 0x1.62e4p-1f;          /* 45426 / 2^16                */
static const float LN2_LO = 0x1.7f7d1cp-20f;       /* fp32(ln 2 - 45426 / 2^16)   */

float or_ln_f32(float x) {
  uint32_t bits = f2u(x);
  int e = (int)((bits >> 23) & 0xFFu) - 127;
  float m = u2f((bits & 0x007FFFFFu) | 0x3F800000u); /* m in [1, 2) */
  if (m >= LN_SQRT2) {
    m = m * 0.5f;                                    /* exact */
    e = e + 1;
  }
  float f = m - 1.0f;                                /* exact (Sterbenz) */
  float p = LN_P9;
  p = fmaf(p, f, LN_P8);
  p = fmaf(p, f, LN_P7);
  p = fmaf(p, f, LN_P6);
  p = fmaf(p, f, LN_P5);
  p = fmaf(p, f, LN_P4);
  p = fmaf(p, f, LN_P3);
  p = fmaf(p, f, LN_P2);
  p = fmaf(p, f, LN_P1);
  p = fmaf(p, f, 1.0f);
  float ln_m = f * p;
  float ef = (float)e;
  return fmaf(ef, LN2_HI, fmaf(ef, LN2_LO, ln_m));
}

/* ------------------------------------------------------------------------- */
/* sin and cos of the angle 2 pi j / 2^24, j < 2^24.                          */
/* The angle is split at the nearest of 256 table angles: j = 2^16 k + r with */
/* k = round(j / 2^16) mod 256 (halves up) and r in [-2^15, 2^15), so that    */
/* angle = 2 pi k / 256 + b, b = 2 pi r / 2^24, |b| <= pi / 256.  The table   */
/* holds sin and cos of 2 pi k / 256 rounded to fp32 (to nearest, exact zeros */
/* positive); b = fp32(r) * fp32(2 pi / 2^24) (one rounding); over |b| <=     */
/* pi/256 sin b = b - b^3/6 and cos b = 1 - b^2/2 are within 2^-30 relative   */
/* of the true values; then the angle-sum formulas, each with one fused       */
/* multiply-add.  Table points on the axes (k a multiple of 64) are exact, so */
/* near the zeros of sin and cos the result is the small term alone and keeps */
/* its relative accuracy.                                                     */
/* ------------------------------------------------------------------------- */
static const float SC_B = 0x1.921fb6p-22f;    /* fp32(2 pi / 2^24)   */
static const float SC_S3 = -0x1.555556p-3f;   /* fp32(-1/6)          */
static float TAB_SIN[256], TAB_COS[256];

/* sin and cos of 2 pi k / 256 rounded to fp32: the first octant (m in 0..32
 * of 64 per quadrant) in long double, the rest by the exact symmetries of
 * the quadrant and the octant. */
__attribute__((constructor)) static void init_sincos_table(void) {
  const long double pi = 3.14159265358979323846264338327950288L;
  for (int k = 0; k < 256; k++) {
    int q = k >> 6, m = k & 63;
    long double sm, cm;
    if (m == 0) {
      sm = 0.0L;
      cm = 1.0L;
    } else if (m <= 32) {
      sm = sinl(pi * (long double)m / 128.0L);
      cm = cosl(pi * (long double)m / 128.0L);
    } else {
      sm = cosl(pi * (long double)(64 - m) / 128.0L);
      cm = sinl(pi * (long double)(64 - m) / 128.0L);
    }
    long double s = q == 0 ? sm : q == 1 ? cm : q == 2 ? -sm : -cm;
    long double c = q == 0 ? cm : q == 1 ? -sm : q == 2 ? -cm : sm;
    TAB_SIN[k] = s == 0.0L ? 0.0f : (float)s;
    TAB_COS[k] = c == 0.0L ? 0.0f : (float)c;
  }
}

void or_sincos_table(float *s, float *c) {
  for (int k = 0; k < 256; k++) {
    s[k] = TAB_SIN[k];
    c[k] = TAB_COS[k];
  }
}

void or_sincos_2pi_f32(uint32_t j24, float *s_out, float *c_out) {
  uint32_t j = j24 & 0x00FFFFFFu;
  uint32_t k = ((j + 0x8000u) >> 16) & 0xFFu;                           /* nearest table angle */
  int32_t r = (int32_t)(j & 0xFFFFu) - (int32_t)((j & 0x8000u) << 1);   /* j - 2^16 k (mod 2^24) */
  float b = (float)r * SC_B;
  float b2 = b * b;
  float sb = fmaf(b, b2 * SC_S3, b);                                     /* sin b */
  float cb = fmaf(b2, -0.5f, 1.0f);                                      /* cos b */
  float sk = TAB_SIN[k], ck = TAB_COS[k];
  *s_out = fmaf(sk, cb, ck * sb);
  *c_out = fmaf(ck, cb, -(sk * sb));
}

/* ------------------------------------------------------------------------- */
/* Box-Muller: u1 = ((wa >> 8) + 1) 2^-24 in (0, 1], u2 = (wb >> 8) 2^-24 in  */
/* [0, 1); r = sqrt(-2 ln u1); z_cos = r cos(2 pi u2), z_sin = r sin(2 pi u2) */
/* ------------------------------------------------------------------------- */
float or_radius_f32(uint32_t k24) {   /* u1 = (k24 + 1) 2^-24 */
  float u1 = (float)((k24 & 0x00FFFFFFu) + 1u) * 0x1p-24f;
  float lnu = or_ln_f32(u1);
  return sqrtf(-2.0f * lnu);
}

void or_box_muller_f32(uint32_t wa, uint32_t wb, float *zc, float *zs) {
  float r = or_radius_f32(wa >> 8);
  float s, c;
  or_sincos_2pi_f32(wb >> 8, &s, &c);
  *zc = r * c;
  *zs = r * s;
}

/* ------------------------------------------------------------------------- */
/* fp32 -> bf16, round to nearest even; NaN stays NaN (quiet bit forced).     */
/* ------------------------------------------------------------------------- */
uint16_t or_bf16_rne(uint32_t x) {
  if ((x & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((x >> 16) | 0x0040u);
  uint32_t lsb = (x >> 16) & 1u;
  return (uint16_t)((x + 0x7FFFu + lsb) >> 16);
}

static float bf16_to_f32(uint16_t h) { return u2f((uint32_t)h << 16); }

/* ------------------------------------------------------------------------- */
/* fp32 -> IEEE binary16 (1 sign, 5 exponent, 10 fraction bits), round to     */
/* nearest even, subnormals kept, beyond the largest finite value -> Inf.      */
/* A NaN keeps its sign and the top 10 bits of its fraction (bit 0 set if      */
/* those are all zero, so that it stays a NaN).                                */
/* ------------------------------------------------------------------------- */
uint16_t or_f16_rne(uint32_t x) {
  uint16_t sign = (uint16_t)((x >> 16) & 0x8000u);
  uint32_t ax = x & 0x7FFFFFFFu;
  if (ax > 0x7F800000u) {                          /* NaN */
    uint16_t frac = (uint16_t)((ax & 0x7FFFFFu) >> 13);
    return (uint16_t)(sign | 0x7C00u | (frac ? frac : 1u));
  }
  /* the halfway point between 65504 (the largest half) and 65536 is 65520; a
   * tie there goes to the even neighbour 65536, which overflows */
  if (ax >= 0x477FF000u) return (uint16_t)(sign | 0x7C00u);
  if (ax <= 0x33000000u) return sign;              /* |v| <= 2^-25: to zero (2^-25 ties to even 0) */
  uint32_t e = ax >> 23;                           /* biased fp32 exponent, 102 .. 142 */
  uint32_t m = (ax & 0x7FFFFFu) | 0x800000u;       /* 24-bit significand */
  /* keep 11 significant bits for a normal half (e >= 113, i.e. |v| >= 2^-14);
   * for a subnormal half the quantum is 2^-24, so drop (126 - e) bits */
  uint32_t drop = e >= 113u ? 13u : 126u - e;
  uint32_t q = m >> drop, rest = m & ((1u << drop) - 1u), half = 1u << (drop - 1u);
  if (rest > half || (rest == half && (q & 1u))) q++;
  if (e >= 113u)                                   /* a carry into bit 11 moves to the next binade */
    return (uint16_t)(sign | (((e - 112u) << 10) + (q - 0x400u)));
  return (uint16_t)(sign | q);                     /* may round up to the smallest normal, 0x0400 */
}

/* binary16 -> fp32, exact */
static float f16_to_f32(uint16_t h) {
  uint32_t sign = ((uint32_t)h & 0x8000u) << 16;
  uint32_t e = (h >> 10) & 0x1Fu, f = h & 0x3FFu;
  if (e == 31u) return u2f(sign | 0x7F800000u | (f << 13));   /* Inf, NaN (fraction kept) */
  float mag = e == 0u ? ldexpf((float)f, -24) : ldexpf((float)(f | 0x400u), (int)e - 25);
  return u2f(sign | f2u(mag));
}

uint16_t or_next_f16(uint16_t x, int up) {
  uint16_t mag = x & 0x7FFFu;
  if (mag > 0x7C00u) return x;
  if (mag == 0) return up ? (uint16_t)0x0001u : (uint16_t)0x8001u;
  if (x == 0x7C00u && up) return x;
  if (x == 0xFC00u && !up) return x;
  int neg = (int)(x >> 15);
  return (uint16_t)((up != neg) ? x + 1u : x - 1u);
}

uint64_t or_next_f64(uint64_t x, int up) {
  uint64_t mag = x & 0x7FFFFFFFFFFFFFFFull;
  if (mag > 0x7FF0000000000000ull) return x;
  if (mag == 0) return up ? 1ull : 0x8000000000000001ull;
  if (x == 0x7FF0000000000000ull && up) return x;
  if (x == 0xFFF0000000000000ull && !up) return x;
  int neg = (int)(x >> 63);
  return (up != neg) ? x + 1u : x - 1u;
}

/* fp32 bits -> fp64 bits: exact for numbers; Inf stays Inf; a NaN keeps its
 * sign and its fraction, moved to the top of the fp64 fraction */
static uint64_t widen_f32_bits(uint32_t b) {
  uint64_t sign = (uint64_t)(b >> 31) << 63;
  if ((b & 0x7F800000u) == 0x7F800000u)
    return sign | 0x7FF0000000000000ull | ((uint64_t)(b & 0x7FFFFFu) << 29);
  double d = (double)u2f(b);
  uint64_t u;
  memcpy(&u, &d, 8);
  return u;
}

static double u2d(uint64_t u) { double d; memcpy(&d, &u, 8); return d; }
static uint64_t d2u(double d) { uint64_t u; memcpy(&u, &d, 8); return u; }

/* ------------------------------------------------------------------------- */
/* One step to the next representable value up (up != 0) or down.            */
/* ------------------------------------------------------------------------- */
uint32_t or_next_f32(uint32_t x, int up) {
  uint32_t mag = x & 0x7FFFFFFFu;
  if (mag > 0x7F800000u) return x;                          /* NaN */
  if (mag == 0) return up ? 0x00000001u : 0x80000001u;      /* +-0 */
  if (x == 0x7F800000u && up) return x;                     /* +Inf up */
  if (x == 0xFF800000u && !up) return x;                    /* -Inf down */
  int neg = (int)(x >> 31);
  return (up != neg) ? x + 1u : x - 1u;   /* magnitude grows when moving away from 0 */
}

uint16_t or_next_bf16(uint16_t x, int up) {
  uint16_t mag = x & 0x7FFFu;
  if (mag > 0x7F80u) return x;
  if (mag == 0) return up ? (uint16_t)0x0001u : (uint16_t)0x8001u;
  if (x == 0x7F80u && up) return x;
  if (x == 0xFF80u && !up) return x;
  int neg = (int)(x >> 15);
  return (uint16_t)((up != neg) ? x + 1u : x - 1u);
}

/* Array forms, one call per element. */
void or_philox_blocks(uint64_t seed, uint64_t stream, uint64_t c0, uint64_t n, uint32_t *out) {
  for (uint64_t k = 0; k < n; k++) or_philox_block(seed, stream, c0 + k, out + 4 * k);
}

void or_ln_f32_n(const float *x, float *y, uint64_t n) {
  for (uint64_t k = 0; k < n; k++) y[k] = or_ln_f32(x[k]);
}

void or_sincos_2pi_f32_n(const uint32_t *j24, float *s, float *c, uint64_t n) {
  for (uint64_t k = 0; k < n; k++) or_sincos_2pi_f32(j24[k], &s[k], &c[k]);
}

void or_radius_f32_n(const uint32_t *k24, float *r, uint64_t n) {
  for (uint64_t k = 0; k < n; k++) r[k] = or_radius_f32(k24[k]);
}

void or_bf16_rne_n(const uint32_t *x, uint16_t *y, uint64_t n) {
  for (uint64_t k = 0; k < n; k++) y[k] = or_bf16_rne(x[k]);
}

void or_f16_rne_n(const uint32_t *x, uint16_t *y, uint64_t n) {
  for (uint64_t k = 0; k < n; k++) y[k] = or_f16_rne(x[k]);
}

/* ------------------------------------------------------------------------- */
/* Synthesis                                                                  */
/* ------------------------------------------------------------------------- */
typedef struct {
  float a, span;           /* uniform: a + span * U                      */
  double a64, span64;      /* uniform into fp64: the same in fp64        */
  float mean, std;         /* normal                                     */
  int64_t lo;              /* integer range, permutation                 */
  uint64_t range;          /* hi - lo + 1 (0 stands for 2^64)            */
  unsigned half;           /* permutation: bits of each Feistel half     */
  uint32_t gate;           /* special: candidates have a gate byte below this */
  uint64_t t_nan, t_inf, t_den, t_zero;   /* cumulative class thresholds */
} prepared;

static uint64_t width32(double p) { return (uint64_t)floor(p * 4294967296.0); }

/* The width of a special class among the candidates: floor(p 2^32 256 / S),
 * evaluated as floor(fp64(p 2^40) / S) (p 2^40 is exact), at most 2^32. */
static uint64_t class_width(double p, uint32_t gate) {
  uint64_t w = (uint64_t)floor(p * 1099511627776.0 / (double)gate);
  return w < (1ull << 32) ? w : (1ull << 32);
}

static int is_float(int32_t dtype) {
  return dtype == OR_F32 || dtype == OR_BF16 || dtype == OR_F16 || dtype == OR_F64;
}
static int is_int(int32_t dtype) { return dtype == OR_I32 || dtype == OR_U8 || dtype == OR_I64; }
static int valid_dtype(int32_t dtype) { return is_float(dtype) || is_int(dtype); }

static int prepare(int32_t dtype, int32_t dist, const or_dist_params *p, prepared *q) {
  memset(q, 0, sizeof(*q));
  if (!valid_dtype(dtype)) return -2;
  if (!p) return -1;
  switch (dist) {
  case OR_UNIFORM: {
    if (!is_float(dtype)) return -2;
    if (dtype == OR_F64) {
      double a = p->a, b = p->b, span = b - a;
      if (!(a < b) || !isfinite(a) || !isfinite(b) || !isfinite(span)) return -1;
      q->a64 = a;
      q->span64 = span;
      return 0;
    }
    float a = (float)p->a, b = (float)p->b;
    float span = b - a;
    if (!(a < b) || isinf(a) || isinf(b) || isinf(span)) return -1;
    q->a = a;
    q->span = span;
    return 0;
  }
  case OR_NORMAL:
  case OR_SPECIAL: {
    if (!is_float(dtype)) return -2;
    q->mean = (float)p->mean;
    q->std = (float)p->std;
    if (!isfinite(q->mean) || !isfinite(q->std) || !(q->std >= 0.0f)) return -1;
    if (dist == OR_SPECIAL) {
      double ps[4] = {p->p_nan, p->p_inf, p->p_denorm, p->p_zero};
      double tot = 0.0;
      for (int k = 0; k < 4; k++) {
        if (!(ps[k] >= 0.0 && ps[k] <= 1.0)) return -1;
        tot += ps[k];
      }
      if (!(tot <= 1.0)) return -1;
      /* a share S / 256 >= tot of the elements are candidates (S = ceil(256 tot));
       * within them the classes take widths p / (S / 256) of the class word */
      q->gate = (uint32_t)ceil(256.0 * tot);
      if (q->gate) {
        const uint64_t full = 1ull << 32;
        q->t_nan = class_width(p->p_nan, q->gate);
        q->t_inf = q->t_nan + class_width(p->p_inf, q->gate);
        q->t_den = q->t_inf + class_width(p->p_denorm, q->gate);
        q->t_zero = q->t_den + class_width(p->p_zero, q->gate);
        if (q->t_inf > full) q->t_inf = full;
        if (q->t_den > full) q->t_den = full;
        if (q->t_zero > full) q->t_zero = full;
      }
    }
    return 0;
  }
  case OR_PERMUTATION:
    /* the N = hi - lo + 1 values lo .. hi in a seeded order, N <= 2^60 */
    if (!is_int(dtype)) return -2;
    if (p->lo > p->hi) return -1;
    if (dtype == OR_I32 && (p->lo < INT32_MIN || p->hi > INT32_MAX)) return -1;
    if (dtype == OR_U8 && (p->lo < 0 || p->hi > 255)) return -1;
    q->lo = p->lo;
    q->range = (uint64_t)p->hi - (uint64_t)p->lo + 1u;
    if (q->range == 0 || q->range > (1ull << 60)) return -1;
    {
      unsigned bits = 0;                      /* smallest b with 2^b >= N */
      while (bits < 64 && (1ull << bits) < q->range) bits++;
      q->half = bits < 2 ? 1u : (bits + 1u) / 2u;
    }
    return 0;
  case OR_INT_RANGE:
    if (!is_int(dtype)) return -2;
    if (p->lo > p->hi) return -1;
    if (dtype == OR_I32 && (p->lo < INT32_MIN || p->hi > INT32_MAX)) return -1;
    if (dtype == OR_U8 && (p->lo < 0 || p->hi > 255)) return -1;
    q->lo = p->lo;
    q->range = (uint64_t)p->hi - (uint64_t)p->lo + 1u;   /* wraps to 0 for the full int64 range */
    return 0;
  default:
    return -2;
  }
}

/* Permutation.  pi is a bijection of [0, N): a permutation G of the 2h-bit
 * words (2^2h the smallest even power of two >= N, h >= 1), followed from i
 * until it lands below N (cycle walking: the walk returns to [0, N) because
 * i's own cycle does, after fewer than 4 steps on average as 2^2h < 4N).
 * G(x) = (Feistel(x) + K_10) mod 2^2h.  The Feistel network has ten rounds
 * (six left the orders of 5 and 6 values measurably uneven); round r maps the
 * halves (L, R) to (R, L xor (F(R xor K_r) mod 2^h)), F the lowbias32 integer
 * hash (C. Wellons, hash-prospector, 2018).  Feistel rounds are even
 * permutations of the words, and the walk from even permutations does not
 * reach every order of [0, N) equally often; the added constant rotates the
 * words, an odd permutation for odd K_10, which evens this out.  The keys
 * K_0 .. K_10 are the words of Philox blocks 0, 1 and 2 of the tensor's
 * (seed, stream) sequence, in order. */
static uint32_t lowbias32(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}

static uint64_t word_permutation(uint64_t x, unsigned h, const uint32_t key[11]) {
  const uint64_t mask = (1ull << h) - 1u;
  uint64_t l = x >> h, r = x & mask;
  for (int k = 0; k < 10; k++) {
    uint64_t f = (uint64_t)lowbias32((uint32_t)r ^ key[k]) & mask;
    uint64_t t = l ^ f;
    l = r;
    r = t;
  }
  const uint64_t words = (1ull << (2u * h)) - 1u;   /* mask of the 2h-bit word */
  return (((l << h) | r) + key[10]) & words;
}

static uint64_t permute(uint64_t seed, uint64_t stream, const prepared *q, uint64_t i) {
  uint32_t key[12];
  or_philox_block(seed, stream, 0, key);
  or_philox_block(seed, stream, 1, key + 4);
  or_philox_block(seed, stream, 2, key + 8);
  uint64_t x = i;
  do {
    x = word_permutation(x, q->half, key);
  } while (x >= q->range);
  return x;
}

#define SPECIAL_CLASS_BLOCKS (1ull << 62)

/* Value of element i: fp32 bits (UNIFORM, NORMAL, SPECIAL; fp64 uniform gives
 * fp64 bits) or the integer (INT_RANGE), in the low bits of a 64-bit word. */
static uint64_t element_value(uint64_t seed, uint64_t stream, int32_t dtype, int32_t dist,
                              const prepared *q, uint64_t i) {
  uint32_t w[4];
  if (dist == OR_PERMUTATION) return (uint64_t)q->lo + permute(seed, stream, q, i);
  if (dist == OR_UNIFORM && dtype == OR_F64) {
    /* two elements per block, R = (w1:w0) for even i and (w3:w2) for odd i;
     * U = (R >> 11) 2^-53 in [0, 1); a + span U in fp64, two roundings */
    or_philox_block(seed, stream, i / 2u, w);
    unsigned h = (unsigned)(i % 2u);
    uint64_t R = ((uint64_t)w[2 * h + 1] << 32) | (uint64_t)w[2 * h];
    double U = (double)(R >> 11) * 0x1p-53;
    double t = q->span64 * U;
    return d2u(q->a64 + t);
  }
  if (dist == OR_UNIFORM && dtype == OR_BF16) {
    /* bf16: one 16-bit draw per element, eight elements per block: element i
     * takes half i mod 2 (the low half first) of word (i mod 8) / 2 of block
     * i / 8; U = h 2^-16 in [0, 1); a + span U in fp32, two roundings, then
     * rounded to bf16.  Sixteen bits reach every bf16 value of the top eight
     * binades of the range; fp16, with three more significand bits, keeps the
     * 24-bit draws below. */
    or_philox_block(seed, stream, i / 8u, w);
    uint32_t h = (w[(i % 8u) / 2u] >> (16u * (unsigned)(i % 2u))) & 0xFFFFu;
    float U = (float)h * 0x1p-16f;
    float t = q->span * U;
    return f2u(q->a + t);
  }
  if (dist == OR_UNIFORM) {
    /* four elements per block: element i takes word i mod 4 of block i / 4 */
    or_philox_block(seed, stream, i / 4u, w);
    float U = (float)(w[i % 4u] >> 8) * 0x1p-24f;
    float t = q->span * U;
    return f2u(q->a + t);
  }
  if (dist == OR_NORMAL) {
    /* words (w0, w1) give elements 4c (cos) and 4c+1 (sin); (w2, w3) give
     * elements 4c+2 (cos) and 4c+3 (sin) */
    or_philox_block(seed, stream, i / 4u, w);
    unsigned pair = (unsigned)((i % 4u) / 2u);
    float zc, zs;
    or_box_muller_f32(w[2 * pair], w[2 * pair + 1], &zc, &zs);
    float z = (i % 2u == 0u) ? zc : zs;
    return f2u(fmaf(q->std, z, q->mean));           /* mean + std z, one rounding */
  }
  if (dist == OR_INT_RANGE && dtype == OR_U8) {
    /* uint8: four elements per block, element i takes word i mod 4 of block
     * i / 4; value = lo + floor(w * range / 2^32) (range <= 256, so the
     * multiply-shift is biased by less than 2^-24) */
    or_philox_block(seed, stream, i / 4u, w);
    return (uint64_t)q->lo + (((uint64_t)w[i % 4u] * q->range) >> 32);
  }
  if (dist == OR_INT_RANGE) {
    /* int32, int64: two elements per block: R = (w1:w0) for even i, (w3:w2) for odd i;
     * value = lo + floor(R * range / 2^64) (Lemire's multiply-shift); a range
     * of 2^64 (the whole int64 line) takes R itself */
    or_philox_block(seed, stream, i / 2u, w);
    unsigned h = (unsigned)(i % 2u);
    uint64_t R = ((uint64_t)w[2 * h + 1] << 32) | (uint64_t)w[2 * h];
    uint64_t off = q->range ? (uint64_t)(((unsigned __int128)R * (unsigned __int128)q->range) >> 64) : R;
    return (uint64_t)q->lo + off;                   /* two's complement wrap-around: exact */
  }
  /* SPECIAL: the normal sequence above with some elements replaced.  Element
   * i = 4c + k is a candidate when its gate, the low byte of word k of normal
   * block c (the eight bits Box-Muller leaves unused), is below S = ceil(256
   * p), p the total probability of the four special classes.  A candidate
   * takes its class from x = word k of Philox block 2^62 + c (block indices
   * the normal values, below 2^58, never reach), against cumulative
   * thresholds of widths floor(p_class 2^32 256 / S) in the order NaN, Inf,
   * denormal, zero; x at or above the last keeps the normal value.  Its sign
   * and payload / mantissa come from r = x 0x9E3779B9 mod 2^32 (Fibonacci
   * hashing, Knuth, TAOCP vol. 3, 6.4): the low bits of r are a bijection of
   * the low bits of x, its top bit mixes all of x's bits. */
  or_philox_block(seed, stream, i / 4u, w);
  if ((w[i % 4u] & 0xFFu) >= q->gate) return element_value(seed, stream, dtype, OR_NORMAL, q, i);
  uint32_t cls[4];
  or_philox_block(seed, stream, SPECIAL_CLASS_BLOCKS + i / 4u, cls);
  const uint64_t x = cls[i % 4u];
  if (x >= q->t_zero) return element_value(seed, stream, dtype, OR_NORMAL, q, i);
  const uint32_t r = (uint32_t)x * 0x9E3779B9u;
  const uint32_t sign = r & 0x80000000u;
  if (x < q->t_nan) return sign | 0x7FC00000u | (r & 0x003FFFFFu);
  if (x < q->t_inf) return sign | 0x7F800000u;
  if (x < q->t_den) {
    const uint32_t m = r & 0x007FFFFFu;
    return sign | (m ? m : 1u);
  }
  return sign;
}

/* Stores an element value in the tensor's format: bf16 and fp16 round the
 * fp32 value to nearest even, fp64 widens it exactly (an fp64 uniform value
 * is already fp64), integers keep their low bits. */
static void store(int32_t dtype, int32_t dist, void *out, uint64_t k, uint64_t v) {
  switch (dtype) {
  case OR_BF16: ((uint16_t *)out)[k] = or_bf16_rne((uint32_t)v); break;
  case OR_F16: ((uint16_t *)out)[k] = or_f16_rne((uint32_t)v); break;
  case OR_F64: ((uint64_t *)out)[k] = dist == OR_UNIFORM ? v : widen_f32_bits((uint32_t)v); break;
  case OR_I64: ((uint64_t *)out)[k] = v; break;
  case OR_U8: ((uint8_t *)out)[k] = (uint8_t)v; break;
  default: ((uint32_t *)out)[k] = (uint32_t)v; break;
  }
}

int or_synth(uint64_t seed, uint64_t stream, int32_t dtype, int32_t dist,
             const or_dist_params *p, uint64_t offset, uint64_t n, void *out) {
  prepared q;
  int rc = prepare(dtype, dist, p, &q);
  if (rc) return rc;
  if (n && !out) return -1;
  if (dist == OR_PERMUTATION && (offset > q.range || n > q.range - offset)) return -1;   /* past the N values */
  for (uint64_t k = 0; k < n; k++)
    store(dtype, dist, out, k, element_value(seed, stream, dtype, dist, &q, offset + k));
  return 0;
}

int or_synth_at(uint64_t seed, uint64_t stream, int32_t dtype, int32_t dist,
                const or_dist_params *p, const uint64_t *idx, uint64_t n, void *out) {
  prepared q;
  int rc = prepare(dtype, dist, p, &q);
  if (rc) return rc;
  if (n && (!out || !idx)) return -1;
  if (dist == OR_PERMUTATION)
    for (uint64_t k = 0; k < n; k++)
      if (idx[k] >= q.range) return -1;
  for (uint64_t k = 0; k < n; k++)
    store(dtype, dist, out, k, element_value(seed, stream, dtype, dist, &q, idx[k]));
  return 0;
}

int or_special_class_counts(uint64_t seed, uint64_t stream, const or_dist_params *p,
                            uint64_t offset, uint64_t n, uint64_t counts[5]) {
  prepared q;
  int rc = prepare(OR_F32, OR_SPECIAL, p, &q);
  if (rc) return rc;
  for (int k = 0; k < 5; k++) counts[k] = 0;
  for (uint64_t i = offset; i < offset + n; i++) {
    uint32_t w[4];
    or_philox_block(seed, stream, i / 4u, w);
    if ((w[i % 4u] & 0xFFu) >= q.gate) {           /* not a candidate */
      counts[4]++;
      continue;
    }
    or_philox_block(seed, stream, SPECIAL_CLASS_BLOCKS + i / 4u, w);
    uint64_t x = w[i % 4u];
    int cls = x < q.t_nan ? 0 : x < q.t_inf ? 1 : x < q.t_den ? 2 : x < q.t_zero ? 3 : 4;
    counts[cls]++;
  }
  return 0;
}

/* ------------------------------------------------------------------------- */
/* Candidate derivation                                                       */
/* ------------------------------------------------------------------------- */
static size_t elem_bytes(int32_t dtype) {
  switch (dtype) {
  case OR_BF16: case OR_F16: return 2;
  case OR_F64: case OR_I64: return 8;
  case OR_U8: return 1;
  default: return 4;
  }
}

static uint64_t load_bits(int32_t dtype, const void *a, uint64_t k) {
  switch (elem_bytes(dtype)) {
  case 1: return ((const uint8_t *)a)[k];
  case 2: return ((const uint16_t *)a)[k];
  case 8: return ((const uint64_t *)a)[k];
  default: return ((const uint32_t *)a)[k];
  }
}

static void store_bits(int32_t dtype, void *a, uint64_t k, uint64_t bits) {
  switch (elem_bytes(dtype)) {
  case 1: ((uint8_t *)a)[k] = (uint8_t)bits; break;
  case 2: ((uint16_t *)a)[k] = (uint16_t)bits; break;
  case 8: ((uint64_t *)a)[k] = bits; break;
  default: ((uint32_t *)a)[k] = (uint32_t)bits; break;
  }
}

/* value of a 16- or 32-bit float element as fp32 (bf16 and fp16 widen exactly) */
static float as_f32(int32_t dtype, uint64_t bits) {
  if (dtype == OR_BF16) return bf16_to_f32((uint16_t)bits);
  if (dtype == OR_F16) return f16_to_f32((uint16_t)bits);
  return u2f((uint32_t)bits);
}

/* fp32 result back to the element format */
static uint64_t from_f32(int32_t dtype, float v) {
  if (dtype == OR_BF16) return or_bf16_rne(f2u(v));
  if (dtype == OR_F16) return or_f16_rne(f2u(v));
  return f2u(v);
}

static uint64_t perturb_element(uint64_t seed, uint64_t stream, int32_t dtype,
                                const or_perturb_plan *plan, uint64_t i, uint64_t b) {
  if (plan->op == OR_OP_COPY) return b;
  /* one Philox block per element: w0 selects (w0 < floor(p 2^32)), the top
   * bit of w1 chooses the direction, w1 gives the NaN payload mask, the top
   * 24 bits of w2 give the uniform variate of SCALE */
  uint32_t w[4];
  or_philox_block(seed, stream, i, w);
  if (!((uint64_t)w[0] < width32(plan->p))) return b;
  int up = (int)(w[1] >> 31);
  if (plan->op == OR_OP_ULP) {
    if (dtype == OR_BF16) return or_next_bf16((uint16_t)b, up);
    if (dtype == OR_F16) return or_next_f16((uint16_t)b, up);
    if (dtype == OR_F64) return or_next_f64(b, up);
    return or_next_f32((uint32_t)b, up);
  }
  if (plan->op == OR_OP_SCALE) {
    float U = (float)(w[2] >> 8) * 0x1p-24f;
    float amp = (float)plan->value;
    float two_amp = 2.0f * amp;
    float t = two_amp * U;
    float u = t - amp;
    float s = 1.0f + u;
    return from_f32(dtype, as_f32(dtype, b) * s);
  }
  /* SPECIAL_FLIP: zeros change sign, NaNs get their payload XOR-ed with a
   * nonzero mask below the quiet bit; everything else is left alone */
  if (dtype == OR_BF16) {
    uint32_t mag = (uint32_t)b & 0x7FFFu;
    if (mag == 0) return b ^ 0x8000u;
    if (mag > 0x7F80u) {
      uint32_t m = w[1] & 0x003Fu;
      return b ^ (m ? m : 1u);
    }
    return b;
  }
  uint32_t mag = (uint32_t)b & 0x7FFFFFFFu;
  if (mag == 0) return b ^ 0x80000000u;
  if (mag > 0x7F800000u) {
    uint32_t m = w[1] & 0x003FFFFFu;
    return b ^ (m ? m : 1u);
  }
  return b;
}

static uint64_t index_op(int32_t dtype, const or_perturb_plan *plan, uint64_t b) {
  if (plan->op == OR_OP_SET_AT) {
    uint64_t mask = elem_bytes(dtype) == 1 ? 0xFFu : elem_bytes(dtype) == 2 ? 0xFFFFu : 0xFFFFFFFFu;
    return plan->bits & mask;
  }
  if (plan->op == OR_OP_ADD_AT) {
    float v = (float)plan->value;
    return from_f32(dtype, as_f32(dtype, b) + v);
  }
  /* FAULT_AT: integers + 1 (wrapping in their width), floats x + (1 + |x|).
   * IEEE 754 leaves open which NaN a sum of two NaNs returns, and x + t has
   * two when x is a NaN (t = 1 + |x| is |x|'s NaN); so a NaN x gives |x| with
   * the quiet bit set, stated here rather than left to the order of the
   * operands.  x = -Inf gives -Inf + Inf, the invalid operation: the quiet
   * NaN with the sign bit set and no payload. */
  if (is_int(dtype)) return b + 1u;
  if (dtype == OR_F64) {
    double x = u2d(b);
    if (isnan(x)) return (b & 0x7FFFFFFFFFFFFFFFull) | 0x0008000000000000ull;
    if (isinf(x) && x < 0) return 0xFFF8000000000000ull;
    double t = 1.0 + fabs(x);
    return d2u(x + t);
  }
  float x = as_f32(dtype, b);
  if (isnan(x)) return from_f32(dtype, u2f((f2u(x) & 0x7FFFFFFFu) | 0x00400000u));
  if (isinf(x) && x < 0) return from_f32(dtype, u2f(0xFFC00000u));
  float t = 1.0f + fabsf(x);
  return from_f32(dtype, x + t);
}

/* Which candidate steps each element type supports. */
static int op_supported(int32_t dtype, int op) {
  if (op == OR_OP_COPY || op == OR_OP_FAULT_AT) return 1;
  switch (dtype) {
  case OR_F32: case OR_BF16: return 1;
  case OR_I32: return op == OR_OP_SET_AT;
  case OR_F16: return op == OR_OP_ULP || op == OR_OP_SET_AT;
  case OR_F64: return op == OR_OP_ULP;
  case OR_U8: return op == OR_OP_SET_AT;
  default: return 0;
  }
}

int or_perturb(uint64_t seed, uint64_t stream, int32_t dtype,
               const or_perturb_plan *plan, uint64_t offset, uint64_t n,
               const void *ref, void *cand) {
  if (!plan) return -1;
  if (!valid_dtype(dtype)) return -2;
  if (n && (!ref || !cand)) return -1;
  int op = plan->op;
  if (op < OR_OP_COPY || op > OR_OP_FAULT_AT) return -2;
  if (!op_supported(dtype, op)) return -2;
  /* the scale width and the added delta are used as fp32 values: they must
   * be finite there */
  if ((op == OR_OP_SCALE || op == OR_OP_ADD_AT) && !isfinite((float)plan->value)) return -1;
  if (op <= OR_OP_SPECIAL_FLIP) {
    if (op != OR_OP_COPY && !(plan->p >= 0.0 && plan->p <= 1.0)) return -1;
    for (uint64_t k = 0; k < n; k++)
      store_bits(dtype, cand, k,
                 perturb_element(seed, stream, dtype, plan, offset + k, load_bits(dtype, ref, k)));
    return 0;
  }
  if (plan->nidx && !plan->idx) return -1;
  for (uint64_t j = 0; j < plan->nidx; j++) {
    uint64_t i = plan->idx[j];
    if (i < offset || i - offset >= n) continue;
    uint64_t k = i - offset;
    store_bits(dtype, cand, k, index_op(dtype, plan, load_bits(dtype, ref, k)));
  }
  return 0;
}

/* ------------------------------------------------------------------------- */
/* Eq. (1) and the report                                                     */
/* ------------------------------------------------------------------------- */
/* exact value of a float element, or of an int32 / uint8 element, in fp64 */
static double load_value(int32_t dtype, const void *a, uint64_t k) {
  switch (dtype) {
  case OR_F32: return (double)((const float *)a)[k];
  case OR_BF16: return (double)bf16_to_f32(((const uint16_t *)a)[k]);
  case OR_F16: return (double)f16_to_f32(((const uint16_t *)a)[k]);
  case OR_F64: return ((const double *)a)[k];
  case OR_U8: return (double)((const uint8_t *)a)[k];
  default: return (double)((const int32_t *)a)[k];
  }
}

int or_compare(const void *ref, const void *cand, uint64_t n, int32_t dtype,
               double rtol, double atol, int32_t equal_nan, or_report *r) {
  if (!r) return -1;
  if (!valid_dtype(dtype)) return -2;
  if (n && (!ref || !cand)) return -1;
  /* integer types compare exactly and ignore the tolerances, which are then
   * not checked either */
  if (!is_int(dtype) && (!(rtol >= 0.0) || !(atol >= 0.0) || isinf(rtol) || isinf(atol))) return -1;
  memset(r, 0, sizeof(*r));
  r->n = n;
  r->first_mismatch = -1;
  double sum = 0.0, comp = 0.0;   /* Neumaier (1974) compensated summation */
  for (uint64_t k = 0; k < n; k++) {
    double y, a;                             /* reference output y, kernel output K(x) */
    int match, finite;
    double d = 0.0;
    if (dtype == OR_I64) {
      /* int64: exact comparison; d is the exact difference rounded once to fp64
       * (fp64 cannot hold every int64, so the values are not compared as fp64) */
      int64_t yi = ((const int64_t *)ref)[k], ai = ((const int64_t *)cand)[k];
      uint64_t mag = ai >= yi ? (uint64_t)ai - (uint64_t)yi : (uint64_t)yi - (uint64_t)ai;
      d = (double)mag;
      y = (double)yi;
      match = (ai == yi);
      finite = 1;
    } else if (is_int(dtype)) {
      /* int32 and uint8 are exact in fp64; checked exactly, tolerances do not apply */
      y = load_value(dtype, ref, k);
      a = load_value(dtype, cand, k);
      d = fabs(a - y);
      match = (a == y);
      finite = 1;
    } else {
      y = load_value(dtype, ref, k);
      a = load_value(dtype, cand, k);
      /* isnan / isinf may return any nonzero value (glibc's isinf gives -1 for
       * -Inf), so normalise to 0 / 1 before counting */
      int nan_y = isnan(y) != 0, nan_a = isnan(a) != 0;
      int inf_y = isinf(y) != 0, inf_a = isinf(a) != 0;
      r->nan_ref += (uint64_t)nan_y;
      r->nan_cand += (uint64_t)nan_a;
      r->inf_ref += (uint64_t)inf_y;
      r->inf_cand += (uint64_t)inf_a;
      if (nan_y || nan_a) {
        match = equal_nan && nan_y && nan_a;
        finite = 0;
      } else if (inf_y || inf_a) {
        match = (a == y);   /* identical infinities agree */
        finite = 0;
      } else {
        d = fabs(a - y);
        double t = atol + rtol * fabs(y);
        match = (d <= t);
        finite = 1;
      }
    }
    if (!match) {
      if (r->mismatches == 0) r->first_mismatch = (int64_t)k;
      r->mismatches++;
    }
    if (finite) {
      if (d > r->max_abs_err) r->max_abs_err = d;
      double rel = (d == 0.0) ? 0.0 : d / fabs(y);   /* y = 0, d > 0 gives +Inf */
      if (rel > r->max_rel_err) r->max_rel_err = rel;
      double t = sum + d;
      if (isinf(t)) {
        /* the running sum (or d itself) has overflowed: every d is >= 0, so
         * the fp64 sum is +Inf from here on in any order; the compensation
         * term has no meaning past this point (it would turn Inf - Inf into
         * NaN) and is dropped */
        comp = 0.0;
      } else if (fabs(sum) >= fabs(d)) {
        comp += (sum - t) + d;
      } else {
        comp += (d - t) + sum;
      }
      sum = t;
    }
  }
  r->err_sum = sum + comp;
  return 0;
}

int or_compare_batched(const or_segment *segs, uint32_t nseg, or_report *reports) {
  if (nseg && (!segs || !reports)) return -1;
  for (uint32_t s = 0; s < nseg; s++) {
    const or_segment *g = &segs[s];
    int rc = or_compare(g->ref, g->cand, g->n, g->dtype, g->rtol, g->atol, g->equal_nan, &reports[s]);
    if (rc) return rc;
  }
  return 0;
}

/* ------------------------------------------------------------ Eq. (3), Eq. (4)
 * Performance of a candidate from its mean latency in milliseconds, Eq. (3)
 * (the latency averaged over repeated runs, Sec. 5.1; the unit is that of the
 * paper's RScore, 1 / ms).  Reward, Eq. (4): r = -1 + C + C V P with C = 1 when
 * the kernel compiled (Eq. (2)), V = 1 when it passed the functional check
 * (Eq. (1)).  The fail-fast order of Sec. 4.2.2 never profiles a kernel that
 * failed an earlier stage, so its performance term is absent (0) whatever p
 * holds; for a profiled kernel p must be a number >= 0, else the result is NaN. */
double or_performance(double mean_latency_ms) { return 1.0 / mean_latency_ms; }

double or_reward(int compiled, int valid, double p) {
  const double c = compiled ? 1.0 : 0.0, v = valid ? 1.0 : 0.0;
  if (c * v == 0.0) return -1.0 + c;
  if (!(p >= 0.0)) return NAN;
  return -1.0 + c + c * v * p;
}

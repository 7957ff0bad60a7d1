/*
 * sv_oracle.h -- declarations of the CPU test oracle for seeded synthesis and
 * elementwise checking (Synthesis-Based Verification, Sec. 4.2 of
 * "CUDA-Harness", arXiv 2609.00058).
 *
 * TEST INFRASTRUCTURE ONLY. This header, sv_oracle.c and the Python wrapper in
 * this directory exist so that tests, the smoke entry and the CPU-baseline leg
 * of the benchmark can check the GPU library against a plain, serial, obviously
 * correct implementation.  Nothing in the product path may include, link or
 * call it, and it includes nothing from the product path.  Every enum value,
 * struct and constant here is the oracle's own.
 *
 * Conventions the paper leaves open (generator, word-to-element mapping,
 * distribution transforms, NaN/Inf rules, report fields) are stated with the
 * functions below and in sv_oracle.c, and followed there step by step.
 */
#ifndef SV_ORACLE_H
#define SV_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { OR_F32 = 0, OR_BF16 = 1, OR_I32 = 2, OR_F16 = 3, OR_F64 = 4, OR_U8 = 5, OR_I64 = 6 };
enum { OR_UNIFORM = 0, OR_NORMAL = 1, OR_INT_RANGE = 2, OR_SPECIAL = 3, OR_PERMUTATION = 4 };
enum {
  OR_OP_COPY = 0,          /* cand = ref                                   */
  OR_OP_ULP = 1,           /* Bernoulli(p): one ulp up or down             */
  OR_OP_SCALE = 2,         /* Bernoulli(p): ref * (1 + u), |u| <= value    */
  OR_OP_SPECIAL_FLIP = 3,  /* Bernoulli(p): sign of zeros, NaN payloads    */
  OR_OP_ADD_AT = 4,        /* cand[idx] = ref[idx] + value                 */
  OR_OP_SET_AT = 5,        /* cand[idx] = raw bit pattern                  */
  OR_OP_FAULT_AT = 6       /* cand[idx] = ref + (1 + |ref|)  (int: ref + 1) */
};

typedef struct {
  double a, b;                              /* uniform [a, b)               */
  double mean, std;                         /* normal, and SPECIAL's normal */
  int64_t lo, hi;                           /* integer range, inclusive     */
  double p_nan, p_inf, p_denorm, p_zero;    /* SPECIAL class probabilities  */
} or_dist_params;

typedef struct {
  int32_t op;
  double p;               /* selection probability of elementwise ops  */
  double value;           /* ADD_AT delta, SCALE half-width            */
  uint32_t bits;          /* SET_AT pattern                            */
  const uint64_t *idx;    /* index list of *_AT ops (global indices)   */
  uint64_t nidx;
} or_perturb_plan;

typedef struct {
  uint64_t n;
  uint64_t mismatches;
  int64_t first_mismatch;   /* -1 when there is none */
  double max_abs_err;
  double max_rel_err;
  double err_sum;
  uint64_t nan_ref, nan_cand, inf_ref, inf_cand;
} or_report;

typedef struct {
  const void *ref;
  const void *cand;
  uint64_t n;
  int32_t dtype;
  double rtol, atol;
  int32_t equal_nan;
} or_segment;

/* Philox4x32-10 on an explicit counter and key. */
void or_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);
/* The block at counter c of substream `stream` under `seed`. */
void or_philox_block(uint64_t seed, uint64_t stream, uint64_t c, uint32_t out[4]);

/* Building blocks exposed so that tests can pin them one at a time. */
float or_ln_f32(float x);
void or_sincos_2pi_f32(uint32_t j24, float *s, float *c);
/* the 256 table values sin, cos of 2 pi k / 256 (fp32, correctly rounded) */
void or_sincos_table(float *s, float *c);
float or_radius_f32(uint32_t k24);   /* Box-Muller radius for u1 = (k24 + 1) 2^-24 */
void or_box_muller_f32(uint32_t wa, uint32_t wb, float *zc, float *zs);
uint16_t or_bf16_rne(uint32_t f32_bits);
uint32_t or_next_f32(uint32_t bits, int up);
uint16_t or_next_bf16(uint16_t bits, int up);
/* Array forms of the building blocks, for tests over many inputs. */
void or_philox_blocks(uint64_t seed, uint64_t stream, uint64_t c0, uint64_t n, uint32_t *out);
void or_ln_f32_n(const float *x, float *y, uint64_t n);
void or_sincos_2pi_f32_n(const uint32_t *j24, float *s, float *c, uint64_t n);
void or_radius_f32_n(const uint32_t *k24, float *r, uint64_t n);
void or_bf16_rne_n(const uint32_t *x, uint16_t *y, uint64_t n);
uint16_t or_f16_rne(uint32_t x);                 /* fp32 bits -> IEEE half bits, round to nearest even */
void or_f16_rne_n(const uint32_t *x, uint16_t *y, uint64_t n);

/* Synthesis of elements [offset, offset + n) into out (host memory). */
int or_synth(uint64_t seed, uint64_t stream, int32_t dtype, int32_t dist,
             const or_dist_params *p, uint64_t offset, uint64_t n, void *out);
/* Synthesis of the listed elements only: out[k] = element idx[k]. */
int or_synth_at(uint64_t seed, uint64_t stream, int32_t dtype, int32_t dist,
                const or_dist_params *p, const uint64_t *idx, uint64_t n, void *out);

/* Class counts of SPECIAL elements [offset, offset + n): counts[0..4] =
 * NaN, Inf, denormal, zero, normal (the class depends on the first word only). */
int or_special_class_counts(uint64_t seed, uint64_t stream, const or_dist_params *p,
                            uint64_t offset, uint64_t n, uint64_t counts[5]);

/* Candidate derivation over the window [offset, offset + n): ref and cand
 * hold that window; index lists carry global indices and entries outside the
 * window are skipped. */
int or_perturb(uint64_t seed, uint64_t stream, int32_t dtype,
               const or_perturb_plan *plan, uint64_t offset, uint64_t n,
               const void *ref, void *cand);

/* Eq. (1) per element plus the report. */
int or_compare(const void *ref, const void *cand, uint64_t n, int32_t dtype,
               double rtol, double atol, int32_t equal_nan, or_report *r);
int or_compare_batched(const or_segment *segs, uint32_t nseg, or_report *reports);

double or_performance(double mean_latency_ms);          /* Eq. (3) */
double or_reward(int compiled, int valid, double p);    /* Eq. (4) */

#ifdef __cplusplus
}
#endif
#endif

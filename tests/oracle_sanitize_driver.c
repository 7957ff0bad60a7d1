/*
 * oracle_sanitize_driver.c -- runs every entry point of the CPU oracle over
 * edge-case sizes, offsets, types and distributions, for a build with
 * AddressSanitizer and UndefinedBehaviorSanitizer (tests/test_oracle_sanitized.py).
 *
 * Every buffer is allocated with exactly the bytes an entry point may touch,
 * so that a read or write one element too far is reported.  Results are not
 * checked here (the other oracle tests pin them); only that no call strays
 * out of bounds or reaches undefined behaviour.  Prints "ok" at the end.
 */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "sv_oracle.h"

static const size_t kItem[7] = {4, 2, 4, 2, 8, 1, 8};   /* OR_F32 .. OR_I64 */

static void *alloc(size_t bytes) {
  void *p = malloc(bytes ? bytes : 1);
  if (!p) {
    fprintf(stderr, "out of memory\n");
    exit(2);
  }
  return p;
}

static or_dist_params params_for(int dtype, int dist) {
  or_dist_params p;
  memset(&p, 0, sizeof p);
  p.a = -4.0;
  p.b = 4.0;
  p.mean = 5.0;
  p.std = 10.0;
  p.lo = dtype == OR_U8 ? 3 : -1000;
  p.hi = dtype == OR_U8 ? 250 : (dtype == OR_I64 ? (int64_t)1 << 40 : 1000);
  if (dist == OR_SPECIAL) {
    p.p_nan = 0.1;
    p.p_inf = 0.05;
    p.p_denorm = 0.1;
    p.p_zero = 0.1;
  }
  return p;
}

int main(void) {
  const uint64_t offsets[] = {0, 3, 7, 1000, ((uint64_t)1 << 40) + 3};
  const uint64_t sizes[] = {0, 1, 2, 5, 17, 33, 257};
  unsigned long calls = 0;

  /* synthesis, windows and random access */
  for (int dtype = 0; dtype < 7; ++dtype) {
    for (int dist = 0; dist < 5; ++dist) {
      const or_dist_params p = params_for(dtype, dist);
      for (size_t io = 0; io < sizeof offsets / sizeof offsets[0]; ++io) {
        for (size_t in = 0; in < sizeof sizes / sizeof sizes[0]; ++in) {
          const uint64_t n = sizes[in];
          void *out = alloc(n * kItem[dtype]);
          (void)or_synth(11, 5, dtype, dist, &p, offsets[io], n, out);
          uint64_t *idx = alloc(n * sizeof *idx);
          for (uint64_t k = 0; k < n; ++k) idx[k] = offsets[io] + (k * 7919u) % (n + 3);
          (void)or_synth_at(11, 5, dtype, dist, &p, idx, n, out);
          free(idx);
          free(out);
          calls += 2;
        }
      }
    }
  }
  {
    const or_dist_params p = params_for(OR_F32, OR_SPECIAL);
    uint64_t counts[5];
    for (size_t in = 0; in < sizeof sizes / sizeof sizes[0]; ++in)
      (void)or_special_class_counts(3, 4, &p, 9, sizes[in], counts);
  }

  /* candidate derivation and the check, every type */
  for (int dtype = 0; dtype < 7; ++dtype) {
    const int dist = (dtype == OR_I32 || dtype == OR_U8 || dtype == OR_I64) ? OR_INT_RANGE : OR_SPECIAL;
    const or_dist_params p = params_for(dtype, dist);
    for (size_t in = 0; in < sizeof sizes / sizeof sizes[0]; ++in) {
      const uint64_t n = sizes[in], off = 5;
      void *ref = alloc(n * kItem[dtype]);
      void *cand = alloc(n * kItem[dtype]);
      (void)or_synth(21, 2, dtype, dist, &p, off, n, ref);
      uint64_t idx[4] = {off, off + n / 2, off + n + 10, 0};   /* inside, inside, past the window, before it */
      for (int op = OR_OP_COPY; op <= OR_OP_FAULT_AT; ++op) {
        or_perturb_plan plan;
        memset(&plan, 0, sizeof plan);
        plan.op = op;
        plan.p = 0.5;
        plan.value = 1e-3;
        plan.bits = 0x7FC00001u;
        plan.idx = idx;
        plan.nidx = n ? 4 : 0;
        if (op != OR_OP_COPY) {
          or_perturb_plan copy;
          memset(&copy, 0, sizeof copy);
          copy.op = OR_OP_COPY;
          (void)or_perturb(21, 9, dtype, &copy, off, n, ref, cand);
        }
        (void)or_perturb(21, 9, dtype, &plan, off, n, ref, cand);
        or_report r;
        (void)or_compare(ref, cand, n, dtype, 1e-5, 1e-8, 0, &r);
        (void)or_compare(ref, cand, n, dtype, 0.0, 0.0, 1, &r);
        (void)or_compare(cand, ref, n, dtype, 1.0, 1e300, 0, &r);
        calls += 4;
      }
      free(ref);
      free(cand);
    }
  }

  /* a batch with empty, one-element and aliased segments of mixed types */
  {
    const uint64_t n = 33;
    float *a = alloc(n * sizeof *a), *b = alloc(n * sizeof *b);
    double *c = alloc(n * sizeof *c);
    unsigned char *u = alloc(n);
    for (uint64_t k = 0; k < n; ++k) {
      a[k] = (float)k;
      b[k] = (float)k + (k % 5 == 0 ? 0.5f : 0.0f);
      c[k] = (double)k * 1e-310;
      u[k] = (unsigned char)k;
    }
    or_segment segs[6] = {
        {a, b, n, OR_F32, 1e-5, 0.0, 0},
        {a, a, 0, OR_F32, 0.0, 0.0, 0},
        {b, a, 1, OR_F32, 0.0, 0.0, 1},
        {c, c, n, OR_F64, 0.0, 0.0, 0},
        {u, u + 1, n - 1, OR_U8, 0.0, 0.0, 0},
        {NULL, NULL, 0, OR_I64, 0.0, 0.0, 0},
    };
    or_report reps[6];
    (void)or_compare_batched(segs, 6, reps);
    free(a);
    free(b);
    free(c);
    free(u);
  }

  /* building blocks, array forms over exact-size buffers */
  {
    const uint64_t n = 1000;
    float *x = alloc(n * sizeof *x), *y = alloc(n * sizeof *y), *z = alloc(n * sizeof *z);
    uint32_t *w = alloc(n * sizeof *w);
    uint16_t *h = alloc(n * sizeof *h);
    uint32_t *blocks = alloc(4 * n * sizeof *blocks);
    for (uint64_t k = 0; k < n; ++k) {
      x[k] = 1e-30f + (float)k * 0.37f;
      w[k] = (uint32_t)(k * 2654435761u);
    }
    or_ln_f32_n(x, y, n);
    for (uint64_t k = 0; k < n; ++k) w[k] &= 0xFFFFFFu;
    or_sincos_2pi_f32_n(w, y, z, n);
    or_radius_f32_n(w, y, n);
    for (uint64_t k = 0; k < n; ++k) w[k] = (uint32_t)(k * 2654435761u);
    or_bf16_rne_n(w, h, n);
    or_f16_rne_n(w, h, n);
    or_philox_blocks(7, 8, ((uint64_t)1 << 62) - 3, n, blocks);
    float s[256], cc[256];
    or_sincos_table(s, cc);
    for (uint64_t k = 0; k < n; ++k) {
      (void)or_next_f32(w[k], (int)(k & 1));
      (void)or_next_bf16((uint16_t)w[k], (int)(k & 1));
    }
    float zc, zs;
    or_box_muller_f32(0xFFFFFFFFu, 0, &zc, &zs);
    or_box_muller_f32(0, 0xFFFFFFFFu, &zc, &zs);
    free(x);
    free(y);
    free(z);
    free(w);
    free(h);
    free(blocks);
  }

  (void)or_performance(0.25);
  (void)or_reward(1, 1, 4.0);
  (void)or_reward(0, 0, 0.0);
  printf("%lu calls\nok\n", calls);
  return 0;
}

/* oracle_check.c -- the CPU oracle run under AddressSanitizer and UndefinedBehaviorSanitizer
 * (built by tests/test_host_sanitized.py; test infrastructure only). It steps tensors of every
 * tier and option through the oracle's own entry points, so that every array the oracle
 * indexes (ragged shapes, vectors, stacked slices, float32 masters, the optional outputs) is
 * checked for out-of-bounds access, and checks the clip bound of Sec. 3 on the way:
 * RMS(U) <= d (1 + 1e-6) for every tensor. */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../../oracle/skew_oracle.h"

static int fails = 0;

static uint16_t bf16_of(float f) { return skew_oracle_f32_to_bf16(f); }

/* a small linear congruential source of test values (not the method's dither) */
static uint32_t lcg = 12345u;
static float uniform_pm1(void) {
  lcg = lcg * 1664525u + 1013904223u;
  return (float)((lcg >> 8) * (1.0 / 16777216.0)) * 2.0f - 1.0f;
}

typedef struct {
  int tier, ndim;
  int64_t rows, cols, batch;
  uint32_t flags;
} shape_t;

static void run(const shape_t *sh, int ns, const skew_oracle_hparams *hp0, int steps) {
  skew_oracle_tensor *t = calloc((size_t)ns, sizeof *t);
  double *rms = calloc((size_t)ns, sizeof *rms);
  for (int k = 0; k < ns; k++) {
    const int64_t E = sh[k].ndim == 3 ? sh[k].batch : 1, n = sh[k].rows, m = sh[k].cols, N = E * n * m;
    const int fp32 = (sh[k].flags & ORACLE_STATE_FP32) != 0;
    const int exact = (sh[k].tier == ORACLE_ROUTER && !(sh[k].flags & ORACLE_STATE_FACTORED)) || sh[k].ndim == 1;
    const int mom = sh[k].tier == ORACLE_BACKBONE || (sh[k].flags & ORACLE_STATE_MOMENTUM);
    t[k].tier = sh[k].tier;
    t[k].ndim = sh[k].ndim;
    t[k].rows = n;
    t[k].cols = m;
    t[k].batch = sh[k].ndim == 3 ? E : 0;
    t[k].state_flags = sh[k].flags;
    t[k].tensor_id = (uint64_t)k;
    t[k].w = malloc((size_t)(N > 0 ? N : 1) * (fp32 ? 4 : 2));
    t[k].g = malloc((size_t)(N > 0 ? N : 1) * (fp32 ? 4 : 2));
    for (int64_t i = 0; i < N; i++) {
      if (fp32)
        ((float *)t[k].w)[i] = 0.02f * uniform_pm1();
      else
        ((uint16_t *)t[k].w)[i] = bf16_of(0.02f * uniform_pm1());
    }
    if (mom) t[k].m = calloc((size_t)(N > 0 ? N : 1), 4);
    if (exact) t[k].v = calloc((size_t)(N > 0 ? N : 1), 4);
    if (!exact) {
      t[k].r = calloc((size_t)(E * n > 0 ? E * n : 1), 4);
      t[k].c = calloc((size_t)(E * m > 0 ? E * m : 1), 4);
    }
    t[k].u_out = malloc((size_t)(N > 0 ? N : 1) * 4);
    t[k].x_out = malloc((size_t)(N > 0 ? N : 1) * 4);
    t[k].y_out = malloc((size_t)(N > 0 ? N : 1) * 4);
    t[k].rms_out = &rms[k];
  }
  for (int s = 1; s <= steps; s++) {
    for (int k = 0; k < ns; k++) {
      const int64_t E = sh[k].ndim == 3 ? sh[k].batch : 1, N = E * sh[k].rows * sh[k].cols;
      const int fp32 = (sh[k].flags & ORACLE_STATE_FP32) != 0;
      float *gf = (float *)t[k].g;
      uint16_t *gb = (uint16_t *)t[k].g;
      for (int64_t i = 0; i < N; i++) {
        const float v = (i % 7 == 3) ? 0.0f : 1e-2f * uniform_pm1();
        if (fp32)
          gf[i] = v;
        else
          gb[i] = bf16_of(v);
      }
    }
    skew_oracle_hparams hp = *hp0;
    hp.step = s;
    float gc = 0.f;
    if (skew_oracle_step_gcoef(&hp, t, ns, &gc) != 0) {
      printf("FAIL step %d refused\n", s);
      fails++;
    }
    for (int k = 0; k < ns; k++) {
      const int64_t E = sh[k].ndim == 3 ? sh[k].batch : 1, N = E * sh[k].rows * sh[k].cols;
      if (N == 0) continue;
      double ss = 0.0;
      for (int64_t i = 0; i < N; i++) ss += (double)t[k].u_out[i] * (double)t[k].u_out[i];
      const double r = sqrt(ss / (double)N);
      if (!(r <= (double)hp.clip_threshold * (1.0 + 1e-6)) || !isfinite(rms[k])) {
        printf("FAIL tensor %d step %d: RMS(U) %g, RMS(U_hat) %g\n", k, s, r, rms[k]);
        fails++;
      }
    }
  }
  for (int k = 0; k < ns; k++) {
    free(t[k].w);
    free((void *)t[k].g);
    free(t[k].m);
    free(t[k].v);
    free(t[k].r);
    free(t[k].c);
    free(t[k].u_out);
    free(t[k].x_out);
    free(t[k].y_out);
  }
  free(t);
  free(rms);
}

int main(void) {
  const shape_t shapes[] = {
      {ORACLE_BACKBONE, 2, 13, 17, 0, 0},  {ORACLE_BACKBONE, 1, 1, 4097, 0, 0}, {ORACLE_EXPERT, 2, 1, 7, 0, 0},
      {ORACLE_EXPERT, 2, 7, 1, 0, 0},      {ORACLE_EXPERT, 2, 33, 1031, 0, 0},  {ORACLE_EXPERT, 3, 5, 9, 4, 0},
      {ORACLE_EXPERT, 3, 0, 9, 2, 0},      {ORACLE_EXPERT, 2, 0, 5, 0, 0},      {ORACLE_ROUTER, 2, 256, 8, 0, 0},
      {ORACLE_ROUTER, 2, 64, 8, 0, ORACLE_STATE_FACTORED},
      {ORACLE_EXPERT, 2, 64, 40, 0, ORACLE_STATE_MOMENTUM},
      {ORACLE_ROUTER, 2, 16, 8, 0, ORACLE_STATE_FP32},
      {ORACLE_BACKBONE, 1, 1, 77, 0, ORACLE_STATE_FP32},
  };
  const int ns = (int)(sizeof shapes / sizeof shapes[0]);
  skew_oracle_hparams hp;
  memset(&hp, 0, sizeof hp);
  hp.lr = 3e-4f;
  hp.beta1 = 0.9f;
  hp.beta2 = 0.999f;
  hp.eps = 1e-8f;
  hp.clip_threshold = 1.0f;
  hp.gsq_total = -1.0;
  run(shapes, ns, &hp, 4);
  hp.weight_decay = 0.05f;
  hp.max_grad_norm = 1e-3f;
  hp.exact_ulp = 1;
  hp.clip_threshold = 0.5f;
  run(shapes, ns, &hp, 3);
  hp.rbar_min_only = 1;
  hp.gsq_total = 2.0;
  run(shapes, ns, &hp, 2);
  if (fails) {
    printf("%d oracle checks failed\n", fails);
    return 1;
  }
  printf("oracle under sanitizers: all steps clean\n");
  return 0;
}

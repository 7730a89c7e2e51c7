/*
 * skew_oracle.h -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-source CPU oracle of one SkewAdam optimizer step
 * (Sec. 3 "SkewAdam: tiered state allocation", Eq. 1, Alg. 1). It exists to
 * check the GPU library; only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load it. It shares no code, header or
 * constant with the GPU library.
 *
 * Arithmetic: float32 as the paper's step is "computed in float32" (Sec. 3,
 * "Update clipping and low-precision updates"); every reduction is carried in
 * double in ascending index order and rounded to float once.
 */
#ifndef SKEW_ORACLE_H
#define SKEW_ORACLE_H
#include <stdint.h>
#ifdef __cplusplus
extern "C" {
#endif

enum { ORACLE_BACKBONE = 0, ORACLE_EXPERT = 1, ORACLE_ROUTER = 2 };

typedef struct {
  int32_t tier;       /* ORACLE_BACKBONE / ORACLE_EXPERT / ORACLE_ROUTER */
  int32_t ndim;       /* 1 = vector, 2 = matrix */
  int64_t rows, cols; /* dense row-major, rows*cols elements */
  uint64_t tensor_id; /* keys the dither */
  void *w;            /* bf16 bits (float with ORACLE_STATE_FP32), updated in place */
  const void *g;      /* bf16 bits (float with ORACLE_STATE_FP32) */
  float *m;           /* momentum [rows*cols] (backbone) or NULL */
  float *v;           /* exact second moment [rows*cols] (router, vectors) or NULL */
  float *r;           /* factored row statistic [rows] or NULL */
  float *c;           /* factored column statistic [cols] or NULL */
  float *u_out;       /* optional [rows*cols]: the clipped update U */
  float *x_out;       /* optional [rows*cols]: W - lr*U before the dither */
  float *y_out;       /* optional [rows*cols]: the float value handed to the bf16 cast */
  double *rms_out;    /* optional: RMS of the unclipped update of this tensor */
  int64_t batch;      /* ndim 3: E >= 1 stacked rows x cols matrices (w, g, m, v [E][rows][cols],
                         r [E][rows], c [E][cols]), factored per slice, one clip over all;
                         0 or 1 otherwise */
  uint32_t state_flags; /* ORACLE_STATE_*: tier variants of the ablation (Table 3) */
} skew_oracle_tensor;

/* Tier variants (Table 3): momentum kept in any tier; router matrices factored; float32
 * master weights and gradients (w, g point at float) for exact-moment tensors, updated in
 * float32 without the dithered cast (the paper's fp32 router and norms, Sec. 4, Table 5). */
enum { ORACLE_STATE_MOMENTUM = 1, ORACLE_STATE_FACTORED = 2, ORACLE_STATE_FP32 = 4 };

typedef struct {
  float lr, beta1, beta2, eps, clip_threshold;
  int64_t step;  /* t >= 1 */
  uint64_t seed;
  float weight_decay;   /* lambda >= 0: decoupled decay in float32 ahead of the dithered cast
                           (Sec. 3 footnote, Sec. 6); the router tier takes none (Table 5) */
  float max_grad_norm;  /* > 0: the gradients of all n tensors are first scaled by
                           min(1, max_grad_norm / (||G||_2 + 1e-6)) (Sec. 4); 0: off */
  double gsq_total;     /* < 0: ||G||_2^2 is summed over the n tensors given; >= 0: its value
                           (a step over a sample of a larger set passes the set's sum) */
  int32_t exact_ulp;    /* 1: the dither spans the exact bf16 ulp of w, xi ~ U(+-ulp(w)/2), in
                           place of the approximation ulp(w) ~ 2^-7 |w| (Sec. 3) */
  int32_t rbar_min_only; /* 1: the other reading of Alg. 1's "eps-clamps" of the factored
                           reconstruction, for a sensitivity check only: mean(R) is guarded
                           at FLT_MIN (against 0/0) instead of being clamped at eps; the
                           clamp max(R_i c'_j, eps) stays. 0: the reading both the oracle and
                           the GPU library take (mean(R) clamped at eps). */
} skew_oracle_hparams;

/* One step over n tensors. Returns 0, -1 when step < 1, -2 when a tensor asks for float32
 * masters but keeps a factored second moment. When gcoef_out is not NULL it receives the
 * gradient scale of the step (1 without max_grad_norm). */
int skew_oracle_step(const skew_oracle_hparams *hp, skew_oracle_tensor *t, int n);
int skew_oracle_step_gcoef(const skew_oracle_hparams *hp, skew_oracle_tensor *t, int n, float *gcoef_out);

/* Pieces exposed for pinning. */
uint16_t skew_oracle_f32_to_bf16(float f);
void skew_oracle_f32_to_bf16_array(const float *x, uint16_t *out, int64_t n);
uint64_t skew_oracle_mix64(uint64_t z);
uint32_t skew_oracle_fmix32(uint32_t h);
uint64_t skew_oracle_key(uint64_t seed, int64_t step, uint64_t tensor_id);
uint32_t skew_oracle_u16(uint64_t key, uint64_t idx);
void skew_oracle_u16_array(uint64_t key, uint64_t idx0, int64_t n, uint32_t *out);
int skew_oracle_threads(void);
/* Sum of squares of n bf16 values in double (squares of bf16 values are exact in double):
 * the squared gradient norm of a whole set, for steps over a sample of it (gsq_total). */
double skew_oracle_sumsq_bf16(const uint16_t *g, int64_t n);
/* Sets the OpenMP thread count of later steps (results do not depend on it). */
void skew_oracle_set_threads(int n);

#ifdef __cplusplus
}
#endif
#endif

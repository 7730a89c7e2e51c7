/*
 * skew_oracle.c -- TEST INFRASTRUCTURE ONLY (see skew_oracle.h).
 *
 * One SkewAdam step, written out in the order of Alg. 1 with plain loops.
 * Build: -O2 -ffp-contract=off -fno-fast-math, so that every float operation
 * below is one IEEE-754 binary32 operation and the only fused multiply-adds
 * are the explicit fmaf() calls. OpenMP splits independent rows (or column
 * ranges); every sum keeps its ascending index order, so the result does not
 * depend on the thread count.
 *
 * Step definition (all scalars float32 unless noted; N = rows*cols; idx = i*cols + j):
 *   host scalars, in double then rounded once:  a1 = 1-b1, a2 = 1-b2,
 *       s_m = sqrt(1-b2^t)/(1-b1^t)  (backbone bias correction, Alg. 1),
 *       s_0 = sqrt(1-b2^t)           (momentum-free tiers, Alg. 1)
 *   factored tensors (matrix, tier != router), Eq. 1 and the rank-one
 *   reconstruction that follows it:
 *       r_i = mean_j g_ij^2, c_j = mean_i g_ij^2   (double, rounded once)
 *       R_i <- fmaf(a2, r_i, b2*R_i);  C_j <- fmaf(a2, c_j, b2*C_j)
 *       Rbar = mean_i R_i (double, rounded once);  c'_j = C_j / max(Rbar, eps)
 *       D_ij = sqrt(max(R_i * c'_j, eps))
 *   exact tensors (router tier, or any vector), Alg. 1:
 *       V <- fmaf(a2, g*g, b2*V);  D = sqrt(max(V, eps))
 *   backbone: M <- fmaf(a1, g, b1*M);  Uhat = (s_m*M) / D
 *   others:   Uhat = (s_0*g) / D
 *   clip (Sec. 3, Alg. 1): k = 1 / max(1, RMS(Uhat)/d) with RMS over all N
 *       (sum of squares in double);  U = Uhat*k
 *   write-back (Sec. 3, Alg. 1): x = fmaf(-lr, U, w)
 *       xi = e * 2^-24 * |w|, e = 2*u16 + 1 - 2^16  (uniform on +-ulp(w)/2 with
 *       ulp(w) taken as 2^-7|w|, on a 2^-16 grid), added with one rounding:
 *       y = fmaf(e*2^-24, |w|, x);  W' = bf16 round-to-nearest-even(y)
 *   max() here propagates NaN (as torch.clamp does), so non-finite gradients
 *   reach the weights instead of being floored away.
 * Tier variants (Table 3) switch momentum on in any tier (then s_m applies) and the
 * factored second moment on for router matrices. A stacked tensor of E matrices
 * (ndim 3) is factored per slice, each slice with its own R, C and mean(R); the clip,
 * the dither's element index and N run over the whole tensor.
 */
#include "skew_oracle.h"
#include <float.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define COL_BLOCK 256

typedef struct {
  float b1, a1, b2, a2, eps, d, lr, s_m, s_0;
  int64_t step;
  uint64_t seed;
  float wd;       /* lr * lambda, rounded once; 0: no decay */
  int gclip;      /* gradient-norm scaling on */
  float gcoef;    /* the gradient scale c (1 when off) */
  double gc2;     /* c * c, exact in double */
  int exact_ulp;  /* dither width from the exact bf16 ulp of w */
  int rbar_min_only;  /* mean(R) guarded at FLT_MIN only (the other reading of the eps-clamps) */
} consts_t;

/* a gradient or weight element: bf16 bits, or float32 for float32 masters */
static float elem_f32(const void *p, int64_t idx, int fp32);

static float bf16_bits_to_f32(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return f;
}

static float elem_f32(const void *p, int64_t idx, int fp32) {
  return fp32 ? ((const float *)p)[idx] : bf16_bits_to_f32(((const uint16_t *)p)[idx]);
}

/* the spacing of bf16 values around w: 2^(E - 134) for biased exponent E >= 1 (8 bits of
 * significand), 2^-133 among the subnormals; exact in float */
static float bf16_ulp(float w) {
  uint32_t u;
  memcpy(&u, &w, sizeof u);
  const int E = (int)((u >> 23) & 0xFF);
  return ldexpf(1.0f, (E >= 1 ? E : 1) - 134);
}

/* round-to-nearest, ties-to-even, from float32 to the upper 16 bits; NaN -> 0x7FC0 */
uint16_t skew_oracle_f32_to_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  if (f != f) return 0x7FC0;
  uint32_t keep = u >> 16, drop = u & 0xFFFFu;
  if (drop > 0x8000u || (drop == 0x8000u && (keep & 1u))) keep += 1u;
  return (uint16_t)keep;
}

void skew_oracle_f32_to_bf16_array(const float *x, uint16_t *out, int64_t n) {
  for (int64_t i = 0; i < n; i++) out[i] = skew_oracle_f32_to_bf16(x[i]);
}

/* SplitMix64 output mixing function (Steele, Lea and Flood, OOPSLA 2014). */
static uint64_t splitmix64_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

/* MurmurHash3 32-bit finalizer (Appleby, public domain). */
static uint32_t murmur3_fmix32(uint32_t h) {
  h ^= h >> 16;
  h *= 0x85EBCA6Bu;
  h ^= h >> 13;
  h *= 0xC2B2AE35u;
  h ^= h >> 16;
  return h;
}

uint64_t skew_oracle_mix64(uint64_t z) { return splitmix64_mix(z); }
uint32_t skew_oracle_fmix32(uint32_t h) { return murmur3_fmix32(h); }

/* per-(seed, step, tensor) dither key */
uint64_t skew_oracle_key(uint64_t seed, int64_t step, uint64_t tensor_id) {
  uint64_t k = splitmix64_mix(seed);
  k = splitmix64_mix(k ^ (uint64_t)step);
  return splitmix64_mix(k ^ tensor_id);
}

/* 16 uniform bits for element idx: one 32-bit hash per element pair (idx>>1);
 * the even element takes the low half, the odd element the high half. */
uint32_t skew_oracle_u16(uint64_t key, uint64_t idx) {
  uint64_t pair = idx >> 1;
  uint32_t hi = murmur3_fmix32((uint32_t)(pair >> 32) ^ (uint32_t)(key >> 32));
  uint32_t h = murmur3_fmix32((uint32_t)pair ^ (uint32_t)key ^ hi);
  return (idx & 1u) ? (h >> 16) : (h & 0xFFFFu);
}

void skew_oracle_u16_array(uint64_t key, uint64_t idx0, int64_t n, uint32_t *out) {
  for (int64_t i = 0; i < n; i++) out[i] = skew_oracle_u16(key, idx0 + (uint64_t)i);
}

int skew_oracle_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

double skew_oracle_sumsq_bf16(const uint16_t *g, int64_t n) {
  /* fixed chunks summed in order, each chunk in ascending index order */
  const int64_t chunk = 1 << 20, nc = (n + chunk - 1) / chunk;
  double *part = (double *)calloc((size_t)(nc > 0 ? nc : 1), sizeof(double));
#pragma omp parallel for schedule(static)
  for (int64_t c = 0; c < nc; c++) {
    const int64_t e = (c + 1) * chunk < n ? (c + 1) * chunk : n;
    double s = 0.0;
    for (int64_t i = c * chunk; i < e; i++) {
      const double v = bf16_bits_to_f32(g[i]);
      s += v * v;
    }
    part[c] = s;
  }
  double total = 0.0;
  for (int64_t c = 0; c < nc; c++) total += part[c];
  free(part);
  return total;
}

void skew_oracle_set_threads(int n) {
#ifdef _OPENMP
  if (n >= 1) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

static float max_nan(float a, float b) { return (a != a) ? a : (a < b ? b : a); }

/* Eq. 1 and the rank-one reconstruction for one n x m matrix (one slice of a stacked
 * tensor): updates R [n] and C [m] in place and writes c'_j = C_j / max(mean R, eps). */
static void factored_stats(const consts_t *K, const uint16_t *g, float *R, float *C, int64_t n, int64_t m,
                           float *cprime) {
  /* rows: mean over columns of G*G, then the EMA of R */
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; i++) {
    double s = 0.0;
    for (int64_t j = 0; j < m; j++) {
      double gv = bf16_bits_to_f32(g[i * m + j]);
      s += gv * gv;
    }
    /* with gradient-norm scaling the statistic is c^2 times the exact sum */
    float ri = (float)((K->gclip ? K->gc2 * s : s) / (double)m);
    R[i] = fmaf(K->a2, ri, K->b2 * R[i]);
  }
  /* columns: mean over rows of G*G (each column summed in row order) */
  double *cs = (double *)calloc((size_t)m, sizeof(double));
#pragma omp parallel for schedule(static)
  for (int64_t jb = 0; jb < m; jb += COL_BLOCK) {
    int64_t je = jb + COL_BLOCK < m ? jb + COL_BLOCK : m;
    for (int64_t i = 0; i < n; i++)
      for (int64_t j = jb; j < je; j++) {
        double gv = bf16_bits_to_f32(g[i * m + j]);
        cs[j] += gv * gv;
      }
  }
  for (int64_t j = 0; j < m; j++) {
    float cj = (float)((K->gclip ? K->gc2 * cs[j] : cs[j]) / (double)n);
    C[j] = fmaf(K->a2, cj, K->b2 * C[j]);
  }
  free(cs);
  /* rank-one reconstruction V = R C^T / mean(R), with the mean clamped at eps */
  double sr = 0.0;
  for (int64_t i = 0; i < n; i++) sr += (double)R[i];
  float rbar = (float)(sr / (double)n);
  float q = max_nan(rbar, K->rbar_min_only ? FLT_MIN : K->eps);
  for (int64_t j = 0; j < m; j++) cprime[j] = C[j] / q;
}

static void step_tensor(const consts_t *K, skew_oracle_tensor *T) {
  /* a stacked tensor is E slices of rows x cols; row ii of the stacked rows is row
     ii % rows of slice ii / rows, and r holds the slices' R one after the other */
  const int64_t E = (T->ndim == 3 && T->batch > 0) ? T->batch : 1;
  const int64_t n1 = T->rows, m = T->cols, n = E * n1, N = n * m;
  if (n1 <= 0 || m <= 0) return;
  const int exact = (T->tier == ORACLE_ROUTER && !(T->state_flags & ORACLE_STATE_FACTORED)) || (T->ndim == 1);
  const int fp32 = (T->state_flags & ORACLE_STATE_FP32) != 0;   /* float32 w and g (exact tensors) */
  const int momentum = (T->tier == ORACLE_BACKBONE) || (T->state_flags & ORACLE_STATE_MOMENTUM);
  float *uhat = (float *)malloc((size_t)N * sizeof(float));
  double *row_ss = (double *)malloc((size_t)n * sizeof(double));
  float *cprime = NULL;

  if (!exact) {
    cprime = (float *)malloc((size_t)(E * m) * sizeof(float));
    for (int64_t e = 0; e < E; e++)
      factored_stats(K, (const uint16_t *)T->g + e * n1 * m, T->r + e * n1, T->c + e * m, n1, m, cprime + e * m);
  }

  /* preconditioned update and its sum of squares, row by row */
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; i++) {
    double s = 0.0;
    for (int64_t j = 0; j < m; j++) {
      const int64_t idx = i * m + j;
      float g = elem_f32(T->g, idx, fp32);
      if (K->gclip) g = K->gcoef * g;   /* the scaled gradient, rounded once */
      float dd;
      if (exact) {
        T->v[idx] = fmaf(K->a2, g * g, K->b2 * T->v[idx]);
        dd = sqrtf(max_nan(T->v[idx], K->eps));
      } else {
        float vhat = T->r[i] * cprime[(i / n1) * m + j];
        dd = sqrtf(max_nan(vhat, K->eps));
      }
      float num;
      if (momentum) {
        T->m[idx] = fmaf(K->a1, g, K->b1 * T->m[idx]);
        num = K->s_m * T->m[idx];
      } else {
        num = K->s_0 * g;
      }
      const float u = num / dd;
      uhat[idx] = u;
      s += (double)u * (double)u;
    }
    row_ss[i] = s;
  }
  double ss = 0.0;
  for (int64_t i = 0; i < n; i++) ss += row_ss[i];

  /* update clipping to RMS d */
  const double rms = sqrt(ss / (double)N);
  if (T->rms_out) *T->rms_out = rms;
  const double ratio = rms / (double)K->d;
  const double den = (ratio != ratio) ? ratio : (ratio < 1.0 ? 1.0 : ratio);
  const float kclip = (float)(1.0 / den);

  /* dithered bf16 write-back */
  const uint64_t key = skew_oracle_key(K->seed, K->step, T->tensor_id);
  const int decay = K->wd != 0.0f && T->tier != ORACLE_ROUTER;
#pragma omp parallel for schedule(static)
  for (int64_t idx = 0; idx < N; idx++) {
    const float w = elem_f32(T->w, idx, fp32);
    const float U = uhat[idx] * kclip;
    /* decoupled weight decay, w - (lr lambda) w with one rounding, ahead of the update */
    const float wdec = decay ? fmaf(-K->wd, w, w) : w;
    const float x = fmaf(-K->lr, U, wdec);
    if (T->u_out) T->u_out[idx] = U;
    if (T->x_out) T->x_out[idx] = x;
    if (fp32) {   /* float32 master: no cast, no dither */
      if (T->y_out) T->y_out[idx] = x;
      ((float *)T->w)[idx] = x;
      continue;
    }
    const int32_t e = 2 * (int32_t)skew_oracle_u16(key, (uint64_t)idx) + 1 - 65536;
    float y;
    if (K->exact_ulp) {
      /* xi = (e * 2^-17) * ulp(w), uniform on +-ulp(w)/2 on a 2^-16 grid; the product is exact */
      y = fmaf((float)e * 0x1p-17f, bf16_ulp(w), x);
    } else {
      y = fmaf((float)e * 0x1p-24f, fabsf(w), x);
    }
    if (T->y_out) T->y_out[idx] = y;
    ((uint16_t *)T->w)[idx] = skew_oracle_f32_to_bf16(y);
  }
  free(cprime);
  free(row_ss);
  free(uhat);
}

int skew_oracle_step(const skew_oracle_hparams *hp, skew_oracle_tensor *t, int n) {
  return skew_oracle_step_gcoef(hp, t, n, NULL);
}

int skew_oracle_step_gcoef(const skew_oracle_hparams *hp, skew_oracle_tensor *t, int n, float *gcoef_out) {
  if (hp->step < 1) return -1;
  for (int i = 0; i < n; i++) {
    const int exact = (t[i].tier == ORACLE_ROUTER && !(t[i].state_flags & ORACLE_STATE_FACTORED)) || t[i].ndim == 1;
    if ((t[i].state_flags & ORACLE_STATE_FP32) && !exact) return -2;
  }
  consts_t K;
  const double b1 = hp->beta1, b2 = hp->beta2, tt = (double)hp->step;
  K.b1 = hp->beta1;
  K.a1 = (float)(1.0 - b1);
  K.b2 = hp->beta2;
  K.a2 = (float)(1.0 - b2);
  K.eps = hp->eps;
  K.d = hp->clip_threshold;
  K.lr = hp->lr;
  K.s_m = (float)(sqrt(1.0 - pow(b2, tt)) / (1.0 - pow(b1, tt)));
  K.s_0 = (float)sqrt(1.0 - pow(b2, tt));
  K.step = hp->step;
  K.seed = hp->seed;
  K.wd = (float)((double)hp->lr * (double)hp->weight_decay);
  K.exact_ulp = hp->exact_ulp != 0;
  K.rbar_min_only = hp->rbar_min_only != 0;
  K.gclip = hp->max_grad_norm > 0.0f;
  K.gcoef = 1.0f;
  if (K.gclip) {
    /* global 2-norm over every element of every tensor, in double, in order */
    double total = 0.0;
    for (int i = 0; i < n && hp->gsq_total < 0.0; i++) {
      const int64_t E = (t[i].ndim == 3 && t[i].batch > 0) ? t[i].batch : 1;
      const int64_t N = E * t[i].rows * t[i].cols;
      for (int64_t idx = 0; idx < N; idx++) {
        const double gv = elem_f32(t[i].g, idx, (t[i].state_flags & ORACLE_STATE_FP32) != 0);
        total += gv * gv;
      }
    }
    if (hp->gsq_total >= 0.0) total = hp->gsq_total;
    double c = (double)hp->max_grad_norm / (sqrt(total) + 1e-6);
    if (c > 1.0) c = 1.0;   /* NaN stays NaN */
    K.gcoef = (float)c;
  }
  K.gc2 = (double)K.gcoef * (double)K.gcoef;
  if (gcoef_out) *gcoef_out = K.gcoef;
  for (int i = 0; i < n; i++) step_tensor(&K, &t[i]);
  return 0;
}

/*
 * skewadam.h -- C ABI of the SkewAdam optimizer step for AMD Instinct MI355X (gfx950).
 *
 * One call to skew_step() applies one SkewAdam step (Sec. 3 "SkewAdam: tiered
 * state allocation", Eq. 1, Alg. 1) to every tensor of a descriptor table.
 * Each tensor gets the state of its tier (Fig. 1; Sec. 3 "The tiers"):
 *   BACKBONE matrix : fp32 momentum M [rows*cols] + factored second moment R [rows], C [cols]
 *   BACKBONE vector : fp32 momentum M + exact second moment V [len]
 *   EXPERT   matrix : factored second moment R, C only
 *   EXPERT   vector : exact V
 *   ROUTER   (any)  : exact V [rows*cols]
 * Every tier then clips its update to RMS <= clip_threshold (Sec. 3 "Update
 * clipping"; Alg. 1) and writes the weight back as bf16 through a dithered
 * round-to-nearest-even cast (Sec. 3 "Update clipping and low-precision
 * updates"; Alg. 1).
 *
 * Conventions
 *  - Every function returns an int status: SKEW_OK (0) or a negative SKEW_E* code.
 *    Nothing aborts or throws. A call that fails validation launches nothing.
 *  - "device" pointers are HIP device allocations on the current device;
 *    "host" pointers are ordinary host memory. The caller owns all of them.
 *  - Streams are hipStream_t values passed as void* (NULL = the default stream).
 *    skew_state_init and skew_step are stream-ordered and never synchronise the
 *    device, except skew_state_init, which waits for its own table upload. Every
 *    kernel of a step runs on the caller's stream.
 *  - bf16 is IEEE binary32 truncated to its upper 16 bits (the bfloat16 format).
 *  - Sizes and element indices are 64-bit throughout (tensors of >= 2^31 elements).
 */
#ifndef SKEWADAM_H
#define SKEWADAM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SKEW_ABI_VERSION 4

enum {
  SKEW_OK = 0,
  SKEW_EINVAL = -1,    /* bad argument: tier, ndim, shape, ld, NULL pointer, hyper-parameter */
  SKEW_ENOSPACE = -2,  /* a caller buffer is smaller than skew_state_bytes() asked for */
  SKEW_EHIP = -3,      /* the HIP runtime reported an error (launch, copy, memset) */
  SKEW_ENOMEM = -4,    /* host allocation of the context failed */
  SKEW_ESTALE = -5,    /* skew_step on a context whose static workspace a newer
                          skew_state_init_static on the same GPU has taken over */
  SKEW_ETOOBIG = -6    /* skew_state_init_static: the table needs more workspace than
                          SKEW_STATIC_WORKSPACE_BYTES */
};

/* Bytes of the library's static workspace (skew_state_init_static), per GPU. */
#define SKEW_STATIC_WORKSPACE_BYTES (64u << 20)

enum { SKEW_TIER_BACKBONE = 0, SKEW_TIER_EXPERT = 1, SKEW_TIER_ROUTER = 2 };

enum { SKEW_FLAG_EXACT_CLIP = 1, SKEW_FLAG_EXACT_ULP = 2 };

/* Per-tensor state variants (the tier ablation, Table 3): SKEW_STATE_MOMENTUM keeps fp32
 * momentum in any tier (then the bias correction of the backbone applies);
 * SKEW_STATE_FACTORED gives router matrices the factored second moment. Vectors always
 * keep the exact one (Alg. 1). "+ momentum on experts" is MOMENTUM on the expert tensors,
 * "factored router" FACTORED on the router, "uniform" both on every tensor.
 * SKEW_STATE_FP32: w and g are float32 (the paper's fp32 norms and router, Table 5),
 * updated in float32 with no dither and no cast; only for tensors with the exact second
 * moment (vectors, unfactored router matrices), else SKEW_EINVAL. */
enum { SKEW_STATE_MOMENTUM = 1, SKEW_STATE_FACTORED = 2, SKEW_STATE_FP32 = 4 };

/* One parameter tensor (Sec. 3 "The tiers": the policy assigns state by parameter role).
 *   tier      SKEW_TIER_*.
 *   ndim      2 = matrix (row-major, `rows` x `cols`, row stride `ld` elements);
 *             1 = vector of rows*cols elements (one of rows, cols must be 1), contiguous;
 *             3 = `batch` stacked matrices of `rows` x `cols` (slice stride rows*ld
 *             elements), factored along the last two axes, each slice with its own R, C
 *             and mean(R) (Sec. 3 footnote); the clip factor, N and the dither's element
 *             index (e*rows*cols + i*cols + j) run over the whole tensor.
 *             Matrices outside the router tier take the factored second moment (Eq. 1);
 *             the router and every vector take the exact one (Alg. 1).
 *   rows, cols  >= 0. A tensor with no elements is accepted and skipped.
 *   ld        row stride in elements, >= cols (ignored for vectors).
 *   tensor_id caller-chosen, stable across runs and checkpoints; keys the dither, so
 *             two tensors should not share an id.
 *   w         device, bf16 [rows x ld] (float32 with SKEW_STATE_FP32), read and written in
 *             place by skew_step.
 *   g         device, bf16 [rows x ld] (float32 with SKEW_STATE_FP32), read only.
 *   m, v, r, c  OUT: filled by skew_state_init with pointers into the caller's state
 *             buffer (NULL where the tier keeps no such state); dense, row-major:
 *             m, v [rows*cols] (element (i, j) at i*cols + j), r [rows], c [cols];
 *             stacked: m, v [batch][rows][cols], r [batch][rows], c [batch][cols].
 *   batch     ndim 3: the number of slices (>= 0; 0 = no elements); otherwise 0 or 1.
 *   state_flags  0 or SKEW_STATE_* bits (tier variants, Table 3).
 * w and g may have any alignment; 16-byte-aligned rows (w, g aligned and ld a
 * multiple of 8) take the vectorised path. */
typedef struct skew_tensor_desc {
  int32_t tier;
  int32_t ndim;
  int64_t rows;
  int64_t cols;
  int64_t ld;
  uint64_t tensor_id;
  void *w;
  const void *g;
  float *m;
  float *v;
  float *r;
  float *c;
  int64_t batch;
  uint32_t state_flags;
  uint32_t reserved;
} skew_tensor_desc;

/* Hyper-parameters of one step (Alg. 1; defaults of Table 5: lr 3e-4,
 * beta = (0.9, 0.999), eps 1e-8; clip threshold 1 from Sec. 3).
 *   lr              eta_t, the caller's schedule value for this step (finite).
 *   beta1, beta2    in [0, 1).
 *   eps             > 0: floor of the second moment, and of mean(R) in the
 *                   factored reconstruction.
 *   clip_threshold  d > 0 (may be +inf: no clipping): U <- U / max(1, RMS(U)/d).
 *   flags           0 or a combination of:
 *                   SKEW_FLAG_EXACT_CLIP: always recompute the sum of squares behind
 *                   the clip factor with the reference float sequence (by default it is
 *                   recomputed only when a faster estimate cannot decide its rounding);
 *                   SKEW_FLAG_EXACT_ULP: the dither spans the exact bf16 ulp of w,
 *                   xi = (e 2^-17) ulp(w), in place of the approximation ulp(w) ~ 2^-7 |w|
 *                   of Sec. 3: unbiased stochastic rounding.
 *   step            t >= 1, the caller's step counter (the library keeps none).
 *   seed            dither seed; with (step, tensor_id, element index) it fixes
 *                   every dither value, so results are bit-reproducible.
 *   weight_decay    lambda >= 0 (finite): decoupled weight decay fused into the float32
 *                   update ahead of the dithered cast, x = fma(-lr, U, w - (lr lambda) w),
 *                   with lr*lambda rounded once to float (Sec. 3 footnote, Sec. 6; Table 5:
 *                   0.05). The router tier takes none. 0: off, bit-identical to no decay.
 *   max_grad_norm   >= 0 (finite); > 0 scales every gradient of the table by
 *                   c = min(1, max_grad_norm / (||G||_2 + 1e-6)), the norm taken over all
 *                   tensors of the table (the trainer's clipping at 1.0, Sec. 4), before
 *                   the step: elementwise terms use fl(c g), the factored statistics c^2
 *                   times the exact sums of g^2. 0: off. */
typedef struct skew_hparams {
  float lr;
  float beta1;
  float beta2;
  float eps;
  float clip_threshold;
  int32_t flags;
  int64_t step;
  uint64_t seed;
  float weight_decay;
  float max_grad_norm;
} skew_hparams;

typedef struct skew_ctx skew_ctx;

/* Sizes of the two caller-owned device buffers for a descriptor table (Eq. 2:
 * S = 4[N_bb + sum(n_W + m_W) + N_rt] bytes, plus the exact v of vectors as in
 * Table 6; each state slice is padded to 256 bytes).
 *   d, n              host array of n >= 0 descriptors (only shape fields are read).
 *   state_bytes       OUT: bytes of fp32 state (>= the closed form).
 *   workspace_bytes   OUT: bytes of scratch the library needs (tables and partial sums).
 * Host only; needs no GPU. Errors: SKEW_EINVAL. */
int skew_state_bytes(const skew_tensor_desc *d, int n, size_t *state_bytes, size_t *workspace_bytes);

/* Create a context for the table d[0..n).
 *   ctx         OUT: the new context (host object) or NULL on error.
 *   d           host array; its m, v, r, c fields are filled in (see above).
 *   state       device buffer of >= skew_state_bytes() bytes; carved into the state
 *               slices and zero-filled on `stream`. It holds every byte of optimizer
 *               state: saving it with the step counter and seed is a checkpoint, and
 *               copying it back after a new skew_state_init() on an identical table
 *               resumes bit-exactly.
 *   workspace   device buffer of >= workspace_bytes; zero-filled on `stream`; the library
 *               owns its contents until skew_destroy().
 *   stream      hipStream_t as void*.
 * All pointers must stay valid and unchanged until skew_destroy(); to change them,
 * destroy and init again. Errors: SKEW_EINVAL, SKEW_ENOSPACE, SKEW_ENOMEM, SKEW_EHIP. */
int skew_state_init(skew_ctx **ctx, skew_tensor_desc *d, int n, void *state, size_t state_bytes,
                    void *workspace, size_t workspace_bytes, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): skew_state_init with the library's own
 * static workspace in place of a caller buffer. The workspace is a file-scope device array
 * of SKEW_STATIC_WORKSPACE_BYTES (64 MiB) that every GPU the library runs on holds until
 * the process ends; this call and the steps of its context make no device allocation (the
 * host context is an ordinary heap object, as with skew_state_init).
 *   ctx, d, n, state, state_bytes, stream   as for skew_state_init.
 * The array is shared by every call on one GPU and keeps the last call's contents: this
 * call zero-fills the part its table uses. There is one such context per GPU at a time: a
 * newer skew_state_init_static on the same GPU takes the array over, and skew_step on the
 * older context then returns SKEW_ESTALE without launching anything. Steps of contexts
 * that share the array must not overlap (they would race on it).
 * Errors: as skew_state_init, and SKEW_ETOOBIG when skew_state_bytes() reports more than
 * SKEW_STATIC_WORKSPACE_BYTES of workspace (nothing is touched then). */
int skew_state_init_static(skew_ctx **ctx, skew_tensor_desc *d, int n, void *state, size_t state_bytes,
                           void *stream);

/* One SkewAdam step (Alg. 1) over every tensor of ctx, enqueued on `stream`
 * (asynchronous; errors of the kernels themselves surface at the caller's next
 * synchronisation). Reads g, updates w and the state in place. One step per
 * context may be in flight at a time. Non-finite gradients propagate into the
 * state and weights (a NaN makes the clip factor NaN, so its whole tensor).
 * The state's and workspace's contents between steps belong to the library.
 * Errors: SKEW_EINVAL (ctx NULL, hp invalid), SKEW_ESTALE (see skew_state_init_static),
 * SKEW_EHIP (launch failed). */
int skew_step(skew_ctx *ctx, const skew_hparams *hp, void *stream);

/* Free the host context. Does not touch device memory. NULL is a no-op. */
void skew_destroy(skew_ctx *ctx);

/* Static description of a status code (never NULL). */
const char *skew_strerror(int status);

/* SKEW_ABI_VERSION of the loaded library. */
int skew_abi_version(void);

/* ---- Diagnostics: per-launch timing (not part of the step's definition) ----
 * skew_timing_enable(ctx, max_steps) creates HIP events for up to max_steps later
 * calls of skew_step on ctx, which then record one event before its first kernel and
 * one after each kernel on the step's stream (no synchronisation, no work skipped).
 * max_steps = 0 frees the events and stops recording. Errors: SKEW_EINVAL, SKEW_EHIP.
 * skew_timing_read(ctx, ms, max_launches, launches, steps) waits for the recorded
 * events, writes into ms[j] (host array of max_launches doubles) the summed duration
 * in milliseconds of the step's j-th kernel over the recorded steps, sets *launches
 * to the number of kernels per step and *steps to the number of steps recorded, and
 * restarts recording. skew_launch_name(ctx, j) names kernel j (static string). */
int skew_timing_enable(skew_ctx *ctx, int max_steps);
int skew_timing_read(skew_ctx *ctx, double *ms, int max_launches, int *launches, int *steps);
const char *skew_launch_name(skew_ctx *ctx, int j);

/* ---- Diagnostics: how the last step decided each tensor's clip factor ----
 * skew_clip_info(ctx, k, route, n, stream) waits for `stream`, then for every tensor i of
 * the table (n >= table size; host arrays of n entries) writes
 *   k[i]      the clip factor the last step applied (Sec. 3 "Update clipping"),
 *   route[i]  bits 0..3: how k was decided: 0 from the fast sums, 4 by the re-check that
 *             tests each element against the eps floor, 2 by the re-check that follows
 *             the reference float sequence;
 *             bits 4..7 (with 2 or 4): why a re-check ran: 1 forced by
 *             SKEW_FLAG_EXACT_CLIP, 2 non-finite values, 3 elements on both sides of the
 *             eps floor, 4 the floor regime changed from the one predicted, 5 a sum's
 *             error bound reaches a rounding boundary of k or the clipping threshold;
 *             bits 8..15: the sums the next step's row-band pass will form
 *             (0 both, 1 only the one above the eps floor, 2 only the floored one).
 * Empty tensors report k = 0, route = 0. Errors: SKEW_EINVAL, SKEW_EHIP. */
int skew_clip_info(skew_ctx *ctx, float *k, int32_t *route, int n, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* SKEWADAM_H */

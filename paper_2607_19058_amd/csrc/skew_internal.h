// skew_internal.h -- structures shared by the planner, the C ABI and the kernels.
#pragma once
#include <cstddef>
#include <cstdint>
#include <vector>

#include "../../include/skewadam.h"

namespace skew {

enum Kind : int32_t { kFactored = 0, kExact = 1 };

constexpr int kThreads = 256;           // threads per work-group (4 wave64)
constexpr int kWaves = kThreads / 64;
constexpr int kChunk = 512;             // columns one wave covers with one 16-byte load per lane
constexpr int kMaxCw = 4;               // chunks per tile row: 1, 2 or 4 (at most 2048 columns)
constexpr int kFold = 256;              // rows (or columns) folded by one work-group
constexpr int64_t kTileElems = 1 << 16; // target elements per tile: 128 KiB of bf16 gradient
constexpr size_t kAlign = 256;

// Row-band pass (pass 1 of factored matrices up to kZMaxCols columns): a work-group of
// kZThreads threads owns whole rows, so it knows each R_i as soon as the row is summed.
constexpr int kSub = 2;                  // update-sum passes: work-groups (row interleaves) per tile
constexpr int kZThreads = 512;           // 8 wave64 (up to 256 VGPRs each: nothing is held in flight)
constexpr int kZWaves = kZThreads / 64;
constexpr int kZMaxSeg = 4;              // 512-column chunks per wave and row
constexpr int64_t kZBandElems = 1 << 21; // elements per row band, at most: 4 MiB of bf16 gradient
constexpr int64_t kZMinBandElems = 1 << 19;   // ... and at least (unless a row is longer)
constexpr double kZTargetBands = 1024.0;      // bands per row-band launch class, about
constexpr int kZVariants = 16;           // kernel variants: lg(nseg) * 4 + (element loads ? 2 : 0) + momentum,
                                         // lg = 0, 1, 2, 3 for nseg = 1, 2, 4, 3 (3: no momentum)
constexpr int kZLdsBytes = 64 * 1024;    // one LDS staging buffer of the row-band pass (two per work-group)
constexpr int kZMaxBlockRows = 64;       // rows staged per block, at most
constexpr int kZMaxBandRows = 2048;      // rows per band, at most (their R are staged in LDS)

// Per-tensor scalars of one step, written by the clip stage and read by the update.
struct TensorScalars {
  float k;            // clip factor 1 / max(1, RMS(U_hat) / d), rounded as the oracle rounds it
  float q;            // max(mean R, eps) (factored tensors)
  int32_t ambiguous;  // bits 0..3: kClip* (how k was decided); bits 4..7: why a re-check ran (kWhy*)
  int32_t regime;     // row-band tensors, set by the clip stage for the next step: which sums the
                      // row-band pass forms (kRegime*); zero (both) after skew_state_init
  float split_spread; // relative spread of the last floor-split re-check's sum (0: none yet)
  int32_t fast_flags; // stacks: the slice's fast sum is open (bits 0..3: why), non-finite
                      // (bit 4), has repeated factors (bit 5)
  double s_fast, e_fast;  // stacks: the slice's fast sum and its error bound
};
// Tensors the clip stage sends to a re-check, listed on the device (so that a re-check
// launch covers only their tiles): l1 for the re-check with the exact floor split, l2 for
// the exact float sequence. Counts are zeroed by the update pass at the end of each step.
struct RecheckLists {
  int32_t n1, n2;
  int32_t pad[62];
  // followed by int32 l1[ntensors], int32 l2[ntensors]
};
constexpr int kRecheckGrid = 1024;   // work-groups of a re-check launch

// States of TensorScalars::ambiguous (bits 0..3)
enum ClipState : int32_t {
  kClipFast = 0,        // decided from the fast sums
  kClipPending1 = 1,    // listed for the re-check with the exact floor split
  kClipExact = 2,       // decided by the exact float sequence
  kClipPending2 = 3,    // listed for the exact float sequence
  kClipSplit = 4        // decided by the re-check with the exact floor split
};

// Why the clip stage sent a tensor to the exact pass.
enum Why : int32_t {
  kWhyForced = 1,       // SKEW_FLAG_EXACT_CLIP
  kWhyNonFinite = 2,    // a non-finite sum or statistic
  kWhyStraddle = 3,     // elements on both sides of the eps floor, and the bound reaches the threshold
  kWhyMissingSum = 4,   // the regime changed from the prediction, and the bound reaches the threshold
  kWhySpread = 5        // the fast sum's spread reaches a rounding boundary of k or the threshold
};
// Which update sums the row-band pass forms: both, only the one above the eps floor
// (the last step had every element clearly above it), or only the floored one.
enum Regime : int32_t { kRegimeBoth = 0, kRegimeAbove = 1, kRegimeFloor = 2 };

// Per row band of the row-band pass: sums and extremes the clip stage needs.
struct BandStats {
  double rsum;    // sum of the band's R_i (after the EMA)
  double ysum;    // sum over the band of RN(s x / sqrt(eps))^2: U_hat^2 of every element on the floor
  double umax;    // bound of max over the band of (s x)^2 / R_i
  float rmin;     // min R_i over rows with R_i > 0 (+inf if none)
  float rmax;     // max R_i
  int32_t bad;    // a row with R_i == 0 but a nonzero gradient (its elements escape the bounds)
  int32_t regime; // the sums this band formed (kRegime*)
  int32_t rdup;   // rows whose R_i > 0 equals the previous row's (repeated factors)
  int32_t pad;
};

// Per fold chunk of columns of a row-band tensor (of a wide factored tensor: per fold chunk of
// rows, then of columns, only cmin, cmax and cdup: extremes and equal neighbours of R or C).
struct ColStats {
  double s;       // sum over the chunk's columns of z_j / c'_j (U_hat^2 summed above the floor)
  float cmin;     // min c'_j over columns with C_j > 0 (+inf if none)
  float cmax;     // max c'_j
  int32_t bad;    // non-finite c'_j, or C_j == 0 with a nonzero column sum
  int32_t cdup;   // columns whose C_j > 0 equals the previous column's within the chunk
  double s2;      // sum over the chunk's columns of z_j / c'_j^2 (bounds the sum of squared terms)
};

// Device-resident description of one tensor, its state and its partial sums.
struct DevTensor {
  uint16_t *w;
  const uint16_t *g;
  float *M, *V, *R, *C;   // state (NULL where the tier keeps none)
  double *rowpart;        // [ntc][n]   partial row sums of g^2, one per column strip
  double *colpart;        // [ntr][m]   partial column sums of g^2, one per row band (row-band pass: [nzb][m])
  double *ainv;           // [n]        1/sqrt(R_i) after the step's EMA
  double *rsum;           // [nfr]      sums of R_i over each fold chunk of rows (row-band
                          //            tensors: [ceil(n / kFold)], in the gradient-norm mode)
  double *zpart;          // [nzb][m]   row-band pass: partial column sums of (s x)^2 / R_i
  BandStats *bst;         // [nzb]      row-band pass: per band
  ColStats *cst;          // [nfc]      row-band pass: per fold chunk of columns; wide factored
                          //            tensors: [nfr + nfc] extremes and equal neighbours of R, C
  double *ssum;           // [ntr*ntc]  per-tile sums of squares of the unclipped update
  double *qsum;           // [ntr*ntc]  per-tile sums of U_hat^4 over the approximated elements
  TensorScalars *sc;      // this step's clip factor and reconstruction clamp
  const uint16_t *zeros;  // 256 zero bytes (never written): the source of padding loads
  int64_t n, m, ld;       // rows, columns, row stride (elements)
  int64_t tr;             // rows per tile
  int32_t cw;             // 512-column chunks per tile (1, 2 or 4)
  int32_t ntc, ntr;       // column strips, row bands
  int32_t nfr, nfc;       // fold work-groups over rows, over columns
  int32_t kind;           // kFactored / kExact
  int32_t momentum;       // backbone tier
  int32_t vec;            // 16-byte aligned rows: vector loads and stores
  int32_t zpath;          // 1: pass 1 is the row-band pass (no separate update-sum pass)
  int32_t nseg;           // row-band pass: 512-column chunks per wave (1, 2, 3 or 4)
  int32_t zcw;            // row-band pass: 512-column chunks per row
  int32_t zrpi;           // row-band pass: row groups per work-group (rows side by side); a group
                          // is wpr = ceil(zcw / nseg) waves, wave w of it takes chunks w, w + wpr
  int32_t nzb;            // row-band pass: row bands
  int32_t zrb;            // row-band pass: rows per group and block
  int32_t decay;          // the decoupled weight decay applies (every tier but the router)
  int64_t zrows;
  int64_t idx0;           // element index of this (sub-)tensor's first element in the caller's
                          // tensor: a stacked tensor's slices are sub-tensors (dither index)
  int32_t grp0, ngrp;     // the sub-tensors that share one clip factor: [grp0, grp0 + ngrp)
  int32_t fp32;           // w and g are float32 (float32 masters: no dither, no cast)
  int32_t pad3;          // row-band pass: rows per band
  uint64_t tensor_id;
};

struct Item {
  int32_t tensor;
  int32_t tile;
};

// Per-step scalars (Alg. 1), computed on the host in double and rounded once.
struct StepConsts {
  float b1, a1, b2, a2, eps, lr, d, s_m, s_0;
  int32_t flags;   // SKEW_FLAG_*
  int64_t step;
  uint64_t seed;
  float wd;                 // lr * lambda of the decoupled weight decay, rounded once (0: off)
  float max_grad_norm;      // > 0: gradients scaled by the global norm's factor
  int32_t gclip;            // max_grad_norm > 0
  int32_t pad;
  float *gscale;            // device: the factor c (written by the norm stage)
  double *gsq;              // device [ntensors]: each tensor's sum of g^2 (norm stage)
};

// Host-side plan of a descriptor table.
struct TensorPlan {
  int32_t desc = 0;            // descriptor this sub-tensor comes from
  int32_t grp0 = 0, ngrp = 1;  // the sub-tensors sharing its clip factor (a stacked tensor's slices)
  int64_t idx0 = 0;            // element index of its first element in the descriptor's tensor
  int64_t n = 0, m = 0, ld = 0, N = 0;
  int32_t tier = 0, kind = 0, momentum = 0, fp32 = 0;
  int64_t tr = 0;
  int32_t cw = 0, ntc = 0, ntr = 0, nfr = 0, nfc = 0;
  bool empty = true;
  // state slice offsets in bytes (SIZE_MAX: none)
  size_t off_m = SIZE_MAX, off_v = SIZE_MAX, off_r = SIZE_MAX, off_c = SIZE_MAX;
  // workspace offsets in bytes
  size_t off_rowpart = SIZE_MAX, off_colpart = SIZE_MAX, off_ainv = SIZE_MAX, off_rsum = SIZE_MAX,
         off_ssum = SIZE_MAX, off_qsum = SIZE_MAX, off_sc = SIZE_MAX, off_zpart = SIZE_MAX, off_bst = SIZE_MAX,
         off_cst = SIZE_MAX;
  // row-band pass geometry
  int32_t zpath = 0, nseg = 0, zcw = 0, zrpi = 0, nzb = 0, zrb = 0;
  int64_t zrows = 0;
};

struct Plan {
  std::vector<TensorPlan> t;                  // sub-tensors (the device table's entries)
  std::vector<int32_t> desc_sub0, desc_nsub;  // per descriptor: its first sub-tensor and their count
  size_t off_lists = 0;                       // workspace offset of the RecheckLists
  size_t off_zero = 0;                        // workspace offset of 256 zero bytes
  size_t off_gscale = 0;                      // workspace offset of the gradient scale (float)
  size_t off_gsq = 0;                         // workspace offset of the per-tensor sums of g^2
  std::vector<Item> p1, fold, p2, p3, clip;   // clip: one item per non-empty tensor
  std::vector<Item> clip_slices;              // every slice of the stacked tensors
  // fold items of the gradient-norm mode's first fold: rows and columns of every factored
  // tensor (row-band tensors: rows [0, ceil(n / kFold)), then columns)
  std::vector<Item> fold_rows;
  std::vector<Item> z;                        // row-band pass items (split by kernel variant at init)
  size_t state_bytes = 0;
  size_t ws_bytes = 0;
  size_t off_table = 0, off_items = 0;   // workspace offsets of the device table and item lists
};

inline size_t align_up(size_t x, size_t a = kAlign) { return (x + a - 1) / a * a; }

// Validates the table and computes sizes, offsets and the work-item lists.
int plan_build(const skew_tensor_desc *d, int n, Plan *out);

// The library's static workspace (skew_state_init_static): the device address of the
// file-scope array on the current device, looked up once per device (skew_kernels.hip).
// Returns a hipError_t value.
int static_workspace(void **ptr);
constexpr size_t static_workspace_bytes() { return (size_t)SKEW_STATIC_WORKSPACE_BYTES; }

// Kernel launchers (skew_kernels.hip). Return a hipError_t value.
int launch_p1(const DevTensor *T, const Item *items, int64_t count, void *stream);
// row-band pass, kernel variant lg(nseg) * 4 + (element loads ? 2 : 0) + (momentum ? 1 : 0)
// mode 0: the whole pass; 1: sums of g^2 only (row sums to ainv); 2: z, floored sum and
// band statistics from the R already folded (the gradient-norm mode's two passes)
int launch_p1z(const DevTensor *T, const Item *items, int64_t count, const StepConsts &k, int variant, int mode,
               void *stream);

// fold phase 0: the step without gradient-norm scaling; 1: its first fold (R and C of every
// factored tensor from the sums of g^2, scaled by c^2); 2: its second fold (row-band tensors:
// c' and sum_j z_j / c'_j)
int launch_fold(const DevTensor *T, const Item *items, int64_t count, const StepConsts &k, int phase, void *stream);
// gradient-norm mode: sums of g^2 of exact tensors over the update-sum items, then the scale
int launch_gsq(const DevTensor *T, const Item *items, int64_t count, void *stream);
int launch_gnorm(const DevTensor *T, int ntensors, const StepConsts &k, void *stream);
int launch_p2(const DevTensor *T, const Item *items, int64_t count, const StepConsts &k, void *stream);
int launch_p3(const DevTensor *T, const Item *items, int64_t count, const StepConsts &k, RecheckLists *L,
              void *stream);
// the clip stage's fast sum of every slice of the stacked tensors (one wave per slice)
int launch_clip_slices(const DevTensor *T, const Item *items, int64_t count, const StepConsts &k, void *stream);
int launch_clip(const DevTensor *T, const Item *items, int64_t count, const StepConsts &k, RecheckLists *L,
                int ntensors, void *stream);
// re-check of the listed tensors: level 1 (exact floor split) or 2 (exact float sequence),
// then their clip factors from the new sums
int launch_recheck(const DevTensor *T, RecheckLists *L, int ntensors, const StepConsts &k, int level, void *stream);
int launch_clip_recheck(const DevTensor *T, RecheckLists *L, int ntensors, const StepConsts &k, int level,
                        void *stream);

}  // namespace skew

// skew_plan.cpp -- host-only planning of a descriptor table: validation, the tier
// state each tensor keeps (Fig. 1; Sec. 3 "The tiers"), the state size of Eq. 2
// (plus the exact v of vectors, Table 6), the tile grids and the work-item lists.
// No HIP calls: this runs without a GPU.
#include <algorithm>
#include <climits>
#include <cmath>

#include "skew_internal.h"

namespace skew {

static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

int plan_build(const skew_tensor_desc *d, int n, Plan *out) {
  if (n < 0 || (n > 0 && d == nullptr) || out == nullptr) return SKEW_EINVAL;
  Plan p;
  p.t.resize(n);
  size_t st = 0;        // state bytes
  size_t ws_part = 0;   // partial-sum bytes (offsets relative to the partial region)
  int64_t items_total = 0;
  for (int i = 0; i < n; i++) {
    const skew_tensor_desc &x = d[i];
    TensorPlan &tp = p.t[i];
    if (x.tier < SKEW_TIER_BACKBONE || x.tier > SKEW_TIER_ROUTER) return SKEW_EINVAL;
    if (x.ndim != 1 && x.ndim != 2) return SKEW_EINVAL;
    if (x.rows < 0 || x.cols < 0) return SKEW_EINVAL;
    if (x.rows > 0 && x.cols > INT64_MAX / x.rows) return SKEW_EINVAL;
    const int64_t N = x.rows * x.cols;
    tp.tier = x.tier;
    tp.N = N;
    if (x.ndim == 1) {
      if (N > 0 && x.rows != 1 && x.cols != 1) return SKEW_EINVAL;
      tp.n = N > 0 ? 1 : 0;
      tp.m = N;
      tp.ld = N;
    } else {
      if (x.ld < x.cols || x.ld < 1) return SKEW_EINVAL;
      if (x.rows > 0 && x.ld > INT64_MAX / x.rows) return SKEW_EINVAL;
      tp.n = x.rows;
      tp.m = x.cols;
      tp.ld = x.ld;
    }
    tp.empty = (N == 0);
    tp.kind = (x.tier == SKEW_TIER_ROUTER || x.ndim == 1) ? kExact : kFactored;
    tp.momentum = (x.tier == SKEW_TIER_BACKBONE);
    if (tp.empty) continue;

    // state slices
    if (tp.momentum) { tp.off_m = st; st = align_up(st + (size_t)N * 4); }
    if (tp.kind == kExact) { tp.off_v = st; st = align_up(st + (size_t)N * 4); }
    if (tp.kind == kFactored) {
      tp.off_r = st; st = align_up(st + (size_t)tp.n * 4);
      tp.off_c = st; st = align_up(st + (size_t)tp.m * 4);
    }

    // tile grid: tr rows x (512 * cw) columns, about kTileElems elements; cw in {1, 2, 4}
    // so that the four waves of a work-group map onto (chunk, row) pairs statically
    tp.cw = tp.m > 2 * kChunk ? 4 : (tp.m > kChunk ? 2 : 1);
    const int64_t tc = (int64_t)kChunk * tp.cw;
    tp.tr = std::max<int64_t>(1, kTileElems / tc);
    const int64_t ntc = ceil_div(tp.m, tc), ntr = ceil_div(tp.n, tp.tr);
    if (ntc * ntr > INT32_MAX / 2 / kSub) return SKEW_EINVAL;   // tile * kSub + part fits an int32
    tp.ntc = (int32_t)ntc;
    tp.ntr = (int32_t)ntr;
    const int64_t tiles = ntc * ntr;

    tp.off_ssum = ws_part; ws_part = align_up(ws_part + (size_t)tiles * kSub * 8);
    tp.off_qsum = ws_part; ws_part = align_up(ws_part + (size_t)tiles * kSub * 8);
    tp.off_sc = ws_part; ws_part = align_up(ws_part + sizeof(TensorScalars));
    p.clip.push_back({i, 0});
    // Row-band pass for factored matrices whose staged rows fit: zcw 512-column chunks per
    // row, nseg (1, 2 or 4) of them per wave, so wpr = ceil(zcw / nseg) <= 8 waves share a
    // row and zrpi = 8 / wpr rows are side by side. A block of zrpi * zrb rows (bf16
    // gradient, plus fp32 momentum on the backbone) fills at most one LDS buffer.
    const int64_t zcw = ceil_div(tp.m, kChunk);
    const int64_t nseg = zcw <= 1 ? 1 : (zcw <= 2 * kZWaves ? 2 : 4);
    const int64_t wpr = ceil_div(zcw, nseg);
    const int64_t row_kb = zcw * (tp.momentum ? 3 : 1);   // staged KiB per row
    const int64_t rpi = wpr <= kZWaves ? kZWaves / wpr : 0;
    int64_t zrb = rpi > 0 ? std::min<int64_t>(nseg <= 2 ? 4 : 1, kZLdsBytes / (rpi * row_kb * 1024)) : 0;
    while (zrb & (zrb - 1)) zrb &= zrb - 1;   // a power of two: 1, 2 or 4
    tp.zpath = (tp.kind == kFactored && rpi > 0 && zrb >= 1) ? 1 : 0;
    if (tp.zpath) {
      tp.zcw = (int32_t)zcw;
      tp.nseg = (int32_t)nseg;
      tp.zrpi = (int32_t)rpi;
      tp.zrb = (int32_t)zrb;
      const int64_t rows_block = rpi * zrb;
      tp.zrows = ceil_div(std::max<int64_t>(1, ceil_div(kZBandElems, tp.m)), rows_block) * rows_block;
      tp.zrows = std::min<int64_t>(tp.zrows, kZMaxBandRows / rows_block * rows_block);
      const int64_t nzb = ceil_div(tp.n, tp.zrows), nfc = ceil_div(tp.m, kFold);
      if (nzb > INT32_MAX / 2 || nfc > INT32_MAX / 2) return SKEW_EINVAL;
      tp.nzb = (int32_t)nzb;
      tp.nfr = 0;
      tp.nfc = (int32_t)nfc;
      tp.off_colpart = ws_part; ws_part = align_up(ws_part + (size_t)nzb * tp.m * 8);
      tp.off_zpart = ws_part; ws_part = align_up(ws_part + (size_t)nzb * tp.m * 8);
      tp.off_ainv = ws_part; ws_part = align_up(ws_part + (size_t)tp.n * 8);
      tp.off_bst = ws_part; ws_part = align_up(ws_part + (size_t)nzb * sizeof(BandStats));
      tp.off_cst = ws_part; ws_part = align_up(ws_part + (size_t)nfc * sizeof(ColStats));
      const int64_t nzr = ceil_div(tp.n, kFold);   // row chunks of the gradient-norm mode's fold
      if (nzr > INT32_MAX / 4) return SKEW_EINVAL;
      tp.off_rsum = ws_part; ws_part = align_up(ws_part + (size_t)nzr * 8);
      for (int32_t k = 0; k < tp.nzb; k++) p.z.push_back({i, k});
      for (int32_t k = 0; k < tp.nfc; k++) p.fold.push_back({i, k});
      for (int32_t k = 0; k < (int32_t)nzr + tp.nfc; k++) p.fold_rows.push_back({i, k});
      items_total += nzb + nfc + nzr + nfc;
    } else if (tp.kind == kFactored) {
      const int64_t nfr = ceil_div(tp.n, kFold), nfc = ceil_div(tp.m, kFold);
      if (nfr + nfc > INT32_MAX / 2) return SKEW_EINVAL;
      tp.nfr = (int32_t)nfr;
      tp.nfc = (int32_t)nfc;
      tp.off_rowpart = ws_part; ws_part = align_up(ws_part + (size_t)ntc * tp.n * 8);
      tp.off_colpart = ws_part; ws_part = align_up(ws_part + (size_t)ntr * tp.m * 8);
      tp.off_ainv = ws_part; ws_part = align_up(ws_part + (size_t)tp.n * 8);
      tp.off_rsum = ws_part; ws_part = align_up(ws_part + (size_t)nfr * 8);
      for (int32_t k = 0; k < tp.ntr * tp.ntc; k++) p.p1.push_back({i, k});
      for (int32_t k = 0; k < tp.nfr + tp.nfc; k++) p.fold.push_back({i, k});
      for (int32_t k = 0; k < tp.nfr + tp.nfc; k++) p.fold_rows.push_back({i, k});
      items_total += tiles + 2 * (nfr + nfc);
    }
    if (!tp.zpath) {
      for (int32_t k = 0; k < tp.ntr * tp.ntc * kSub; k++) p.p2.push_back({i, k});   // tile * kSub + part
      items_total += tiles * kSub;
    }
    for (int32_t k = 0; k < tp.ntr * tp.ntc; k++) p.p3.push_back({i, k});
    items_total += tiles;
    if (items_total > INT32_MAX / 2) return SKEW_EINVAL;
  }
  // pipeline groups: consecutive tensors, about equal algorithmic bytes (gradient, weight
  // read and write, and the state each tier reads and writes)
  {
    std::vector<double> bytes(n, 0.0);
    double total = 0.0;
    int nonempty = 0;
    for (int i = 0; i < n; i++) {
      const TensorPlan &tp = p.t[i];
      if (tp.empty) continue;
      bytes[i] = (double)tp.N * (6.0 + (tp.momentum ? 8.0 : 0.0) + (tp.kind == kExact ? 8.0 : 0.0));
      total += bytes[i];
      nonempty++;
    }
    p.ngroups = std::max(1, std::min(kMaxGroups, nonempty));
    p.tgroup.assign(n, 0);
    double acc = 0.0;
    for (int i = 0; i < n; i++) {
      const int g = total > 0.0 ? (int)(acc / total * p.ngroups) : 0;
      p.tgroup[i] = std::min(g, p.ngroups - 1);
      acc += bytes[i];
    }
  }
  p.state_bytes = st;
  // workspace: [device tensor table][items p1|z (by variant)|fold|p2|p3|clip][re-check lists][partials]
  size_t ws = 0;
  p.off_table = ws; ws = align_up(ws + sizeof(DevTensor) * (size_t)std::max(n, 1));
  p.off_items = ws;
  ws = align_up(ws + sizeof(Item) * (p.p1.size() + p.z.size() + p.fold.size() + p.p2.size() + p.p3.size() +
                                     p.clip.size() + p.fold_rows.size() + 1));
  p.off_lists = ws;
  ws = align_up(ws + sizeof(RecheckLists) + sizeof(int32_t) * 2 * (size_t)std::max(n, 1));
  p.off_zero = ws;   // zero-filled with the workspace at set-up and never written
  ws = align_up(ws + 256);
  p.off_gscale = ws;
  ws = align_up(ws + sizeof(float));
  p.off_gsq = ws;
  ws = align_up(ws + sizeof(double) * (size_t)std::max(n, 1));
  auto shift = [ws](size_t &off) {
    if (off != SIZE_MAX) off += ws;
  };
  for (auto &tp : p.t) {
    if (tp.empty) continue;
    for (size_t *o : {&tp.off_ssum, &tp.off_qsum, &tp.off_sc, &tp.off_rowpart, &tp.off_colpart, &tp.off_ainv,
                      &tp.off_rsum, &tp.off_zpart, &tp.off_bst, &tp.off_cst})
      shift(*o);
  }
  p.ws_bytes = ws + ws_part;
  *out = std::move(p);
  return SKEW_OK;
}

}  // namespace skew

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

// Row-band pass for factored matrices whose staged rows fit: zcw 512-column chunks per
// row, nseg (1, 2, 3 or 4) of them per wave, so wpr = ceil(zcw / nseg) <= 8 waves share a
// row and rpi = 8 / wpr rows are side by side. Three chunks per wave (rows of 8193 to
// 12288 columns, e.g. 11008) keep the lean loads and the block in registers; they are
// used without momentum only (with it, the general loop's four chunks per wave). A block of rpi * zrb rows (bf16 gradient,
// plus fp32 momentum on the backbone) fills at most one LDS buffer. zrb = 0: no row band.
struct RowBandShape {
  int64_t zcw, nseg, rpi, zrb;
};
static RowBandShape rowband_shape(int64_t m, bool momentum) {
  RowBandShape r;
  r.zcw = ceil_div(m, kChunk);
  r.nseg = r.zcw <= 1 ? 1 : (r.zcw <= 2 * kZWaves ? 2 : (!momentum && r.zcw <= 3 * kZWaves ? 3 : 4));
  const int64_t wpr = ceil_div(r.zcw, r.nseg);
  const int64_t row_kb = r.zcw * (momentum ? 3 : 1);   // staged KiB per row
  r.rpi = wpr <= kZWaves ? kZWaves / wpr : 0;
  r.zrb = r.rpi > 0 ? std::min<int64_t>(r.nseg <= 2 ? 4 : (r.nseg == 3 ? 2 : 1), kZLdsBytes / (r.rpi * row_kb * 1024))
                    : 0;
  while (r.zrb & (r.zrb - 1)) r.zrb &= r.zrb - 1;   // a power of two: 1, 2 or 4
  return r;
}

int plan_build(const skew_tensor_desc *d, int n, Plan *out) {
  if (n < 0 || (n > 0 && d == nullptr) || out == nullptr) return SKEW_EINVAL;
  Plan p;
  // descriptors -> sub-tensors: a stacked (ndim 3) descriptor of E matrices becomes E
  // sub-tensors (one per slice, factored on its own, Sec. 3 footnote) that share one clip
  // factor; every other descriptor is one sub-tensor
  p.desc_sub0.assign((size_t)n, 0);
  p.desc_nsub.assign((size_t)n, 1);
  int64_t nsub = 0;
  for (int i = 0; i < n; i++) {
    const skew_tensor_desc &x = d[i];
    if (x.tier < SKEW_TIER_BACKBONE || x.tier > SKEW_TIER_ROUTER) return SKEW_EINVAL;
    if (x.ndim < 1 || x.ndim > 3) return SKEW_EINVAL;
    if ((x.state_flags & ~(uint32_t)(SKEW_STATE_MOMENTUM | SKEW_STATE_FACTORED | SKEW_STATE_FP32)) != 0)
      return SKEW_EINVAL;
    if (x.ndim == 3 ? x.batch < 0 : (x.batch != 0 && x.batch != 1)) return SKEW_EINVAL;
    const int64_t E = (x.ndim == 3 && x.batch > 1) ? x.batch : 1;
    if (E > INT32_MAX / 4) return SKEW_EINVAL;
    p.desc_sub0[(size_t)i] = (int32_t)nsub;
    p.desc_nsub[(size_t)i] = (int32_t)E;
    nsub += E;
    if (nsub > INT32_MAX / 4) return SKEW_EINVAL;
  }
  p.t.resize((size_t)nsub);
  // Row-band size per launch class (with and without momentum, the row-band pass's two
  // kinds of launch): about kZTargetBands bands over the class, so that a class of few
  // tensors still fills the chip, between kZMinBandElems and kZBandElems elements
  int64_t band_elems[2] = {kZBandElems, kZBandElems};
  {
    double cls[2] = {0.0, 0.0};
    for (int i = 0; i < n; i++) {
      const skew_tensor_desc &x = d[i];
      if (x.ndim == 1 || x.rows <= 0 || x.cols <= 0) continue;
      if (x.tier == SKEW_TIER_ROUTER && !(x.state_flags & SKEW_STATE_FACTORED)) continue;
      const bool mom = x.tier == SKEW_TIER_BACKBONE || (x.state_flags & SKEW_STATE_MOMENTUM) != 0;
      if (rowband_shape(x.cols, mom).zrb < 1) continue;
      const double E = (x.ndim == 3) ? (double)x.batch : 1.0;
      cls[mom ? 1 : 0] += E * (double)x.rows * (double)x.cols;
    }
    for (int c = 0; c < 2; c++) {
      int64_t b = kZBandElems;
      while (b > kZMinBandElems && (double)b * kZTargetBands > cls[c]) b >>= 1;
      band_elems[c] = b;
    }
  }
  size_t st = 0;        // state bytes
  size_t ws_part = 0;   // partial-sum bytes (offsets relative to the partial region)
  int64_t items_total = 0;
  for (int di = 0; di < n; di++) {
  const skew_tensor_desc &x = d[di];
  const int32_t sub0 = p.desc_sub0[(size_t)di], E = p.desc_nsub[(size_t)di];
  for (int32_t e = 0; e < E; e++) {
    const int i = sub0 + e;   // the sub-tensor
    TensorPlan &tp = p.t[(size_t)i];
    tp.desc = di;
    tp.grp0 = sub0;
    tp.ngrp = E;
    if (x.rows < 0 || x.cols < 0) return SKEW_EINVAL;
    if (x.rows > 0 && x.cols > INT64_MAX / x.rows) return SKEW_EINVAL;
    const int64_t N = (x.ndim == 3 && x.batch == 0) ? 0 : x.rows * x.cols;
    if (N > 0 && E > INT64_MAX / N) return SKEW_EINVAL;
    tp.tier = x.tier;
    tp.N = N;
    tp.idx0 = (int64_t)e * N;   // the slice's first element in the stacked tensor
    if (x.ndim == 1) {
      if (N > 0 && x.rows != 1 && x.cols != 1) return SKEW_EINVAL;
      tp.n = N > 0 ? 1 : 0;
      tp.m = N;
      tp.ld = N;
    } else {
      if (x.ld < x.cols || x.ld < 1) return SKEW_EINVAL;
      if (x.rows > 0 && x.ld > INT64_MAX / x.rows / E) return SKEW_EINVAL;
      tp.n = x.rows;
      tp.m = x.cols;
      tp.ld = x.ld;
    }
    tp.empty = (N == 0);
    // tiers (Fig. 1) and their variants (Table 3): momentum in the backbone or on request;
    // the exact second moment for vectors and router matrices unless factoring is requested
    const bool factor_router = (x.state_flags & SKEW_STATE_FACTORED) != 0;
    tp.kind = ((x.tier == SKEW_TIER_ROUTER && !factor_router) || x.ndim == 1) ? kExact : kFactored;
    tp.momentum = (x.tier == SKEW_TIER_BACKBONE || (x.state_flags & SKEW_STATE_MOMENTUM) != 0) ? 1 : 0;
    tp.fp32 = (x.state_flags & SKEW_STATE_FP32) != 0 ? 1 : 0;
    if (tp.fp32 && tp.kind != kExact) return SKEW_EINVAL;   // float32 masters: exact-moment tensors
    if (tp.empty) continue;

    // state slices: one contiguous array per descriptor (slice e at e times the slice)
    if (e == 0) {
      if (tp.momentum) { tp.off_m = st; st = align_up(st + (size_t)E * N * 4); }
      if (tp.kind == kExact) { tp.off_v = st; st = align_up(st + (size_t)E * N * 4); }
      if (tp.kind == kFactored) {
        tp.off_r = st; st = align_up(st + (size_t)E * tp.n * 4);
        tp.off_c = st; st = align_up(st + (size_t)E * tp.m * 4);
      }
    } else {
      const TensorPlan &t0 = p.t[(size_t)sub0];
      if (tp.momentum) tp.off_m = t0.off_m + (size_t)e * N * 4;
      if (tp.kind == kExact) tp.off_v = t0.off_v + (size_t)e * N * 4;
      if (tp.kind == kFactored) {
        tp.off_r = t0.off_r + (size_t)e * tp.n * 4;
        tp.off_c = t0.off_c + (size_t)e * tp.m * 4;
      }
    }

    // tile grid: tr rows x (512 * cw) columns, about kTileElems elements; cw in {1, 2, 4}
    // so that the four waves of a work-group map onto (chunk, row) pairs statically. The widest
    // strip that fits; a narrower one when the last strip would leave more than 1/16 of the
    // row's width in idle lanes (1536 columns: 512 of 2048; 11008: 1280 of 12288)
    tp.cw = tp.m > 2 * kChunk ? 4 : (tp.m > kChunk ? 2 : 1);
    {
      auto waste = [&](int64_t cw) { return ceil_div(tp.m, (int64_t)kChunk * cw) * kChunk * cw - tp.m; };
      if (16 * waste(tp.cw) > tp.m)
        for (int32_t cw = tp.cw / 2; cw >= 1; cw /= 2)
          if (waste(cw) < waste(tp.cw)) tp.cw = cw;
    }
    const int64_t tc = (int64_t)kChunk * tp.cw;
    // (exact-moment tensors take a quarter of that: their element-by-element path is the
    // slowest per element, and their few tiles would otherwise finish last)
    tp.tr = std::max<int64_t>(1, kTileElems / tc / (tp.kind == kExact ? 4 : 1));
    const int64_t ntc = ceil_div(tp.m, tc), ntr = ceil_div(tp.n, tp.tr);
    if (ntc * ntr > INT32_MAX / 2 / kSub) return SKEW_EINVAL;   // tile * kSub + part fits an int32
    tp.ntc = (int32_t)ntc;
    tp.ntr = (int32_t)ntr;
    const int64_t tiles = ntc * ntr;

    tp.off_ssum = ws_part; ws_part = align_up(ws_part + (size_t)tiles * kSub * 8);
    tp.off_qsum = ws_part; ws_part = align_up(ws_part + (size_t)tiles * kSub * 8);
    tp.off_sc = ws_part; ws_part = align_up(ws_part + sizeof(TensorScalars));
    if (e == 0) p.clip.push_back({i, 0});   // one clip item per group (its first slice)
    if (E > 1) p.clip_slices.push_back({i, 0});
    // the row-band pass (see rowband_shape)
    const RowBandShape rbs = rowband_shape(tp.m, tp.momentum != 0);
    const int64_t zcw = rbs.zcw, nseg = rbs.nseg, rpi = rbs.rpi, zrb = rbs.zrb;
    tp.zpath = (tp.kind == kFactored && rpi > 0 && zrb >= 1) ? 1 : 0;
    if (tp.zpath) {
      tp.zcw = (int32_t)zcw;
      tp.nseg = (int32_t)nseg;
      tp.zrpi = (int32_t)rpi;
      tp.zrb = (int32_t)zrb;
      const int64_t rows_block = rpi * zrb;
      tp.zrows = ceil_div(std::max<int64_t>(1, ceil_div(band_elems[tp.momentum ? 1 : 0], tp.m)), rows_block) *
                 rows_block;
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
      tp.off_cst = ws_part; ws_part = align_up(ws_part + (size_t)(nfr + nfc) * sizeof(ColStats));
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
  }
  const int nt = (int)p.t.size();   // sub-tensors: the device table's entries
  // update-pass and update-sum items: tiles that take longest go first, so that they do not
  // finish last: the exact second moment's element-by-element path, and matrices narrower
  // than a 512-column strip (idle lanes)
  {
    auto slow = [&](const Item &it) {
      const TensorPlan &tp = p.t[(size_t)it.tensor];
      return tp.kind == kExact || tp.m < 512;
    };
    auto order = [&](std::vector<Item> &v) {
      std::stable_sort(v.begin(), v.end(), [&](const Item &a, const Item &b) { return slow(a) && !slow(b); });
    };
    order(p.p3);
    order(p.p2);
  }
  p.state_bytes = st;
  // workspace: [device tensor table][items p1|z (by variant)|fold|p2|p3|clip][re-check lists][partials]
  size_t ws = 0;
  p.off_table = ws; ws = align_up(ws + sizeof(DevTensor) * (size_t)std::max(nt, 1));
  // the item lists as the device keeps them: the fold's items appear twice (the whole list,
  // and split into row-band and other tensors)
  p.off_items = ws;
  ws = align_up(ws + sizeof(Item) * (p.p1.size() + p.z.size() + 2 * p.fold.size() + p.p2.size() + p.p3.size() +
                                     p.clip.size() + p.clip_slices.size() + p.fold_rows.size() + 1));
  p.off_lists = ws;
  ws = align_up(ws + sizeof(RecheckLists) + sizeof(int32_t) * 2 * (size_t)std::max(nt, 1));
  p.off_zero = ws;   // zero-filled with the workspace at set-up and never written
  ws = align_up(ws + 256);
  p.off_gscale = ws;
  ws = align_up(ws + sizeof(float));
  p.off_gsq = ws;
  ws = align_up(ws + sizeof(double) * (size_t)std::max(nt, 1));
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

// skew_api.cpp -- the C ABI declared in include/skewadam.h.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <new>
#include <vector>

#include "skew_internal.h"

using namespace skew;

namespace {
constexpr int kLaunches = 10;
const char *const kLaunchNames[kLaunches] = {"p1z_rowband_stats", "p1z_rowband_stats_momentum", "p1_rowcol_sumsq",
                                             "fold_rc_ema", "p2_update_sumsq", "clip_factor",
                                             "recheck_update_sumsq", "clip_factor_recheck", "p3_apply_dither",
                                             "grad_norm"};
}  // namespace

// an item list with the bounds of each pipeline group in it
struct GroupedList {
  Item *d = nullptr;
  std::vector<int64_t> bound;   // group g: items [bound[g], bound[g + 1])
  int64_t count(int g) const { return bound[g + 1] - bound[g]; }
  const Item *at(int g) const { return d + bound[g]; }
};

struct skew_ctx {
  Plan plan;
  char *ws = nullptr;   // workspace base (device)
  DevTensor *d_table = nullptr;
  RecheckLists *lists = nullptr;
  GroupedList p1, fold, p2, p3, clip, fold_rows;
  GroupedList fold_z, fold_w;   // the fold's items of row-band tensors and of the others
  float *gscale = nullptr;   // device: the gradient-norm mode's scale
  double *gsq = nullptr;     // device: per-tensor sums of g^2
  GroupedList z[kZVariants];   // row-band pass items, one list per kernel variant
  hipStream_t side = nullptr;  // the update pass of the pipeline runs here
  // [0]: step start, [1]: update pass done, [2 + g]: group g ready, [2 + ngroups]: the side
  // stream's statistics of wide and exact tensors done
  std::vector<hipEvent_t> sync;
  // diagnostics: per recorded step, (launch kind, start event, end event) of every launch
  struct Timed {
    int kind;
    hipEvent_t a, b;
  };
  std::vector<hipEvent_t> ev_pool;
  std::vector<std::vector<Timed>> timed;
  int ev_steps = 0, ev_used = 0;
  size_t ev_next = 0;
  ~skew_ctx() {
    for (hipEvent_t e : ev_pool) (void)hipEventDestroy(e);
    for (hipEvent_t e : sync) (void)hipEventDestroy(e);
    if (side) (void)hipStreamDestroy(side);
  }
};

namespace {

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

// Step scalars (Alg. 1): bias corrections s_m = sqrt(1-b2^t)/(1-b1^t) (backbone, with
// momentum) and s_0 = sqrt(1-b2^t) (momentum-free tiers), in double, rounded once.
StepConsts make_consts(const skew_hparams &hp) {
  StepConsts k;
  std::memset(&k, 0, sizeof k);
  const double b1 = hp.beta1, b2 = hp.beta2, t = (double)hp.step;
  k.b1 = hp.beta1;
  k.a1 = (float)(1.0 - b1);
  k.b2 = hp.beta2;
  k.a2 = (float)(1.0 - b2);
  k.eps = hp.eps;
  k.lr = hp.lr;
  k.d = hp.clip_threshold;
  const double bc2 = 1.0 - std::pow(b2, t), bc1 = 1.0 - std::pow(b1, t);
  k.s_m = (float)(std::sqrt(bc2) / bc1);
  k.s_0 = (float)std::sqrt(bc2);
  k.step = hp.step;
  k.seed = hp.seed;
  k.flags = hp.flags;
  k.wd = (float)((double)hp.lr * (double)hp.weight_decay);
  k.max_grad_norm = hp.max_grad_norm;
  k.gclip = hp.max_grad_norm > 0.0f ? 1 : 0;
  return k;
}

bool hparams_ok(const skew_hparams *hp) {
  if (hp == nullptr) return false;
  if ((hp->flags & ~(SKEW_FLAG_EXACT_CLIP | SKEW_FLAG_EXACT_ULP)) != 0 || hp->step < 1) return false;
  if (!std::isfinite(hp->lr)) return false;
  if (!(hp->beta1 >= 0.0f && hp->beta1 < 1.0f)) return false;
  if (!(hp->beta2 >= 0.0f && hp->beta2 < 1.0f)) return false;
  if (!(hp->eps > 0.0f) || !std::isfinite(hp->eps)) return false;
  if (!(hp->clip_threshold > 0.0f)) return false;  // +inf allowed: no clipping
  if (!(hp->weight_decay >= 0.0f) || !std::isfinite(hp->weight_decay)) return false;
  if (!(hp->max_grad_norm >= 0.0f) || !std::isfinite(hp->max_grad_norm)) return false;
  return true;
}

}  // namespace

extern "C" {

int skew_abi_version(void) { return SKEW_ABI_VERSION; }

const char *skew_strerror(int status) {
  switch (status) {
    case SKEW_OK: return "ok";
    case SKEW_EINVAL: return "invalid argument (tier, ndim, shape, ld, null pointer or hyper-parameter)";
    case SKEW_ENOSPACE: return "a caller buffer is smaller than skew_state_bytes() requires";
    case SKEW_EHIP: return "HIP runtime error (launch, copy or memset failed)";
    case SKEW_ENOMEM: return "host allocation failed";
    default: return "unknown status";
  }
}

int skew_state_bytes(const skew_tensor_desc *d, int n, size_t *state_bytes, size_t *workspace_bytes) {
  Plan p;
  const int rc = plan_build(d, n, &p);
  if (rc != SKEW_OK) return rc;
  if (state_bytes) *state_bytes = p.state_bytes;
  if (workspace_bytes) *workspace_bytes = p.ws_bytes;
  return SKEW_OK;
}

int skew_state_init(skew_ctx **ctx, skew_tensor_desc *d, int n, void *state, size_t state_bytes, void *workspace,
                    size_t workspace_bytes, void *stream) {
  if (ctx == nullptr) return SKEW_EINVAL;
  *ctx = nullptr;
  Plan p;
  int rc = plan_build(d, n, &p);
  if (rc != SKEW_OK) return rc;
  if (state_bytes < p.state_bytes || workspace_bytes < p.ws_bytes) return SKEW_ENOSPACE;
  if ((p.state_bytes > 0 && state == nullptr) || workspace == nullptr) return SKEW_EINVAL;
  const int nt = (int)p.t.size();   // sub-tensors (a stacked tensor's slices are several)
  for (int i = 0; i < nt; i++)
    if (!p.t[i].empty && (d[p.t[i].desc].w == nullptr || d[p.t[i].desc].g == nullptr)) return SKEW_EINVAL;

  char *st = static_cast<char *>(state);
  char *ws = static_cast<char *>(workspace);
  auto sp = [&](size_t off) { return off == SIZE_MAX ? nullptr : reinterpret_cast<float *>(st + off); };
  for (int di = 0; di < n; di++) {   // the caller's view: each descriptor's state from its first slice
    const TensorPlan &tp = p.t[(size_t)p.desc_sub0[(size_t)di]];
    d[di].m = sp(tp.off_m);
    d[di].v = sp(tp.off_v);
    d[di].r = sp(tp.off_r);
    d[di].c = sp(tp.off_c);
  }
  std::vector<DevTensor> table((size_t)(nt > 0 ? nt : 1));
  std::memset(table.data(), 0, sizeof(DevTensor) * table.size());
  for (int i = 0; i < nt; i++) {
    const TensorPlan &tp = p.t[i];
    if (tp.empty) continue;
    const skew_tensor_desc &dd = d[tp.desc];
    // bytes to this slice's first row (elements of 2 bytes, or 4 for float32 masters)
    const int64_t slice = (int64_t)(i - tp.grp0) * tp.n * tp.ld * (tp.fp32 ? 4 : 2);
    DevTensor &x = table[i];
    x.w = reinterpret_cast<uint16_t *>(static_cast<char *>(dd.w) + slice);
    x.g = reinterpret_cast<const uint16_t *>(static_cast<const char *>(dd.g) + slice);
    x.fp32 = tp.fp32;
    x.M = sp(tp.off_m);
    x.V = sp(tp.off_v);
    x.R = sp(tp.off_r);
    x.C = sp(tp.off_c);
    x.idx0 = tp.idx0;
    x.grp0 = tp.grp0;
    x.ngrp = tp.ngrp;
    x.ssum = reinterpret_cast<double *>(ws + tp.off_ssum);
    x.qsum = reinterpret_cast<double *>(ws + tp.off_qsum);
    x.sc = reinterpret_cast<TensorScalars *>(ws + tp.off_sc);
    x.zeros = reinterpret_cast<const uint16_t *>(ws + p.off_zero);
    auto wsp = [&](size_t off) { return off == SIZE_MAX ? nullptr : static_cast<void *>(ws + off); };
    x.rowpart = static_cast<double *>(wsp(tp.off_rowpart));
    x.colpart = static_cast<double *>(wsp(tp.off_colpart));
    x.zpart = static_cast<double *>(wsp(tp.off_zpart));
    x.ainv = static_cast<double *>(wsp(tp.off_ainv));
    x.rsum = static_cast<double *>(wsp(tp.off_rsum));
    x.bst = static_cast<BandStats *>(wsp(tp.off_bst));
    x.cst = static_cast<ColStats *>(wsp(tp.off_cst));
    x.zpath = tp.zpath;
    x.nseg = tp.nseg;
    x.zcw = tp.zcw;
    x.zrpi = tp.zrpi;
    x.nzb = tp.nzb;
    x.zrb = tp.zrb;
    x.zrows = tp.zrows;
    x.n = tp.n;
    x.m = tp.m;
    x.ld = tp.ld;
    x.tr = tp.tr;
    x.cw = tp.cw;
    x.ntc = tp.ntc;
    x.ntr = tp.ntr;
    x.nfr = tp.nfr;
    x.nfc = tp.nfc;
    x.kind = tp.kind;
    x.decay = tp.tier != SKEW_TIER_ROUTER ? 1 : 0;
    x.momentum = tp.momentum;
    x.vec = !tp.fp32 && aligned16(x.w) && aligned16(x.g) && (tp.ld % 8 == 0) && (tp.m % 8 == 0);
    x.tensor_id = dd.tensor_id;
  }
  // row-band pass items by kernel variant (16-byte aligned rows or element loads is known
  // only here, from the pointers); every list keeps tensor order, so each pipeline group
  // is a contiguous range of it
  std::vector<Item> zv[kZVariants];
  for (const Item &it : p.z) {
    const DevTensor &x = table[it.tensor];
    const int lg = x.nseg == 1 ? 0 : (x.nseg == 2 ? 1 : 2);
    zv[lg * 4 + (x.vec ? 0 : 2) + (x.momentum ? 1 : 0)].push_back(it);
  }
  skew_ctx *c = new (std::nothrow) skew_ctx;
  if (c == nullptr) return SKEW_ENOMEM;
  c->d_table = reinterpret_cast<DevTensor *>(ws + p.off_table);
  c->lists = reinterpret_cast<RecheckLists *>(ws + p.off_lists);
  Item *const base = reinterpret_cast<Item *>(ws + p.off_items);
  std::vector<Item> items;
  items.reserve(p.p1.size() + p.z.size() + p.fold.size() + p.p2.size() + p.p3.size() + p.clip.size() +
                p.fold_rows.size() + 1);
  auto add = [&](GroupedList &gl, const std::vector<Item> &v) {
    gl.d = base + items.size();
    gl.bound.assign((size_t)p.ngroups + 1, 0);
    for (const Item &it : v) gl.bound[(size_t)p.tgroup[it.tensor] + 1]++;
    for (int g = 0; g < p.ngroups; g++) gl.bound[g + 1] += gl.bound[g];
    items.insert(items.end(), v.begin(), v.end());
  };
  add(c->p1, p.p1);
  for (int v = 0; v < kZVariants; v++) add(c->z[v], zv[v]);
  add(c->fold, p.fold);
  add(c->p2, p.p2);
  add(c->p3, p.p3);
  add(c->clip, p.clip);
  add(c->fold_rows, p.fold_rows);
  {
    std::vector<Item> fz, fw;
    for (const Item &it : p.fold) (table[it.tensor].zpath ? fz : fw).push_back(it);
    add(c->fold_z, fz);
    add(c->fold_w, fw);
  }
  if (items.empty()) items.push_back({0, 0});
  if (sizeof(Item) * items.size() > p.off_lists - p.off_items) {   // the planner's region must hold them
    delete c;
    return SKEW_EINVAL;
  }
  c->gscale = reinterpret_cast<float *>(ws + p.off_gscale);
  c->gsq = reinterpret_cast<double *>(ws + p.off_gsq);

  hipStream_t s = static_cast<hipStream_t>(stream);
  // the side stream (it takes a hardware queue) runs the update pass of a pipeline of several
  // groups, or the statistics of wide and exact tensors beside the row-band pass
  const bool side = p.ngroups > 1 || !p.p1.empty() || !p.p2.empty();
  hipError_t e = side ? hipStreamCreateWithFlags(&c->side, hipStreamNonBlocking) : hipSuccess;
  for (int i = 0; e == hipSuccess && i < p.ngroups + 3; i++) {
    hipEvent_t ev;
    e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
    if (e == hipSuccess) c->sync.push_back(ev);
  }
  // zero state and workspace (the per-tensor scalars start with no regime prediction)
  if (e == hipSuccess && p.state_bytes > 0) e = hipMemsetAsync(state, 0, p.state_bytes, s);
  if (e == hipSuccess) e = hipMemsetAsync(ws, 0, p.ws_bytes, s);
  if (e == hipSuccess)
    e = hipMemcpyAsync(c->d_table, table.data(), sizeof(DevTensor) * table.size(), hipMemcpyHostToDevice, s);
  if (e == hipSuccess)
    e = hipMemcpyAsync(base, items.data(), sizeof(Item) * items.size(), hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);  // the host staging vectors die on return
  if (e != hipSuccess) {
    delete c;
    return SKEW_EHIP;
  }
  c->plan = std::move(p);
  c->ws = ws;
  *ctx = c;
  return SKEW_OK;
}

// the re-check lists of tensor group g
static RecheckLists *group_lists(skew_ctx *ctx, int g) {
  return reinterpret_cast<RecheckLists *>(reinterpret_cast<unsigned char *>(ctx->lists) +
                                          (size_t)g * ctx->plan.lists_stride);
}

int skew_step(skew_ctx *ctx, const skew_hparams *hp, void *stream) {
  if (ctx == nullptr || !hparams_ok(hp)) return SKEW_EINVAL;
  StepConsts k = make_consts(*hp);
  k.gscale = ctx->gscale;
  k.gsq = ctx->gsq;
  const Plan &p = ctx->plan;
  if (k.gclip && p.ngroups != 1) return SKEW_EINVAL;   // the global norm couples every tensor
  hipStream_t s0 = static_cast<hipStream_t>(stream), s1 = ctx->side;
  std::vector<skew_ctx::Timed> *rec = nullptr;
  if (ctx->ev_used < ctx->ev_steps) {
    rec = &ctx->timed[(size_t)ctx->ev_used++];
    rec->clear();
  }
  int e = 0;
  // one launch of kind j on stream st, bracketed by timing events when recording
  auto run = [&](int j, hipStream_t st, auto &&launch) {
    if (e != 0) return;
    if (rec && ctx->ev_next + 2 <= ctx->ev_pool.size()) {
      skew_ctx::Timed t{j, ctx->ev_pool[ctx->ev_next], ctx->ev_pool[ctx->ev_next + 1]};
      ctx->ev_next += 2;
      e = (int)hipEventRecord(t.a, st);
      if (e == 0) e = launch();
      if (e == 0) e = (int)hipEventRecord(t.b, st);
      rec->push_back(t);
    } else {
      e = launch();
    }
  };
  const DevTensor *T = ctx->d_table;
  // the side stream starts after everything the caller queued before the step
  if (p.ngroups > 1) {
    e = (int)hipEventRecord(ctx->sync[0], s0);
    if (e == 0) e = (int)hipStreamWaitEvent(s1, ctx->sync[0], 0);
  }
  const int nt = (int)p.t.size();
  for (int g = 0; g < p.ngroups && e == 0; g++) {
    // pass 1, fold and clip stage of group g on the caller's stream
    bool p2_done = false;
    if (!k.gclip && p.ngroups == 1 && s1 != nullptr) {
      // the wide tensors' pass 1 and fold and the update sums of wide and exact tensors
      // run on the side stream, beside the row-band pass (which leaves ALU time and
      // registers free); the clip stage waits for both
      e = (int)hipEventRecord(ctx->sync[0], s0);
      if (e == 0) e = (int)hipStreamWaitEvent(s1, ctx->sync[0], 0);
      if (ctx->p1.count(g) > 0) run(2, s1, [&] { return launch_p1(T, ctx->p1.at(g), ctx->p1.count(g), s1); });
      if (ctx->fold_w.count(g) > 0)
        run(3, s1, [&] { return launch_fold(T, ctx->fold_w.at(g), ctx->fold_w.count(g), k, 0, s1); });
      if (ctx->p2.count(g) > 0) run(4, s1, [&] { return launch_p2(T, ctx->p2.at(g), ctx->p2.count(g), k, s1); });
      if (e == 0) e = (int)hipEventRecord(ctx->sync[2 + p.ngroups], s1);
      for (int v = 0; v < kZVariants; v++)
        if (ctx->z[v].count(g) > 0)
          run(v & 1, s0, [&] { return launch_p1z(T, ctx->z[v].at(g), ctx->z[v].count(g), k, v, 0, s0); });
      if (ctx->fold_z.count(g) > 0)
        run(3, s0, [&] { return launch_fold(T, ctx->fold_z.at(g), ctx->fold_z.count(g), k, 0, s0); });
      if (e == 0) e = (int)hipStreamWaitEvent(s0, ctx->sync[2 + p.ngroups], 0);
      p2_done = true;
    } else if (!k.gclip) {
      for (int v = 0; v < kZVariants; v++)
        if (ctx->z[v].count(g) > 0)
          run(v & 1, s0, [&] { return launch_p1z(T, ctx->z[v].at(g), ctx->z[v].count(g), k, v, 0, s0); });
      if (ctx->p1.count(g) > 0) run(2, s0, [&] { return launch_p1(T, ctx->p1.at(g), ctx->p1.count(g), s0); });
      if (ctx->fold.count(g) > 0)
        run(3, s0, [&] { return launch_fold(T, ctx->fold.at(g), ctx->fold.count(g), k, 0, s0); });
    } else {
      // gradient-norm mode (one group): the scale needs every tensor's sum of g^2 before
      // any statistic, so the row-band pass runs twice: sums, then z with R folded
      for (int v = 0; v < kZVariants; v++)
        if (ctx->z[v].count(g) > 0)
          run(v & 1, s0, [&] { return launch_p1z(T, ctx->z[v].at(g), ctx->z[v].count(g), k, v, 1, s0); });
      if (ctx->p1.count(g) > 0) run(2, s0, [&] { return launch_p1(T, ctx->p1.at(g), ctx->p1.count(g), s0); });
      if (ctx->p2.count(g) > 0) run(9, s0, [&] { return launch_gsq(T, ctx->p2.at(g), ctx->p2.count(g), s0); });
      run(9, s0, [&] { return launch_gnorm(T, nt, k, s0); });
      if (ctx->fold_rows.count(g) > 0)
        run(3, s0, [&] { return launch_fold(T, ctx->fold_rows.at(g), ctx->fold_rows.count(g), k, 1, s0); });
      for (int v = 0; v < kZVariants; v++)
        if (ctx->z[v].count(g) > 0)
          run(v & 1, s0, [&] { return launch_p1z(T, ctx->z[v].at(g), ctx->z[v].count(g), k, v, 2, s0); });
      if (ctx->fold.count(g) > 0)
        run(3, s0, [&] { return launch_fold(T, ctx->fold.at(g), ctx->fold.count(g), k, 2, s0); });
    }
    if (!p2_done && ctx->p2.count(g) > 0)
      run(4, s0, [&] { return launch_p2(T, ctx->p2.at(g), ctx->p2.count(g), k, s0); });
    if (ctx->clip.count(g) > 0) {
      RecheckLists *L = group_lists(ctx, g);
      run(5, s0, [&] { return launch_clip(T, ctx->clip.at(g), ctx->clip.count(g), k, L, nt, s0); });
      // re-checks of the tensors the clip stage listed (launches with empty lists exit at once)
      run(6, s0, [&] { return launch_recheck(T, L, nt, k, 1, s0); });
      run(7, s0, [&] { return launch_clip_recheck(T, L, nt, k, 1, s0); });
      run(6, s0, [&] { return launch_recheck(T, L, nt, k, 2, s0); });
      run(7, s0, [&] { return launch_clip_recheck(T, L, nt, k, 2, s0); });
    }
    if (p.ngroups == 1) {
      if (ctx->p3.count(g) > 0)
        run(8, s0, [&] { return launch_p3(T, ctx->p3.at(g), ctx->p3.count(g), k, group_lists(ctx, g), s0); });
      continue;
    }
    if (e == 0) e = (int)hipEventRecord(ctx->sync[2 + g], s0);
    // the update pass of group g on the side stream, concurrent with pass 1 of group g + 1
    if (e == 0) e = (int)hipStreamWaitEvent(s1, ctx->sync[2 + g], 0);
    if (ctx->p3.count(g) > 0)
      run(8, s1, [&] { return launch_p3(T, ctx->p3.at(g), ctx->p3.count(g), k, group_lists(ctx, g), s1); });
  }
  // the caller's stream continues after the last update
  if (e == 0 && p.ngroups > 1) {
    e = (int)hipEventRecord(ctx->sync[1], s1);
    if (e == 0) e = (int)hipStreamWaitEvent(s0, ctx->sync[1], 0);
  }
  return e == 0 ? SKEW_OK : SKEW_EHIP;
}

int skew_timing_enable(skew_ctx *ctx, int max_steps) {
  if (ctx == nullptr || max_steps < 0) return SKEW_EINVAL;
  for (hipEvent_t e : ctx->ev_pool) (void)hipEventDestroy(e);
  ctx->ev_pool.clear();
  ctx->timed.clear();
  ctx->ev_steps = ctx->ev_used = 0;
  ctx->ev_next = 0;
  // at most one launch of each kind per group and step (the row-band variants share two kinds)
  const size_t per_step = (size_t)ctx->plan.ngroups * (kLaunches + 2 * kZVariants + 8) * 2;
  const size_t n = (size_t)max_steps * per_step;
  ctx->ev_pool.reserve(n);
  for (size_t i = 0; i < n; i++) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) {
      for (hipEvent_t x : ctx->ev_pool) (void)hipEventDestroy(x);
      ctx->ev_pool.clear();
      return SKEW_EHIP;
    }
    ctx->ev_pool.push_back(e);
  }
  ctx->timed.resize((size_t)max_steps);
  ctx->ev_steps = max_steps;
  return SKEW_OK;
}

int skew_timing_read(skew_ctx *ctx, double *ms, int max_launches, int *launches, int *steps) {
  if (ctx == nullptr || ms == nullptr || max_launches < kLaunches) return SKEW_EINVAL;
  for (int j = 0; j < kLaunches; j++) ms[j] = 0.0;
  for (int st = 0; st < ctx->ev_used; st++) {
    for (const skew_ctx::Timed &t : ctx->timed[(size_t)st]) {
      float ms1 = 0.f;
      if (hipEventSynchronize(t.b) != hipSuccess || hipEventElapsedTime(&ms1, t.a, t.b) != hipSuccess)
        return SKEW_EHIP;
      ms[t.kind] += ms1;
    }
  }
  if (launches) *launches = kLaunches;
  if (steps) *steps = ctx->ev_used;
  ctx->ev_used = 0;
  ctx->ev_next = 0;
  return SKEW_OK;
}

const char *skew_launch_name(skew_ctx *ctx, int j) {
  (void)ctx;
  return (j >= 0 && j < kLaunches) ? kLaunchNames[j] : "";
}

int skew_clip_info(skew_ctx *ctx, float *k, int32_t *route, int n, void *stream) {
  const int nd = ctx ? (int)ctx->plan.desc_sub0.size() : 0;
  if (ctx == nullptr || k == nullptr || route == nullptr || n < nd) return SKEW_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  // per descriptor: the scalars of its first sub-tensor (a stacked tensor's slices share k)
  const int nt = nd;
  std::vector<TensorScalars> sc((size_t)std::max(nt, 1));
  for (int i = 0; i < nt; i++) {
    const TensorPlan &tp = ctx->plan.t[(size_t)ctx->plan.desc_sub0[(size_t)i]];
    if (tp.empty) {
      std::memset(&sc[i], 0, sizeof(TensorScalars));
      continue;
    }
    if (hipMemcpyAsync(&sc[i], ctx->ws + tp.off_sc, sizeof(TensorScalars), hipMemcpyDeviceToHost, s) != hipSuccess)
      return SKEW_EHIP;
  }
  if (hipStreamSynchronize(s) != hipSuccess) return SKEW_EHIP;
  for (int i = 0; i < nt; i++) {
    k[i] = sc[i].k;
    const TensorPlan &tp = ctx->plan.t[(size_t)ctx->plan.desc_sub0[(size_t)i]];
    route[i] = (sc[i].ambiguous & 0xFF) | ((tp.zpath ? sc[i].regime & 0xFF : 0) << 8);
  }
  return SKEW_OK;
}

void skew_destroy(skew_ctx *ctx) { delete ctx; }

}  // extern "C"

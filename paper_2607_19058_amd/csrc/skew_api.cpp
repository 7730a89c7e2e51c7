// skew_api.cpp -- the C ABI declared in include/skewadam.h.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
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

// a contiguous list of work items in the workspace
struct ItemList {
  const Item *d = nullptr;
  int64_t n = 0;
};

struct skew_ctx {
  Plan plan;
  char *ws = nullptr;   // workspace base (device)
  DevTensor *d_table = nullptr;
  RecheckLists *lists = nullptr;
  ItemList p1, fold, p2, p3, clip, clip_slices, fold_rows;
  float *gscale = nullptr;   // device: the gradient-norm mode's scale
  double *gsq = nullptr;     // device: per-tensor sums of g^2
  ItemList z[kZVariants];    // row-band pass items, one list per kernel variant
  int static_dev = -1;       // >= 0: the workspace is the library's static one on this device
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
  }
};

namespace {

// The context that currently owns each device's static workspace (skew_state_init_static):
// a newer one replaces it, and the older one's steps are then refused.
constexpr int kMaxDevices = 64;
std::mutex g_static_mu;
skew_ctx *g_static_owner[kMaxDevices] = {};

bool static_owner_is(const skew_ctx *c) {
  std::lock_guard<std::mutex> lk(g_static_mu);
  return c->static_dev >= 0 && c->static_dev < kMaxDevices && g_static_owner[c->static_dev] == c;
}

}  // namespace

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
    case SKEW_ESTALE:
      return "this context's static workspace was taken over by a newer skew_state_init_static on its GPU";
    case SKEW_ETOOBIG: return "the table needs more workspace than the library's static workspace holds";
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

}  // extern "C"

namespace {

// Context set-up on a planned table with the workspace `ws` of ws_bytes: fills the state
// pointers of d, zero-fills state and workspace on `stream` and uploads the device table
// and item lists (waiting for the upload: the host staging vectors die on return).
int init_ctx(skew_ctx **ctx, Plan &p, skew_tensor_desc *d, int n, void *state, size_t state_bytes, char *ws,
             size_t ws_bytes, hipStream_t s) {
  if (state_bytes < p.state_bytes || ws_bytes < p.ws_bytes) return SKEW_ENOSPACE;
  if ((p.state_bytes > 0 && state == nullptr) || ws == nullptr) return SKEW_EINVAL;
  const int nt = (int)p.t.size();   // sub-tensors (a stacked tensor's slices are several)
  for (int i = 0; i < nt; i++)
    if (!p.t[i].empty && (d[p.t[i].desc].w == nullptr || d[p.t[i].desc].g == nullptr)) return SKEW_EINVAL;

  char *st = static_cast<char *>(state);
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
  // only here, from the pointers). The aligned variants without momentum and up to two
  // chunks per wave address a block of rows by 32-bit byte offsets; a row stride that makes a
  // block span 2^31 bytes or more takes the element-load variant instead.
  std::vector<Item> zv[kZVariants];
  for (const Item &it : p.z) {
    const DevTensor &x = table[it.tensor];
    const int lg = x.nseg == 1 ? 0 : (x.nseg == 2 ? 1 : (x.nseg == 4 ? 2 : 3));
    const bool wide_span = (int64_t)x.zrpi * x.zrb * x.ld * 2 > 0x7FFFFFFF;
    const bool vec = x.vec && !(wide_span && !x.momentum && x.nseg <= 2);
    zv[lg * 4 + (vec ? 0 : 2) + (x.momentum ? 1 : 0)].push_back(it);
  }
  skew_ctx *c = new (std::nothrow) skew_ctx;
  if (c == nullptr) return SKEW_ENOMEM;
  c->d_table = reinterpret_cast<DevTensor *>(ws + p.off_table);
  c->lists = reinterpret_cast<RecheckLists *>(ws + p.off_lists);
  Item *const base = reinterpret_cast<Item *>(ws + p.off_items);
  std::vector<Item> items;
  items.reserve(p.p1.size() + p.z.size() + p.fold.size() + p.p2.size() + p.p3.size() + p.clip.size() +
                p.clip_slices.size() + p.fold_rows.size() + 1);
  auto add = [&](ItemList &l, const std::vector<Item> &v) {
    l.d = base + items.size();
    l.n = (int64_t)v.size();
    items.insert(items.end(), v.begin(), v.end());
  };
  add(c->p1, p.p1);
  for (int v = 0; v < kZVariants; v++) add(c->z[v], zv[v]);
  add(c->fold, p.fold);
  add(c->p2, p.p2);
  add(c->p3, p.p3);
  add(c->clip, p.clip);
  add(c->clip_slices, p.clip_slices);
  add(c->fold_rows, p.fold_rows);
  if (items.empty()) items.push_back({0, 0});
  if (sizeof(Item) * items.size() > p.off_lists - p.off_items) {   // the planner's region must hold them
    delete c;
    return SKEW_EINVAL;
  }
  c->gscale = reinterpret_cast<float *>(ws + p.off_gscale);
  c->gsq = reinterpret_cast<double *>(ws + p.off_gsq);

  // zero state and workspace (the per-tensor scalars start with no regime prediction)
  hipError_t e = hipSuccess;
  if (p.state_bytes > 0) e = hipMemsetAsync(state, 0, p.state_bytes, s);
  if (e == hipSuccess) e = hipMemsetAsync(ws, 0, p.ws_bytes, s);
  if (e == hipSuccess)
    e = hipMemcpyAsync(c->d_table, table.data(), sizeof(DevTensor) * table.size(), hipMemcpyHostToDevice, s);
  if (e == hipSuccess)
    e = hipMemcpyAsync(base, items.data(), sizeof(Item) * items.size(), hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) {
    delete c;
    return SKEW_EHIP;
  }
  c->plan = std::move(p);
  c->ws = ws;
  *ctx = c;
  return SKEW_OK;
}

}  // namespace

extern "C" {

int skew_state_init(skew_ctx **ctx, skew_tensor_desc *d, int n, void *state, size_t state_bytes, void *workspace,
                    size_t workspace_bytes, void *stream) {
  if (ctx == nullptr) return SKEW_EINVAL;
  *ctx = nullptr;
  Plan p;
  const int rc = plan_build(d, n, &p);
  if (rc != SKEW_OK) return rc;
  return init_ctx(ctx, p, d, n, state, state_bytes, static_cast<char *>(workspace), workspace_bytes,
                  static_cast<hipStream_t>(stream));
}

int skew_state_init_static(skew_ctx **ctx, skew_tensor_desc *d, int n, void *state, size_t state_bytes,
                           void *stream) {
  if (ctx == nullptr) return SKEW_EINVAL;
  *ctx = nullptr;
  Plan p;
  int rc = plan_build(d, n, &p);
  if (rc != SKEW_OK) return rc;
  if (p.ws_bytes > static_workspace_bytes()) return SKEW_ETOOBIG;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return SKEW_EHIP;
  if (dev < 0 || dev >= kMaxDevices) return SKEW_EINVAL;
  void *ws = nullptr;
  if (static_workspace(&ws) != (int)hipSuccess || ws == nullptr) return SKEW_EHIP;
  // the set-up below rewrites the array: from here on an older context on it is stale
  {
    std::lock_guard<std::mutex> lk(g_static_mu);
    g_static_owner[dev] = nullptr;
  }
  rc = init_ctx(ctx, p, d, n, state, state_bytes, static_cast<char *>(ws), static_workspace_bytes(),
                static_cast<hipStream_t>(stream));
  if (rc != SKEW_OK) return rc;
  (*ctx)->static_dev = dev;
  std::lock_guard<std::mutex> lk(g_static_mu);
  g_static_owner[dev] = *ctx;
  return SKEW_OK;
}

int skew_step(skew_ctx *ctx, const skew_hparams *hp, void *stream) {
  if (ctx == nullptr || !hparams_ok(hp)) return SKEW_EINVAL;
  if (ctx->static_dev >= 0 && !static_owner_is(ctx)) return SKEW_ESTALE;
  StepConsts k = make_consts(*hp);
  k.gscale = ctx->gscale;
  k.gsq = ctx->gsq;
  const Plan &p = ctx->plan;
  hipStream_t s = static_cast<hipStream_t>(stream);
  std::vector<skew_ctx::Timed> *rec = nullptr;
  if (ctx->ev_used < ctx->ev_steps) {
    rec = &ctx->timed[(size_t)ctx->ev_used++];
    rec->clear();
  }
  int e = 0;
  // one launch of kind j, bracketed by timing events when recording
  auto run = [&](int j, auto &&launch) {
    if (e != 0) return;
    if (rec && ctx->ev_next + 2 <= ctx->ev_pool.size()) {
      skew_ctx::Timed t{j, ctx->ev_pool[ctx->ev_next], ctx->ev_pool[ctx->ev_next + 1]};
      ctx->ev_next += 2;
      e = (int)hipEventRecord(t.a, s);
      if (e == 0) e = launch();
      if (e == 0) e = (int)hipEventRecord(t.b, s);
      rec->push_back(t);
    } else {
      e = launch();
    }
  };
  const DevTensor *T = ctx->d_table;
  const int nt = (int)p.t.size();
  RecheckLists *L = ctx->lists;
  auto rowband = [&](int mode) {
    for (int v = 0; v < kZVariants; v++)
      if (ctx->z[v].n > 0) run(v & 1, [&] { return launch_p1z(T, ctx->z[v].d, ctx->z[v].n, k, v, mode, s); });
  };
  if (!k.gclip) {
    // statistics: the row-band pass, pass 1 of wide factored tensors, the fold
    rowband(0);
    if (ctx->p1.n > 0) run(2, [&] { return launch_p1(T, ctx->p1.d, ctx->p1.n, s); });
    if (ctx->fold.n > 0) run(3, [&] { return launch_fold(T, ctx->fold.d, ctx->fold.n, k, 0, s); });
  } else {
    // gradient-norm mode: the scale needs every tensor's sum of g^2 before any statistic,
    // so the row-band pass runs twice: sums, then z with R folded
    rowband(1);
    if (ctx->p1.n > 0) run(2, [&] { return launch_p1(T, ctx->p1.d, ctx->p1.n, s); });
    if (ctx->p2.n > 0) run(9, [&] { return launch_gsq(T, ctx->p2.d, ctx->p2.n, s); });
    run(9, [&] { return launch_gnorm(T, nt, k, s); });
    if (ctx->fold_rows.n > 0) run(3, [&] { return launch_fold(T, ctx->fold_rows.d, ctx->fold_rows.n, k, 1, s); });
    rowband(2);
    if (ctx->fold.n > 0) run(3, [&] { return launch_fold(T, ctx->fold.d, ctx->fold.n, k, 2, s); });
  }
  // update sums of wide and exact tensors, the clip stage and its re-checks (launches with
  // empty lists exit at once), then the update
  if (ctx->p2.n > 0) run(4, [&] { return launch_p2(T, ctx->p2.d, ctx->p2.n, k, s); });
  if (ctx->clip.n > 0) {
    if (ctx->clip_slices.n > 0)
      run(5, [&] { return launch_clip_slices(T, ctx->clip_slices.d, ctx->clip_slices.n, k, s); });
    run(5, [&] { return launch_clip(T, ctx->clip.d, ctx->clip.n, k, L, nt, s); });
    run(6, [&] { return launch_recheck(T, L, nt, k, 1, s); });
    run(7, [&] { return launch_clip_recheck(T, L, nt, k, 1, s); });
    run(6, [&] { return launch_recheck(T, L, nt, k, 2, s); });
    run(7, [&] { return launch_clip_recheck(T, L, nt, k, 2, s); });
  }
  if (ctx->p3.n > 0) run(8, [&] { return launch_p3(T, ctx->p3.d, ctx->p3.n, k, L, s); });
  return e == 0 ? SKEW_OK : SKEW_EHIP;
}

int skew_timing_enable(skew_ctx *ctx, int max_steps) {
  if (ctx == nullptr || max_steps < 0) return SKEW_EINVAL;
  for (hipEvent_t e : ctx->ev_pool) (void)hipEventDestroy(e);
  ctx->ev_pool.clear();
  ctx->timed.clear();
  ctx->ev_steps = ctx->ev_used = 0;
  ctx->ev_next = 0;
  // at most one launch of each kind per step (the row-band variants share two kinds)
  const size_t per_step = (size_t)(kLaunches + 2 * kZVariants + 8) * 2;
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

void skew_destroy(skew_ctx *ctx) {
  if (ctx != nullptr && ctx->static_dev >= 0) {
    std::lock_guard<std::mutex> lk(g_static_mu);
    if (g_static_owner[ctx->static_dev] == ctx) g_static_owner[ctx->static_dev] = nullptr;
  }
  delete ctx;
}

}  // extern "C"

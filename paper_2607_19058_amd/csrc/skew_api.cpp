// skew_api.cpp -- the C ABI declared in include/skewadam.h.
#include <hip/hip_runtime_api.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <new>
#include <vector>

#include "skew_internal.h"

using namespace skew;

namespace {
constexpr int kLaunches = 9;
const char *const kLaunchNames[kLaunches] = {"p1z_rowband_stats", "p1z_rowband_stats_other", "p1_rowcol_sumsq",
                                             "fold_rc_ema", "p2_update_sumsq", "clip_factor",
                                             "p2_exact_recheck", "clip_factor_recheck", "p3_apply_dither"};
}  // namespace

struct skew_ctx {
  Plan plan;
  DevTensor *d_table = nullptr;
  Item *d_p1 = nullptr, *d_fold = nullptr, *d_p2 = nullptr, *d_p3 = nullptr, *d_clip = nullptr;
  Item *d_z[kZVariants] = {};     // row-band pass items, one list per kernel variant
  int64_t n_z[kZVariants] = {};
  // diagnostics: events [step][kLaunches + 1]
  std::vector<hipEvent_t> ev;
  int ev_steps = 0, ev_used = 0;
  ~skew_ctx() {
    for (hipEvent_t e : ev) (void)hipEventDestroy(e);
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
  return k;
}

bool hparams_ok(const skew_hparams *hp) {
  if (hp == nullptr) return false;
  if ((hp->flags & ~SKEW_FLAG_EXACT_CLIP) != 0 || hp->step < 1) return false;
  if (!std::isfinite(hp->lr)) return false;
  if (!(hp->beta1 >= 0.0f && hp->beta1 < 1.0f)) return false;
  if (!(hp->beta2 >= 0.0f && hp->beta2 < 1.0f)) return false;
  if (!(hp->eps > 0.0f) || !std::isfinite(hp->eps)) return false;
  if (!(hp->clip_threshold > 0.0f)) return false;  // +inf allowed: no clipping
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
  for (int i = 0; i < n; i++)
    if (!p.t[i].empty && (d[i].w == nullptr || d[i].g == nullptr)) return SKEW_EINVAL;

  char *st = static_cast<char *>(state);
  char *ws = static_cast<char *>(workspace);
  auto sp = [&](size_t off) { return off == SIZE_MAX ? nullptr : reinterpret_cast<float *>(st + off); };
  std::vector<DevTensor> table((size_t)(n > 0 ? n : 1));
  std::memset(table.data(), 0, sizeof(DevTensor) * table.size());
  for (int i = 0; i < n; i++) {
    const TensorPlan &tp = p.t[i];
    d[i].m = sp(tp.off_m);
    d[i].v = sp(tp.off_v);
    d[i].r = sp(tp.off_r);
    d[i].c = sp(tp.off_c);
    if (tp.empty) continue;
    DevTensor &x = table[i];
    x.w = static_cast<uint16_t *>(d[i].w);
    x.g = static_cast<const uint16_t *>(d[i].g);
    x.M = d[i].m;
    x.V = d[i].v;
    x.R = d[i].r;
    x.C = d[i].c;
    x.ssum = reinterpret_cast<double *>(ws + tp.off_ssum);
    x.qsum = reinterpret_cast<double *>(ws + tp.off_qsum);
    x.sc = reinterpret_cast<TensorScalars *>(ws + tp.off_sc);
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
    x.momentum = tp.momentum;
    x.vec = aligned16(d[i].w) && aligned16(d[i].g) && (tp.ld % 8 == 0) && (tp.m % 8 == 0);
    x.tensor_id = d[i].tensor_id;
  }
  // row-band pass items by kernel variant (16-byte aligned rows or element loads is known
  // only here, from the pointers)
  std::vector<Item> zv[kZVariants];
  for (const Item &it : p.z) {
    const DevTensor &x = table[it.tensor];
    const int lg = x.nseg == 1 ? 0 : (x.nseg == 2 ? 1 : 2);
    zv[lg * 4 + (x.vec ? 0 : 2) + (x.momentum ? 1 : 0)].push_back(it);
  }
  std::vector<Item> items;
  items.reserve(p.p1.size() + p.z.size() + p.fold.size() + p.p2.size() + p.p3.size() + p.clip.size() + 1);
  items.insert(items.end(), p.p1.begin(), p.p1.end());
  for (const auto &v : zv) items.insert(items.end(), v.begin(), v.end());
  items.insert(items.end(), p.fold.begin(), p.fold.end());
  items.insert(items.end(), p.p2.begin(), p.p2.end());
  items.insert(items.end(), p.p3.begin(), p.p3.end());
  items.insert(items.end(), p.clip.begin(), p.clip.end());
  if (items.empty()) items.push_back({0, 0});

  skew_ctx *c = new (std::nothrow) skew_ctx;
  if (c == nullptr) return SKEW_ENOMEM;
  c->d_table = reinterpret_cast<DevTensor *>(ws + p.off_table);
  Item *base = reinterpret_cast<Item *>(ws + p.off_items);
  c->d_p1 = base;
  Item *cur = c->d_p1 + p.p1.size();
  for (int v = 0; v < kZVariants; v++) {
    c->d_z[v] = cur;
    c->n_z[v] = (int64_t)zv[v].size();
    cur += zv[v].size();
  }
  c->d_fold = cur;
  c->d_p2 = c->d_fold + p.fold.size();
  c->d_p3 = c->d_p2 + p.p2.size();
  c->d_clip = c->d_p3 + p.p3.size();

  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipSuccess;
  if (p.state_bytes > 0) e = hipMemsetAsync(state, 0, p.state_bytes, s);
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
  *ctx = c;
  return SKEW_OK;
}

int skew_step(skew_ctx *ctx, const skew_hparams *hp, void *stream) {
  if (ctx == nullptr || !hparams_ok(hp)) return SKEW_EINVAL;
  const StepConsts k = make_consts(*hp);
  const Plan &p = ctx->plan;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipEvent_t *ev = nullptr;
  if (ctx->ev_used < ctx->ev_steps) ev = &ctx->ev[(size_t)ctx->ev_used++ * (kLaunches + 1)];
  int e = ev ? (int)hipEventRecord(ev[0], s) : 0;
  // launch j of the step, then (with timing on) the event that ends it
  auto run = [&](int j, int rc) {
    if (e == 0) e = rc;
    if (e == 0 && ev) e = (int)hipEventRecord(ev[j + 1], s);
  };
  const DevTensor *T = ctx->d_table;
  // row-band pass: the main variant (aligned rows, no momentum) is launch 0, the rest launch 1
  if (e == 0) run(0, launch_p1z(T, ctx->d_z[0], ctx->n_z[0], k, 0, stream));
  if (e == 0) {
    int rc = 0;
    for (int v = 1; v < kZVariants && rc == 0; v++) rc = launch_p1z(T, ctx->d_z[v], ctx->n_z[v], k, v, stream);
    run(1, rc);
  }
  if (e == 0) run(2, launch_p1(T, ctx->d_p1, (int64_t)p.p1.size(), stream));
  if (e == 0) run(3, launch_fold(T, ctx->d_fold, (int64_t)p.fold.size(), k, stream));
  if (e == 0) run(4, launch_p2(T, ctx->d_p2, (int64_t)p.p2.size(), k, stream));
  if (e == 0) run(5, launch_clip(T, ctx->d_clip, (int64_t)p.clip.size(), k, 0, stream));
  // the exact re-check runs over every tile; tensors the clip stage did not flag exit at once
  if (e == 0) run(6, launch_p2_exact(T, ctx->d_p3, (int64_t)p.p3.size(), k, stream));
  if (e == 0) run(7, launch_clip(T, ctx->d_clip, (int64_t)p.clip.size(), k, 1, stream));
  if (e == 0) run(8, launch_p3(T, ctx->d_p3, (int64_t)p.p3.size(), k, stream));
  return e == 0 ? SKEW_OK : SKEW_EHIP;
}

int skew_timing_enable(skew_ctx *ctx, int max_steps) {
  if (ctx == nullptr || max_steps < 0) return SKEW_EINVAL;
  for (hipEvent_t e : ctx->ev) (void)hipEventDestroy(e);
  ctx->ev.clear();
  ctx->ev_steps = ctx->ev_used = 0;
  const size_t n = (size_t)max_steps * (kLaunches + 1);
  ctx->ev.reserve(n);
  for (size_t i = 0; i < n; i++) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) {
      for (hipEvent_t x : ctx->ev) (void)hipEventDestroy(x);
      ctx->ev.clear();
      return SKEW_EHIP;
    }
    ctx->ev.push_back(e);
  }
  ctx->ev_steps = max_steps;
  return SKEW_OK;
}

int skew_timing_read(skew_ctx *ctx, double *ms, int max_launches, int *launches, int *steps) {
  if (ctx == nullptr || ms == nullptr || max_launches < kLaunches) return SKEW_EINVAL;
  for (int j = 0; j < kLaunches; j++) ms[j] = 0.0;
  for (int st = 0; st < ctx->ev_used; st++) {
    hipEvent_t *ev = &ctx->ev[(size_t)st * (kLaunches + 1)];
    if (hipEventSynchronize(ev[kLaunches]) != hipSuccess) return SKEW_EHIP;
    for (int j = 0; j < kLaunches; j++) {
      float t = 0.f;
      if (hipEventElapsedTime(&t, ev[j], ev[j + 1]) != hipSuccess) return SKEW_EHIP;
      ms[j] += t;
    }
  }
  if (launches) *launches = kLaunches;
  if (steps) *steps = ctx->ev_used;
  ctx->ev_used = 0;
  return SKEW_OK;
}

const char *skew_launch_name(skew_ctx *ctx, int j) {
  (void)ctx;
  return (j >= 0 && j < kLaunches) ? kLaunchNames[j] : "";
}

void skew_destroy(skew_ctx *ctx) { delete ctx; }

}  // extern "C"

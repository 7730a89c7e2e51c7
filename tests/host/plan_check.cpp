// plan_check.cpp -- host-only checks of the planner and of the C ABI's host code, built
// with AddressSanitizer and UndefinedBehaviorSanitizer by tests/test_host_sanitized.py.
//
// No GPU is involved: the few HIP runtime calls of the C ABI are replaced below by
// versions that act on host memory (the "device" buffers are host allocations), and the
// kernel launchers by versions that check every work item they are handed against the
// device table the set-up wrote. Checked for each descriptor table:
//   * every row and every column of every sub-tensor lies in exactly one update tile
//     (p3), and in exactly one row band (row-band pass) or pass-1 tile (wide tensors);
//     a tile is a set of rows times a set of columns, so this covers every element, also
//     for tensors of more than 2^31 elements (64-bit tiling, Sec. 3 "Memory model" footnote);
//   * the row-band geometry fits the kernel: a block fits one LDS staging buffer, a band
//     holds whole blocks, every 512-column chunk of a row has exactly one wave;
//   * every state and workspace region is 256-byte aligned, lies inside its buffer and
//     overlaps no other region;
//   * the set-up and a step over the table launch exactly the planned items, each naming a
//     tensor and tile that exist, with the table's pointers inside the caller's buffers.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <set>
#include <string>
#include <vector>

#include "../../paper_2607_19058_amd/csrc/skew_internal.h"

using namespace skew;

static int g_fail = 0;
static long g_checks = 0;
#define CHECK(cond, ...)                                        \
  do {                                                          \
    g_checks++;                                                 \
    if (!(cond)) {                                              \
      if (g_fail < 40) {                                        \
        std::printf("FAIL %s:%d: %s: ", __FILE__, __LINE__, #cond); \
        std::printf(__VA_ARGS__);                               \
        std::printf("\n");                                      \
      }                                                         \
      g_fail++;                                                 \
    }                                                           \
  } while (0)

// ---- HIP runtime calls of the C ABI, acting on host memory ----
extern "C" {
hipError_t hipMemsetAsync(void *dst, int value, size_t n, hipStream_t) {
  std::memset(dst, value, n);
  return hipSuccess;
}
hipError_t hipMemcpyAsync(void *dst, const void *src, size_t n, hipMemcpyKind, hipStream_t) {
  std::memcpy(dst, src, n);
  return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
hipError_t hipGetDevice(int *d) {
  *d = 0;
  return hipSuccess;
}
hipError_t hipEventCreate(hipEvent_t *e) {
  *e = reinterpret_cast<hipEvent_t>(new char[8]);
  return hipSuccess;
}
hipError_t hipEventDestroy(hipEvent_t e) {
  delete[] reinterpret_cast<char *>(e);
  return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hipSuccess; }
hipError_t hipEventSynchronize(hipEvent_t) { return hipSuccess; }
hipError_t hipEventElapsedTime(float *ms, hipEvent_t, hipEvent_t) {
  *ms = 0.f;
  return hipSuccess;
}
}

// ---- kernel launchers: record and check the items each launch covers ----
struct Buffers {
  const char *state = nullptr, *ws = nullptr;
  size_t state_bytes = 0, ws_bytes = 0;
  int nt = 0;
};
static Buffers g_buf;
static std::map<std::string, std::multiset<std::pair<int, int>>> g_launched;

static void check_items(const char *kind, const DevTensor *T, const Item *items, int64_t count) {
  const char *ib = reinterpret_cast<const char *>(items);
  CHECK(ib >= g_buf.ws && ib + count * sizeof(Item) <= g_buf.ws + g_buf.ws_bytes, "%s: item list outside workspace",
        kind);
  CHECK(reinterpret_cast<const char *>(T) >= g_buf.ws, "%s: table outside workspace", kind);
  for (int64_t q = 0; q < count; q++) {
    const Item it = items[q];
    CHECK(it.tensor >= 0 && it.tensor < g_buf.nt, "%s: tensor %d of %d", kind, it.tensor, g_buf.nt);
    if (it.tensor < 0 || it.tensor >= g_buf.nt) continue;
    g_launched[kind].insert({it.tensor, it.tile});
  }
}
namespace skew {
int launch_p1(const DevTensor *T, const Item *items, int64_t count, void *) {
  check_items("p1", T, items, count);
  return 0;
}
int launch_p1z(const DevTensor *T, const Item *items, int64_t count, const StepConsts &, int variant, int mode,
               void *) {
  check_items(mode == 0 ? "z0" : (mode == 1 ? "z1" : "z2"), T, items, count);
  for (int64_t q = 0; q < count; q++) {
    const DevTensor &t = T[items[q].tensor];
    const int lg = t.nseg == 1 ? 0 : (t.nseg == 2 ? 1 : (t.nseg == 4 ? 2 : 3));
    // the aligned variants without momentum and up to two chunks per wave address a block by
    // 32-bit offsets: a wider block span takes the element-load variant
    const bool wide_span = (int64_t)t.zrpi * t.zrb * t.ld * 2 > 0x7FFFFFFF;
    const bool vec = t.vec && !(wide_span && !t.momentum && t.nseg <= 2);
    CHECK(variant == lg * 4 + (vec ? 0 : 2) + (t.momentum ? 1 : 0), "row-band variant %d", variant);
  }
  return 0;
}
int launch_fold(const DevTensor *T, const Item *items, int64_t count, const StepConsts &, int phase, void *) {
  check_items(phase == 1 ? "fold_rows" : "fold", T, items, count);
  return 0;
}
int launch_gsq(const DevTensor *T, const Item *items, int64_t count, void *) {
  check_items("gsq", T, items, count);
  return 0;
}
int launch_gnorm(const DevTensor *, int, const StepConsts &, void *) { return 0; }
int launch_p2(const DevTensor *T, const Item *items, int64_t count, const StepConsts &, void *) {
  check_items("p2", T, items, count);
  return 0;
}
int launch_p3(const DevTensor *T, const Item *items, int64_t count, const StepConsts &, RecheckLists *, void *) {
  check_items("p3", T, items, count);
  return 0;
}
int launch_clip(const DevTensor *T, const Item *items, int64_t count, const StepConsts &, RecheckLists *, int, void *) {
  check_items("clip", T, items, count);
  return 0;
}
int launch_clip_slices(const DevTensor *T, const Item *items, int64_t count, const StepConsts &, void *) {
  check_items("clip_slices", T, items, count);
  return 0;
}
int launch_recheck(const DevTensor *, RecheckLists *, int, const StepConsts &, int, void *) { return 0; }
int launch_clip_recheck(const DevTensor *, RecheckLists *, int, const StepConsts &, int, void *) { return 0; }
int static_workspace(void **ptr) {
  static std::vector<char> buf(static_workspace_bytes());
  *ptr = buf.data();
  return 0;
}
}  // namespace skew

// ---- the checks ----
static int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

struct Region {
  size_t a, b;
  std::string what;
};
static void check_regions(std::vector<Region> r, size_t limit, const char *buf) {
  for (const Region &x : r) {
    CHECK(x.a % kAlign == 0, "%s region %s at %zu not 256-byte aligned", buf, x.what.c_str(), x.a);
    CHECK(x.b <= limit, "%s region %s ends at %zu past %zu", buf, x.what.c_str(), x.b, limit);
  }
  std::sort(r.begin(), r.end(), [](const Region &p, const Region &q) { return p.a < q.a; });
  for (size_t i = 1; i < r.size(); i++)
    CHECK(r[i].a >= r[i - 1].b, "%s regions %s [%zu, %zu) and %s [%zu, %zu) overlap", buf, r[i - 1].what.c_str(),
          r[i - 1].a, r[i - 1].b, r[i].what.c_str(), r[i].a, r[i].b);
}

static void check_plan(const std::string &name, const std::vector<skew_tensor_desc> &d) {
  Plan p;
  const int rc = plan_build(d.data(), (int)d.size(), &p);
  CHECK(rc == SKEW_OK, "%s: plan_build %d", name.c_str(), rc);
  if (rc != SKEW_OK) return;
  const int nt = (int)p.t.size();
  std::vector<Region> st, ws;
  std::set<std::pair<int, int>> p3, z, p1, fold, p2, clip;
  for (const Item &it : p.p3) CHECK(p3.insert({it.tensor, it.tile}).second, "%s: p3 item repeated", name.c_str());
  for (const Item &it : p.z) CHECK(z.insert({it.tensor, it.tile}).second, "%s: band item repeated", name.c_str());
  for (const Item &it : p.p1) CHECK(p1.insert({it.tensor, it.tile}).second, "%s: p1 item repeated", name.c_str());
  for (const Item &it : p.fold) CHECK(fold.insert({it.tensor, it.tile}).second, "%s: fold item repeated", name.c_str());
  for (const Item &it : p.p2) CHECK(p2.insert({it.tensor, it.tile}).second, "%s: p2 item repeated", name.c_str());
  for (const Item &it : p.clip) CHECK(clip.insert({it.tensor, it.tile}).second, "%s: clip item repeated", name.c_str());
  size_t n_p3 = 0, n_z = 0, n_p1 = 0, n_fold = 0, n_p2 = 0, n_clip = 0;
  for (int i = 0; i < nt; i++) {
    const TensorPlan &tp = p.t[i];
    const std::string tn = name + "[" + std::to_string(i) + "]";
    if (tp.empty) continue;
    const int64_t E = tp.ngrp;
    // state: one array per descriptor, held by its first slice
    if (i == tp.grp0) {
      if (tp.off_m != SIZE_MAX) st.push_back({tp.off_m, tp.off_m + (size_t)(E * tp.N) * 4, tn + ".m"});
      if (tp.off_v != SIZE_MAX) st.push_back({tp.off_v, tp.off_v + (size_t)(E * tp.N) * 4, tn + ".v"});
      if (tp.off_r != SIZE_MAX) st.push_back({tp.off_r, tp.off_r + (size_t)(E * tp.n) * 4, tn + ".r"});
      if (tp.off_c != SIZE_MAX) st.push_back({tp.off_c, tp.off_c + (size_t)(E * tp.m) * 4, tn + ".c"});
      n_clip++;
      CHECK(clip.count({i, 0}), "%s: no clip item", tn.c_str());
    } else {
      const TensorPlan &t0 = p.t[tp.grp0];
      const size_t e = (size_t)(i - tp.grp0);
      if (tp.off_m != SIZE_MAX) CHECK(tp.off_m == t0.off_m + e * tp.N * 4, "%s: slice m", tn.c_str());
      if (tp.off_r != SIZE_MAX) CHECK(tp.off_r == t0.off_r + e * tp.n * 4, "%s: slice r", tn.c_str());
      if (tp.off_c != SIZE_MAX) CHECK(tp.off_c == t0.off_c + e * tp.m * 4, "%s: slice c", tn.c_str());
      CHECK(tp.idx0 == (int64_t)e * tp.N, "%s: slice element offset", tn.c_str());
    }
    CHECK((tp.kind == kExact) == (tp.off_v != SIZE_MAX), "%s: exact tensors keep V", tn.c_str());
    CHECK((tp.kind == kFactored) == (tp.off_r != SIZE_MAX && tp.off_c != SIZE_MAX), "%s: R, C", tn.c_str());
    CHECK((tp.momentum != 0) == (tp.off_m != SIZE_MAX), "%s: momentum", tn.c_str());
    // update tiles: band b holds rows b, b + ntr, ...; strip s columns [s 512 cw, (s + 1) 512 cw)
    const int64_t tc = (int64_t)kChunk * tp.cw;
    CHECK(tp.cw == 1 || tp.cw == 2 || tp.cw == 4, "%s: cw", tn.c_str());
    CHECK((int64_t)tp.ntc * tc >= tp.m && (int64_t)(tp.ntc - 1) * tc < tp.m, "%s: strips cover columns once",
          tn.c_str());
    CHECK((int64_t)tp.ntr <= tp.n && (int64_t)tp.ntr * tp.tr >= tp.n, "%s: bands", tn.c_str());
    // each row in exactly one band: row i is in band i % ntr at local row i / ntr, and band
    // b has ceil((n - b) / ntr) rows, so the local rows of band b are exactly its rows
    int64_t rows_seen = 0;
    for (int64_t b = 0; b < tp.ntr; b++) rows_seen += cdiv(tp.n - b, tp.ntr);
    CHECK(rows_seen == tp.n, "%s: bands hold %lld rows of %lld", tn.c_str(), (long long)rows_seen, (long long)tp.n);
    for (int64_t k = 0; k < (int64_t)tp.ntr * tp.ntc; k++) {
      CHECK(p3.count({i, (int)k}) == 1, "%s: update tile %lld", tn.c_str(), (long long)k);
      n_p3++;
    }
    // workspace regions of the tensor
    const int64_t tiles = (int64_t)tp.ntr * tp.ntc;
    ws.push_back({tp.off_ssum, tp.off_ssum + (size_t)tiles * kSub * 8, tn + ".ssum"});
    ws.push_back({tp.off_qsum, tp.off_qsum + (size_t)tiles * kSub * 8, tn + ".qsum"});
    ws.push_back({tp.off_sc, tp.off_sc + sizeof(TensorScalars), tn + ".sc"});
    if (tp.zpath) {
      // row bands: rows [b zrows, min((b + 1) zrows, n)), whole blocks of rpi * zrb rows
      const int64_t blk = (int64_t)tp.zrpi * tp.zrb;
      CHECK(tp.zrows % blk == 0 && tp.zrows <= kZMaxBandRows && blk <= kZMaxBlockRows, "%s: band geometry",
            tn.c_str());
      CHECK((int64_t)tp.nzb * tp.zrows >= tp.n && (int64_t)(tp.nzb - 1) * tp.zrows < tp.n, "%s: bands cover rows once",
            tn.c_str());
      const int64_t wpr = cdiv(tp.zcw, tp.nseg);
      CHECK(tp.zcw == cdiv(tp.m, kChunk) && wpr * tp.zrpi <= kZWaves && tp.zcw <= wpr * tp.nseg &&
                tp.nseg <= kZMaxSeg,
            "%s: chunk layout zcw %d nseg %d rpi %d", tn.c_str(), tp.zcw, tp.nseg, tp.zrpi);
      const int64_t block_bytes = blk * tp.zcw * 1024 * (tp.momentum ? 3 : 1);
      CHECK(block_bytes <= kZLdsBytes, "%s: block of %lld bytes", tn.c_str(), (long long)block_bytes);
      CHECK(tp.nseg != 3 || (!tp.momentum && tp.zrb <= 2), "%s: three chunks per wave without momentum, 2 rows",
            tn.c_str());
      for (int b = 0; b < tp.nzb; b++) {
        CHECK(z.count({i, b}) == 1, "%s: band %d", tn.c_str(), b);
        n_z++;
      }
      for (int c = 0; c < tp.nfc; c++) n_fold += fold.count({i, c});
      CHECK(tp.nfc == cdiv(tp.m, kFold), "%s: fold chunks", tn.c_str());
      ws.push_back({tp.off_colpart, tp.off_colpart + (size_t)tp.nzb * tp.m * 8, tn + ".colpart"});
      ws.push_back({tp.off_zpart, tp.off_zpart + (size_t)tp.nzb * tp.m * 8, tn + ".zpart"});
      ws.push_back({tp.off_ainv, tp.off_ainv + (size_t)tp.n * 8, tn + ".ainv"});
      ws.push_back({tp.off_bst, tp.off_bst + (size_t)tp.nzb * sizeof(BandStats), tn + ".bst"});
      ws.push_back({tp.off_cst, tp.off_cst + (size_t)tp.nfc * sizeof(ColStats), tn + ".cst"});
      ws.push_back({tp.off_rsum, tp.off_rsum + (size_t)cdiv(tp.n, kFold) * 8, tn + ".rsum"});
    } else if (tp.kind == kFactored) {
      for (int64_t k = 0; k < tiles; k++) {
        CHECK(p1.count({i, (int)k}) == 1, "%s: pass-1 tile %lld", tn.c_str(), (long long)k);
        n_p1++;
      }
      CHECK(tp.nfr == cdiv(tp.n, kFold) && tp.nfc == cdiv(tp.m, kFold), "%s: fold chunks", tn.c_str());
      for (int c = 0; c < tp.nfr + tp.nfc; c++) n_fold += fold.count({i, c});
      ws.push_back({tp.off_rowpart, tp.off_rowpart + (size_t)tp.ntc * tp.n * 8, tn + ".rowpart"});
      ws.push_back({tp.off_colpart, tp.off_colpart + (size_t)tp.ntr * tp.m * 8, tn + ".colpart"});
      ws.push_back({tp.off_ainv, tp.off_ainv + (size_t)tp.n * 8, tn + ".ainv"});
      ws.push_back({tp.off_rsum, tp.off_rsum + (size_t)tp.nfr * 8, tn + ".rsum"});
      ws.push_back({tp.off_cst, tp.off_cst + (size_t)(tp.nfr + tp.nfc) * sizeof(ColStats), tn + ".cst"});
    }
    if (!tp.zpath)
      for (int64_t k = 0; k < tiles * kSub; k++) {
        CHECK(p2.count({i, (int)k}) == 1, "%s: update-sum item %lld", tn.c_str(), (long long)k);
        n_p2++;
      }
  }
  CHECK(n_p3 == p.p3.size() && n_z == p.z.size() && n_p1 == p.p1.size() && n_p2 == p.p2.size() &&
            n_fold == p.fold.size() && n_clip == p.clip.size(),
        "%s: item lists hold items of no tensor", name.c_str());
  check_regions(st, p.state_bytes, (name + " state").c_str());
  const size_t nt1 = (size_t)std::max(nt, 1);
  ws.push_back({p.off_table, p.off_table + sizeof(DevTensor) * nt1, "table"});
  ws.push_back({p.off_items, p.off_lists, "items"});
  ws.push_back({p.off_lists, p.off_lists + sizeof(RecheckLists) + 8 * nt1, "lists"});
  ws.push_back({p.off_zero, p.off_zero + 256, "zero"});
  ws.push_back({p.off_gscale, p.off_gscale + 4, "gscale"});
  ws.push_back({p.off_gsq, p.off_gsq + 8 * nt1, "gsq"});
  check_regions(ws, p.ws_bytes, (name + " workspace").c_str());
}

// set-up and one step on host stand-ins of every buffer (tables small enough to allocate)
static void check_init_and_step(const std::string &name, std::vector<skew_tensor_desc> d, bool gnorm) {
  size_t sb = 0, wb = 0;
  CHECK(skew_state_bytes(d.data(), (int)d.size(), &sb, &wb) == SKEW_OK, "%s: sizes", name.c_str());
  std::vector<char> state(sb + 1), ws(wb + 1);
  std::vector<std::vector<char>> data;
  for (auto &x : d) {
    const int64_t E = x.ndim == 3 ? x.batch : 1;
    const size_t bytes = (size_t)(E * (x.ndim == 1 ? x.rows * x.cols : x.rows * x.ld)) *
                         ((x.state_flags & SKEW_STATE_FP32) ? 4 : 2) + 16;
    data.emplace_back(bytes);
    x.w = data.back().data();
    data.emplace_back(bytes);
    x.g = data.back().data();
  }
  g_buf = Buffers{state.data(), ws.data(), sb, wb, 0};
  Plan p;
  plan_build(d.data(), (int)d.size(), &p);
  g_buf.nt = (int)p.t.size();
  skew_ctx *ctx = nullptr;
  CHECK(skew_state_init(&ctx, d.data(), (int)d.size(), state.data(), sb, ws.data(), wb, nullptr) == SKEW_OK,
        "%s: init", name.c_str());
  if (!ctx) return;
  // the device table the set-up wrote: every pointer inside the caller's buffers
  const DevTensor *T = reinterpret_cast<const DevTensor *>(ws.data() + p.off_table);
  for (int i = 0; i < g_buf.nt; i++) {
    const TensorPlan &tp = p.t[i];
    if (tp.empty) continue;
    const DevTensor &t = T[i];
    auto in_state = [&](const float *q, size_t n) {
      const char *c = reinterpret_cast<const char *>(q);
      return q == nullptr || (c >= state.data() && c + n * 4 <= state.data() + sb);
    };
    auto in_ws = [&](const void *q, size_t n) {
      const char *c = static_cast<const char *>(q);
      return q == nullptr || (c >= ws.data() && c + n <= ws.data() + wb);
    };
    CHECK(in_state(t.M, (size_t)tp.N) && in_state(t.V, (size_t)tp.N) && in_state(t.R, (size_t)tp.n) &&
              in_state(t.C, (size_t)tp.m),
          "%s[%d]: state pointers", name.c_str(), i);
    CHECK(in_ws(t.ssum, (size_t)t.ntr * t.ntc * kSub * 8) && in_ws(t.sc, sizeof(TensorScalars)) &&
              in_ws(t.zeros, 256),
          "%s[%d]: workspace pointers", name.c_str(), i);
    CHECK(t.n == tp.n && t.m == tp.m && t.ld == tp.ld && t.zpath == tp.zpath && t.nzb == tp.nzb,
          "%s[%d]: table fields", name.c_str(), i);
  }
  g_launched.clear();
  skew_hparams hp{3e-4f, 0.9f, 0.999f, 1e-8f, 1.0f, 0, 1, 0, 0.0f, gnorm ? 1.0f : 0.0f};
  CHECK(skew_step(ctx, &hp, nullptr) == SKEW_OK, "%s: step", name.c_str());
  auto same = [&](const char *kind, const std::vector<Item> &v) {
    std::multiset<std::pair<int, int>> want;
    for (const Item &it : v) want.insert({it.tensor, it.tile});
    CHECK(g_launched[kind] == want, "%s: %s launched %zu items, planned %zu", name.c_str(), kind,
          g_launched[kind].size(), want.size());
  };
  same("p3", p.p3);
  same("clip", p.clip);
  same("clip_slices", p.clip_slices);
  {
    // the clip stage's slice items: every non-empty slice of a stacked tensor, once
    std::multiset<std::pair<int, int>> want;
    for (int i = 0; i < g_buf.nt; i++)
      if (!p.t[i].empty && p.t[i].ngrp > 1) want.insert({i, 0});
    std::multiset<std::pair<int, int>> got;
    for (const Item &it : p.clip_slices) got.insert({it.tensor, it.tile});
    CHECK(got == want, "%s: clip slice items %zu, stacked slices %zu", name.c_str(), got.size(), want.size());
  }
  same("p1", p.p1);
  same(gnorm ? "z1" : "z0", p.z);
  if (gnorm) {
    same("z2", p.z);
    same("fold_rows", p.fold_rows);
  }
  same("fold", p.fold);
  same("p2", p.p2);
  // bad hyper-parameters launch nothing
  g_launched.clear();
  skew_hparams bad = hp;
  bad.step = 0;
  CHECK(skew_step(ctx, &bad, nullptr) == SKEW_EINVAL && g_launched.empty(), "%s: step 0 refused", name.c_str());
  skew_destroy(ctx);
}

static skew_tensor_desc mk(int tier, int ndim, int64_t rows, int64_t cols, int64_t ld, uint64_t id, int64_t batch = 0,
                           uint32_t flags = 0) {
  skew_tensor_desc x;
  std::memset(&x, 0, sizeof x);
  x.tier = tier;
  x.ndim = ndim;
  x.rows = rows;
  x.cols = cols;
  x.ld = ld;
  x.tensor_id = id;
  x.batch = batch;
  x.state_flags = flags;
  x.w = reinterpret_cast<void *>(0x1000);
  x.g = reinterpret_cast<const void *>(0x1000);
  return x;
}

int main() {
  std::vector<skew_tensor_desc> unit, ragged, big, stacked, variants;
  const int64_t shapes[][2] = {{1, 1},  {1, 7},    {7, 1},     {3, 5},      {13, 17},   {256, 8},   {64, 520},
                               {33, 1031}, {2, 2048}, {300, 2056}, {1000, 1000}, {17, 8200}, {5, 11008}, {3, 16384},
                               {2, 16392}, {2, 50304}};
  uint64_t id = 0;
  for (int tier = 0; tier < 3; tier++) {
    for (auto &s : shapes) unit.push_back(mk(tier, 2, s[0], s[1], s[1] + (id % 3) * 8, id++));
    for (int64_t len : {1, 5, 4097}) unit.push_back(mk(tier, 1, 1, len, len, id++));
    unit.push_back(mk(tier, 2, 0, 64, 64, id++));   // empty
    unit.push_back(mk(tier, 1, 1, 0, 1, id++));
  }
  // the ragged tier mix: 4 x 4096^2 + 8 vectors; 64 x {1536x6144, 6144x1536} + 64 x {4096x11008, 11008x4096}
  for (int k = 0; k < 4; k++) ragged.push_back(mk(0, 2, 4096, 4096, 4096, id++));
  for (int k = 0; k < 8; k++) ragged.push_back(mk(0, 1, 1, 4096, 4096, id++));
  for (int e = 0; e < 64; e++) {
    ragged.push_back(mk(1, 2, 1536, 6144, 6144, id++));
    ragged.push_back(mk(1, 2, 6144, 1536, 1536, id++));
  }
  for (int e = 0; e < 64; e++) {
    ragged.push_back(mk(1, 2, 4096, 11008, 11008, id++));
    ragged.push_back(mk(1, 2, 11008, 4096, 4096, id++));
  }
  ragged.push_back(mk(2, 2, 4096, 64, 64, id++));
  // more than 2^31 elements
  big.push_back(mk(1, 2, 65537, 32768, 32768, id++));
  big.push_back(mk(0, 1, 1, (int64_t(1) << 31) + 3, 1, id++));
  big.push_back(mk(1, 3, 4096, 4096, 4096, id++, 129));
  big.push_back(mk(0, 2, 50304, 2048, 2048, id++));
  big.push_back(mk(0, 2, 2048, 50304, 50304, id++));
  // stacked and empty stacks
  stacked.push_back(mk(1, 3, 256, 1024, 1024, id++, 8));
  stacked.push_back(mk(1, 3, 64, 0, 64, id++, 3));
  stacked.push_back(mk(1, 3, 64, 64, 64, id++, 0));
  stacked.push_back(mk(0, 3, 33, 520, 528, id++, 3));
  // tier variants (Table 3) and float32 masters
  for (uint32_t f : {1u, 2u, 3u}) {
    variants.push_back(mk(1, 2, 256, 1024, 1024, id++, 0, f));
    variants.push_back(mk(2, 2, 256, 8, 8, id++, 0, f));
    variants.push_back(mk(0, 1, 1, 300, 300, id++, 0, f));
  }
  variants.push_back(mk(2, 2, 64, 8, 8, id++, 0, 4));
  variants.push_back(mk(0, 1, 1, 77, 77, id++, 0, 4));

  check_plan("unit", unit);
  check_plan("ragged", ragged);
  check_plan("big", big);
  check_plan("stacked", stacked);
  check_plan("variants", variants);
  for (bool gn : {false, true}) {
    check_init_and_step(gn ? "unit+gnorm" : "unit", unit, gn);
    check_init_and_step(gn ? "stacked+gnorm" : "stacked", stacked, gn);
    check_init_and_step(gn ? "variants+gnorm" : "variants", variants, gn);
  }
  // the static workspace: a second set-up on the same device makes the first one stale
  {
    std::vector<skew_tensor_desc> d = unit;
    std::vector<std::vector<char>> data;
    for (auto &x : d) {
      data.emplace_back((size_t)(x.ndim == 1 ? x.rows * x.cols : x.rows * x.ld) * 2 + 16);
      x.w = data.back().data();
      x.g = data.back().data();
    }
    size_t sb = 0, wb = 0;
    skew_state_bytes(d.data(), (int)d.size(), &sb, &wb);
    std::vector<char> s1(sb), s2(sb);
    skew_ctx *a = nullptr, *b = nullptr;
    g_buf = Buffers{nullptr, nullptr, 0, 0, 0};
    g_buf.ws = nullptr;
    CHECK(skew_state_init_static(&a, d.data(), (int)d.size(), s1.data(), sb, nullptr) == SKEW_OK, "static init 1");
    CHECK(skew_state_init_static(&b, d.data(), (int)d.size(), s2.data(), sb, nullptr) == SKEW_OK, "static init 2");
    skew_hparams hp{3e-4f, 0.9f, 0.999f, 1e-8f, 1.0f, 0, 1, 0, 0.0f, 0.0f};
    void *sw = nullptr;
    static_workspace(&sw);
    g_buf = Buffers{s2.data(), static_cast<char *>(sw), sb, static_workspace_bytes(), 0};
    Plan p;
    plan_build(d.data(), (int)d.size(), &p);
    g_buf.nt = (int)p.t.size();
    CHECK(skew_step(a, &hp, nullptr) == SKEW_ESTALE, "the older static context is stale");
    CHECK(skew_step(b, &hp, nullptr) == SKEW_OK, "the newer static context steps");
    skew_destroy(a);
    skew_destroy(b);
    skew_ctx *c = nullptr;
    CHECK(skew_state_init_static(&c, big.data(), (int)big.size(), nullptr, 0, nullptr) == SKEW_ETOOBIG,
          "a table beyond the static workspace");
    CHECK(c == nullptr, "no context on failure");
  }
  // validation: bad descriptors are refused before anything is touched
  {
    std::vector<skew_tensor_desc> bad = {mk(3, 2, 4, 4, 4, 0)};
    size_t sb, wb;
    CHECK(skew_state_bytes(bad.data(), 1, &sb, &wb) == SKEW_EINVAL, "tier 3");
    bad = {mk(0, 2, 4, 8, 4, 0)};
    CHECK(skew_state_bytes(bad.data(), 1, &sb, &wb) == SKEW_EINVAL, "ld < cols");
    bad = {mk(0, 4, 4, 8, 8, 0)};
    CHECK(skew_state_bytes(bad.data(), 1, &sb, &wb) == SKEW_EINVAL, "ndim 4");
    bad = {mk(1, 2, 4, 8, 8, 0, 0, 4)};
    CHECK(skew_state_bytes(bad.data(), 1, &sb, &wb) == SKEW_EINVAL, "fp32 factored");
    bad = {mk(1, 2, int64_t(1) << 40, int64_t(1) << 40, int64_t(1) << 40, 0)};
    CHECK(skew_state_bytes(bad.data(), 1, &sb, &wb) == SKEW_EINVAL, "element count overflow");
  }
  if (g_fail) {
    std::printf("%d checks failed\n", g_fail);
    return 1;
  }
  std::printf("all %ld planner and host checks passed\n", g_checks);
  return 0;
}

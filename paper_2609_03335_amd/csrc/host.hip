// Host side of the C ABI declared in include/wf_plan.h: contexts, window
// validation and derivation (levels, Eq. 3 fusibility, unique successors),
// the device copy of the window, launch geometry, and the two entry points
// that enqueue work.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "kernels.h"
#include "wf_plan.h"

namespace {

thread_local std::string g_thread_err;  // errors without a context

struct HostWindow {
  int32_t N = 0, W = 0, M = 0, D = 0, n_levels = 0, wmax = 0;
  int64_t min_arrival = 0;
  std::vector<int32_t> act_model, act_wf, chain_next, pred_off, pred_idx, lat, mem, cap, wmib,
      load, level_off;
  std::vector<uint8_t> fusible;
  std::vector<int64_t> arrival, free0;
  std::vector<uint64_t> init_res;
  std::vector<uint8_t> wf_class;  // [W] priority class of the ranking key
  int32_t victim_order = WF_VICTIM_REMAINING_LRU;
  std::vector<int32_t> batch;  // [D] batch limit
  std::vector<int32_t> rcap;   // [M] replica cap, empty = none
  float w_mk = 1.f, w_p95 = 0.f;
  int64_t pf_slack = 0;        // dispatch slack of the prefetch rule
};

wf_status fail(std::string* err, wf_status st, const char* fmt, ...) __attribute__((format(printf, 3, 4)));
wf_status fail(std::string* err, wf_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (err) *err = buf;
  return st;
}

// Validate a window description and, when `out` is given, derive the
// structures the kernels use.  No side effects on failure.
wf_status validate(const wf_window_desc* w, std::string* err, HostWindow* out) {
  if (!w) return fail(err, WF_EINVAL, "window descriptor is NULL");
  const int64_t N = w->n_act, W = w->n_wf, M = w->n_models, D = w->n_dev;
  if (N < 0 || N > WF_MAX_ACT) return fail(err, WF_EINVAL, "n_act=%lld outside [0, %d]", (long long)N, WF_MAX_ACT);
  if (M < 1 || M > WF_MAX_MODELS) return fail(err, WF_EINVAL, "n_models=%lld outside [1, %d]", (long long)M, WF_MAX_MODELS);
  if (D < 1 || D > WF_MAX_DEV) return fail(err, WF_EINVAL, "n_dev=%lld outside [1, %d]", (long long)D, WF_MAX_DEV);
  if (W < 0 || W > N) return fail(err, WF_EINVAL, "n_wf=%lld outside [0, n_act=%lld]", (long long)W, (long long)N);
  if (N > 0 && W < 1) return fail(err, WF_EINVAL, "n_wf must be >= 1 when n_act > 0");
  if (!w->pred_off) return fail(err, WF_EINVAL, "pred_off is NULL");
  if (N > 0 && (!w->act_wf || !w->act_model || !w->lat_us || !w->mem_mib))
    return fail(err, WF_EINVAL, "an activation array (act_wf, act_model, lat_us, mem_mib) is NULL");
  if (W > 0 && !w->wf_arrival_us) return fail(err, WF_EINVAL, "wf_arrival_us is NULL");
  if (!w->dev_cap_mib || !w->model_mib || !w->load_us || !w->init_resident)
    return fail(err, WF_EINVAL, "a pool array (dev_cap_mib, model_mib, load_us, init_resident) is NULL");
  if (!(std::isfinite(w->w_makespan) && std::isfinite(w->w_p95)) || w->w_makespan < 0.f || w->w_p95 < 0.f)
    return fail(err, WF_EINVAL, "objective weights must be finite and >= 0");
  if (w->pred_off[0] != 0) return fail(err, WF_EINVAL, "pred_off[0] must be 0");
  for (int64_t i = 0; i < N; ++i)
    if (w->pred_off[i + 1] < w->pred_off[i])
      return fail(err, WF_EINVAL, "pred_off decreases at row %lld", (long long)i);
  const int64_t nnz = w->pred_off[N];
  if (nnz > 0 && !w->pred_idx) return fail(err, WF_EINVAL, "pred_idx is NULL");

  std::vector<int32_t> level((size_t)N);
  for (int64_t i = 0; i < N; ++i) {
    int32_t lv = 0;
    for (int64_t k = w->pred_off[i]; k < w->pred_off[i + 1]; ++k) {
      const int32_t p = w->pred_idx[k];
      if (p < 0 || p >= i)
        return fail(err, WF_EINVAL, "activation %lld: predecessor %d is not an earlier activation", (long long)i, p);
      if (k > w->pred_off[i] && p <= w->pred_idx[k - 1])
        return fail(err, WF_EINVAL, "activation %lld: predecessors not strictly increasing", (long long)i);
      lv = std::max(lv, level[p] + 1);
    }
    level[i] = lv;
    if (i > 0 && lv < level[i - 1])
      return fail(err, WF_EINVAL, "activation %lld (level %d) follows level %d: numbering must be level-sorted",
                  (long long)i, lv, level[i - 1]);
    if (w->act_wf[i] < 0 || w->act_wf[i] >= W)
      return fail(err, WF_EINVAL, "activation %lld: workflow %d outside [0, %lld)", (long long)i, w->act_wf[i], (long long)W);
    if (w->act_model[i] < 0 || w->act_model[i] >= M)
      return fail(err, WF_EINVAL, "activation %lld: model %d outside [0, %lld)", (long long)i, w->act_model[i], (long long)M);
    for (int64_t d = 0; d < D; ++d) {
      const int32_t l = w->lat_us[i * D + d], m = w->mem_mib[i * D + d];
      if (l < -1) return fail(err, WF_EINVAL, "lat_us[%lld][%lld] = %d (use -1 for ineligible)", (long long)i, (long long)d, l);
      if (m < 0 || m > WF_MAX_MEM_MIB)
        return fail(err, WF_EINVAL, "mem_mib[%lld][%lld] = %d outside [0, %d]", (long long)i, (long long)d, m, WF_MAX_MEM_MIB);
    }
  }
  std::vector<uint8_t> has_act((size_t)W, 0);
  for (int64_t i = 0; i < N; ++i) has_act[w->act_wf[i]] = 1;
  for (int64_t f = 0; f < W; ++f) {
    if (!has_act[f]) return fail(err, WF_EINVAL, "workflow %lld has no activation", (long long)f);
    if (w->wf_arrival_us[f] < 0 || w->wf_arrival_us[f] > WF_MAX_TIME_US)
      return fail(err, WF_EINVAL, "wf_arrival_us[%lld] outside [0, 2^52]", (long long)f);
  }
  for (int64_t m = 0; m < M; ++m) {
    if (w->model_mib[m] < 0 || w->model_mib[m] > WF_MAX_MEM_MIB)
      return fail(err, WF_EINVAL, "model_mib[%lld] = %d outside [0, %d]", (long long)m, w->model_mib[m], WF_MAX_MEM_MIB);
    for (int64_t d = 0; d < D; ++d)
      if (w->load_us[m * D + d] < 0)
        return fail(err, WF_EINVAL, "load_us[%lld][%lld] is negative", (long long)m, (long long)d);
  }
  for (int64_t d = 0; d < D; ++d) {
    if (w->dev_cap_mib[d] < 0 || w->dev_cap_mib[d] > WF_MAX_CAP_MIB)
      return fail(err, WF_EINVAL, "dev_cap_mib[%lld] = %d outside [0, %d]", (long long)d, w->dev_cap_mib[d], WF_MAX_CAP_MIB);
    if (w->dev_free0_us && (w->dev_free0_us[d] < 0 || w->dev_free0_us[d] > WF_MAX_TIME_US))
      return fail(err, WF_EINVAL, "dev_free0_us[%lld] outside [0, 2^52]", (long long)d);
    const uint64_t r = w->init_resident[d];
    if (M < 64 && (r >> M) != 0)
      return fail(err, WF_EINVAL, "init_resident[%lld] names a model >= n_models", (long long)d);
    int64_t used = 0;
    for (int64_t m = 0; m < M; ++m)
      if ((r >> m) & 1ull) used += w->model_mib[m];
    if (used > w->dev_cap_mib[d])
      return fail(err, WF_EINVAL, "initial residency of device %lld (%lld MiB) exceeds its capacity %d MiB",
                  (long long)d, (long long)used, w->dev_cap_mib[d]);
  }
  if (w->wf_class)
    for (int64_t f = 0; f < W; ++f)
      if (w->wf_class[f] >= WF_MAX_CLASSES)
        return fail(err, WF_EINVAL, "wf_class[%lld] = %d outside [0, %d)", (long long)f,
                    (int)w->wf_class[f], WF_MAX_CLASSES);
  if (w->victim_order != WF_VICTIM_REMAINING_LRU && w->victim_order != WF_VICTIM_PAPER)
    return fail(err, WF_EINVAL, "victim_order = %d is not a WF_VICTIM_* value", (int)w->victim_order);
  if (w->dev_batch)
    for (int64_t d = 0; d < D; ++d)
      if (w->dev_batch[d] < 1 || w->dev_batch[d] > WF_MAX_BATCH)
        return fail(err, WF_EINVAL, "dev_batch[%lld] = %d outside [1, %d]", (long long)d,
                    (int)w->dev_batch[d], WF_MAX_BATCH);
  if (w->model_replica_cap)
    for (int64_t m = 0; m < M; ++m) {
      if (w->model_replica_cap[m] < 1)
        return fail(err, WF_EINVAL, "model_replica_cap[%lld] = %d is below 1", (long long)m,
                    (int)w->model_replica_cap[m]);
      int64_t copies = 0;
      for (int64_t d = 0; d < D; ++d) copies += (int64_t)((w->init_resident[d] >> m) & 1ull);
      if (copies > w->model_replica_cap[m])
        return fail(err, WF_EINVAL, "initial residency holds %lld copies of model %lld, above its replica cap %d",
                    (long long)copies, (long long)m, (int)w->model_replica_cap[m]);
    }
  if (w->prefetch_slack_us < 0 || w->prefetch_slack_us > WF_MAX_TIME_US)
    return fail(err, WF_EINVAL, "prefetch_slack_us = %lld outside [0, 2^52]",
                (long long)w->prefetch_slack_us);
  if (!out) return WF_OK;

  HostWindow& h = *out;
  h.pf_slack = w->prefetch_slack_us;
  h.victim_order = w->victim_order;
  h.batch.assign((size_t)D, 1);
  if (w->dev_batch) h.batch.assign(w->dev_batch, w->dev_batch + D);
  if (w->model_replica_cap) h.rcap.assign(w->model_replica_cap, w->model_replica_cap + M);
  h.wf_class.assign((size_t)W, 0);
  if (w->wf_class) h.wf_class.assign(w->wf_class, w->wf_class + W);
  h.N = (int32_t)N;
  h.W = (int32_t)W;
  h.M = (int32_t)M;
  h.D = (int32_t)D;
  h.act_model.assign(w->act_model, w->act_model + N);
  h.act_wf.assign(w->act_wf, w->act_wf + N);
  h.pred_off.assign(w->pred_off, w->pred_off + N + 1);
  h.pred_idx.assign(w->pred_idx, w->pred_idx + nnz);
  if (h.pred_idx.empty()) h.pred_idx.push_back(0);
  h.lat.assign(w->lat_us, w->lat_us + N * D);
  h.mem.assign(w->mem_mib, w->mem_mib + N * D);
  h.arrival.assign(w->wf_arrival_us, w->wf_arrival_us + W);
  h.cap.assign(w->dev_cap_mib, w->dev_cap_mib + D);
  h.wmib.assign(w->model_mib, w->model_mib + M);
  h.load.assign(w->load_us, w->load_us + M * D);
  h.init_res.assign(w->init_resident, w->init_resident + D);
  h.free0.assign((size_t)D, 0);
  if (w->dev_free0_us) h.free0.assign(w->dev_free0_us, w->dev_free0_us + D);
  h.w_mk = w->w_makespan;
  h.w_p95 = w->w_p95;
  h.min_arrival = W > 0 ? *std::min_element(h.arrival.begin(), h.arrival.end()) : 0;
  // topological levels -> contiguous index ranges
  h.level_off.clear();
  h.level_off.push_back(0);
  for (int64_t i = 1; i <= N; ++i)
    if (i == N || level[i] != level[i - 1]) h.level_off.push_back((int32_t)i);
  if (N == 0) h.level_off.assign(1, 0);
  h.n_levels = (int32_t)h.level_off.size() - 1;
  h.wmax = 0;
  for (int32_t l = 0; l < h.n_levels; ++l) h.wmax = std::max(h.wmax, h.level_off[l + 1] - h.level_off[l]);
  // Eq. 3: edge (u, v) fuses iff pred(v) = {u}, succ(u) = {v}, same model
  std::vector<int32_t> n_succ((size_t)N, 0), succ((size_t)N, -1);
  for (int64_t v = 0; v < N; ++v)
    for (int64_t k = h.pred_off[v]; k < h.pred_off[v + 1]; ++k) {
      ++n_succ[h.pred_idx[k]];
      succ[h.pred_idx[k]] = (int32_t)v;
    }
  h.fusible.assign((size_t)std::max<int64_t>(N, 1), 0);
  h.chain_next.assign((size_t)std::max<int64_t>(N, 1), -1);
  for (int64_t v = 0; v < N; ++v) {
    if (h.pred_off[v + 1] - h.pred_off[v] != 1) continue;
    const int32_t u = h.pred_idx[h.pred_off[v]];
    if (n_succ[u] == 1 && h.act_model[u] == h.act_model[v]) {
      h.fusible[v] = 1;
      h.chain_next[u] = (int32_t)v;
    }
  }
  if (N == 0) {  // keep every device array non-empty
    h.act_model.assign(1, 0);
    h.act_wf.assign(1, 0);
    h.lat.assign((size_t)D, 0);
    h.mem.assign((size_t)D, 0);
  }
  if (h.arrival.empty()) h.arrival.push_back(0);
  return WF_OK;
}

struct DeviceWindow {
  void* tab = nullptr;          // table image in HBM
  void* rules = nullptr;        // rule tables of the candidate generator
  const unsigned long long* rule_pf = nullptr;
  const int8_t* rule_best = nullptr;
  void* tab64 = nullptr;        // fp64-time table image of the rescoring pass
  void* scratch = nullptr;      // per-wave regions for windows too big for LDS
  void* tab_lean = nullptr;     // the lean kernel's table image
  wfp::ScoreParams sp{};        // scoring plans read from HBM
  wfp::ScoreParams sp_search{}; // scoring candidates generated around an incumbent
  // the same with more than kPatchMaxMut mutations when sp_search keeps
  // candidates as changed sites (the ring layout)
  wfp::ScoreParams sp_search_wide{};
  // uint32 times without a proof that none reaches 2^32: plans whose times
  // saturate are rescored with fp64 times
  bool checked = false;
  wfp::ScoreParams sp64{}, sp64_search{};
  // the lean kernel for scores of plans read from HBM, when the window
  // qualifies (lean.ok)
  wfp::LeanParams lean{};
};

}  // namespace

struct wf_plan_ctx {
  int device = 0;
  int n_cu = 0;
  int lds_per_block = 0;
  int lds_per_cu = 0;
  std::string err;
  bool has_window = false;
  HostWindow host;
  DeviceWindow dw;
  void* key_work = nullptr;  // partial results of the argmins
};

namespace {

wf_status hip_fail(wf_plan_ctx* ctx, hipError_t e, const char* what) {
  ctx->err = std::string(what) + ": " + hipGetErrorString(e);
  return WF_EHIP;
}

void free_device_window(DeviceWindow& dw) {
  if (dw.tab) (void)hipFree(dw.tab);
  if (dw.tab64) (void)hipFree(dw.tab64);
  if (dw.scratch) (void)hipFree(dw.scratch);
  if (dw.tab_lean) (void)hipFree(dw.tab_lean);
  if (dw.rules) (void)hipFree(dw.rules);
  dw = DeviceWindow{};
}

// The rule tables of the candidate generator (Algorithm 1, Sec. 3.5), as a
// byte image: [N][2] 64-bit masks of the devices on which PlanPrefetch sets
// activation i's prefetch bit, then [N] best feasible bindings (-1: no
// eligible device).  A unit is ready when it has no predecessor and its
// workflow has arrived by time 0.
std::vector<unsigned char> rule_image(const HostWindow& h, size_t* best_at) {
  const int32_t N = h.N, D = h.D, M = h.M;
  const size_t n = (size_t)std::max(N, 1);
  std::vector<unsigned char> img(n * 16 + n, 0);
  *best_at = n * 16;
  uint64_t* pf = reinterpret_cast<uint64_t*>(img.data());
  int8_t* best = reinterpret_cast<int8_t*>(img.data() + n * 16);
  std::vector<uint8_t> ready((size_t)N);
  std::vector<int64_t> work((size_t)M * D, 0);  // ready work a load of (m, d) unlocks
  std::vector<int64_t> rel((size_t)N), fastest((size_t)N);
  for (int32_t i = 0; i < N; ++i) {
    const int32_t* li = &h.lat[(size_t)i * D];
    ready[i] = h.pred_off[i] == h.pred_off[i + 1] && h.arrival[h.act_wf[i]] <= 0;
    int64_t f = -1;
    for (int32_t d = 0; d < D; ++d) {
      if (li[d] < 0) continue;
      if (f < 0 || li[d] < f) f = li[d];
      if (ready[i]) work[(size_t)h.act_model[i] * D + d] += li[d];
    }
    fastest[i] = f < 0 ? 0 : f;
    // activations are in topological order: predecessors are final here
    int64_t r = h.arrival[h.act_wf[i]];
    for (int32_t k = h.pred_off[i]; k < h.pred_off[i + 1]; ++k)
      r = std::max(r, rel[h.pred_idx[k]] + fastest[h.pred_idx[k]]);
    rel[i] = r;
  }
  for (int32_t i = 0; i < N; ++i) {
    const int32_t m = h.act_model[i];
    const int32_t* li = &h.lat[(size_t)i * D];
    const int32_t* lm = &h.load[(size_t)m * D];
    const int64_t* wm = &work[(size_t)m * D];
    int b = -1;
    bool b_res = false;
    for (int32_t d = 0; d < D; ++d) {
      if (li[d] < 0) continue;
      const bool res = (h.init_res[d] >> m) & 1ull;
      bool take;
      if (b < 0 || res != b_res) {
        take = b < 0 || res;  // a resident replica beats any load
      } else if (res) {
        take = li[d] < li[b];
      } else {
        // value = work / load, a free load above every ratio
        int v;
        if (lm[d] == 0 || lm[b] == 0) {
          v = (lm[d] == 0) - (lm[b] == 0);
        } else {
          const unsigned __int128 x = (unsigned __int128)(uint64_t)wm[d] * (uint32_t)lm[b];
          const unsigned __int128 y = (unsigned __int128)(uint64_t)wm[b] * (uint32_t)lm[d];
          v = (x > y) - (x < y);
        }
        take = v > 0 || (v == 0 && li[d] < li[b]);
      }
      if (take) {
        b = d;
        b_res = res;
      }
    }
    best[i] = (int8_t)b;
    if (ready[i]) continue;
    for (int32_t d = 0; d < D; ++d)
      if (rel[i] <= (int64_t)lm[d] + h.pf_slack) pf[(size_t)i * 2 + d / 64] |= 1ull << (d % 64);
  }
  return img;
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Append a table to the image; returns its byte offset (16-byte aligned).
struct Image {
  std::vector<unsigned char> bytes;
  int put(const void* p, size_t n) {
    const size_t off = align_up(bytes.size(), 16);
    bytes.resize(off + std::max<size_t>(n, 4), 0);
    if (n) std::memcpy(bytes.data() + off, p, n);
    return (int)off;
  }
};

// Per-wave region for G plans; returns the wave's byte size.  In LDS
// (global = false) it is one block.  With regions in HBM (global = true) the
// small per-(device, model) arrays come first, [0, o.split), and stay in LDS;
// the per-activation arrays follow in HBM.
int wave_layout(const HostWindow& h, int G, int tsz, int nwa, int qmode, bool search,
                wfp::WaveOffsets& o, bool global, int ring_fin = 0) {
  const bool nibble = qmode > 0, paper = qmode == -1 || qmode == -3;
  size_t off = 0;
  auto take = [&](size_t n) {
    const size_t at = off;
    off = align_up(off + std::max<size_t>(n, 1), 16);
    return (int)at;
  };
  const int NB = (h.N + 3) / 4;
  // (ring_fin > 0, regions in HBM: the finishes are a ring of ring_fin
  // positions per plan, in the LDS part with the per-workflow finishes)
  ring_fin = global ? ring_fin : 0;
  const size_t fin_bytes = (size_t)G * (ring_fin > 0 ? ring_fin : h.N) * tsz,
               last_bytes = (size_t)G * h.D * h.M * 4;
  const size_t dm2 = (size_t)G * h.D * h.M * 2;
  // generated candidates keep their device and priority rows in fin's
  // storage (after last[] when that shares it) while the order is built
  const size_t rows_at = nibble ? align_up(last_bytes, 16) : 0;
  const size_t rows_bytes = search ? align_up((size_t)G * h.N, 16) + (size_t)G * h.N * 2 : 0;
  o = wfp::WaveOffsets{};
  if (global) {
    // LDS part: the arrays read per reclamation candidate and the totals
    o.acc = take((size_t)G * sizeof(wfp::PlanAcc));
    if (!nibble) {
      if (!paper) o.last = take(last_bytes);
      o.stamp = take(dm2);
    }
    if (paper) {
      o.nxu = take(dm2);
      o.snap = take((size_t)G * h.D * 8);
    }
    o.hstate = take(h.D > 64 ? 2 * 64 * sizeof(wfp::HState) : 0);
    o.hold = take(h.rcap.empty() ? 0 : (size_t)G * h.D * 8);
    if (ring_fin > 0) {
      o.fin = take(std::max(fin_bytes, rows_bytes));
      o.wfm = take((size_t)G * std::max(1, h.W) * tsz);
    }
    o.split = (int)off;
  }
  o.flags = take((size_t)G * NB);
  o.rec = take((size_t)G * h.N * 4);
  o.mask = take((size_t)G * h.D * nwa * 8);
  if (!global) o.acc = take((size_t)G * sizeof(wfp::PlanAcc));
  if (nibble) {
    o.fin = take(std::max(std::max(fin_bytes, last_bytes), rows_at + rows_bytes));
    o.last = o.fin;
  } else if (paper) {
    // the paper order keeps no last[] (it is never written)
    if (ring_fin == 0) o.fin = take(std::max(fin_bytes, rows_bytes));
    o.last = o.fin;
    if (!global) o.stamp = take(dm2);
  } else {
    if (ring_fin == 0) o.fin = take(std::max(fin_bytes, rows_bytes));
    if (!global) {
      o.last = take(last_bytes);
      o.stamp = take(dm2);
    }
  }
  o.rows = o.fin + (int)rows_at;
  o.rows_prio = o.rows + (int)align_up((size_t)G * h.N, 16);
  if (ring_fin == 0) o.wfm = take((size_t)G * std::max(1, h.W) * tsz);
  // unused arrays point at the start of their part
  o.nx = global ? o.split : 0;
  if (paper) {
    o.nx = take((size_t)G * h.N * 2);
    if (!global) {
      o.nxu = take(dm2);
      o.snap = take((size_t)G * h.D * 8);
    }
  }
  if (!global) {
    o.hstate = take(h.D > 64 ? 2 * 64 * sizeof(wfp::HState) : 0);
    o.hold = take(h.rcap.empty() ? 0 : (size_t)G * h.D * 8);
  }
  o.bytes = (int)off;
  return o.bytes;
}

// Per-wave LDS region of the ring layout for G plans (kernel PLACE 2): the
// per-plan arrays of the current level and of the ring's levels only.
int ring_layout(const HostWindow& h, const wfp::ScoreParams& sp, int G, int tsz, int nwl,
                bool search, wfp::WaveOffsets& o) {
  size_t off = 0;
  auto take = [&](size_t n) {
    const size_t at = off;
    off = align_up(off + std::max<size_t>(n, 1), 16);
    return (int)at;
  };
  const size_t dm = (size_t)G * h.D * h.M;
  o = wfp::WaveOffsets{};
  o.flags = take((size_t)G * ((h.N + 3) / 4));
  o.rec = take((size_t)G * sp.ring_w * 4);
  o.mask = take((size_t)G * h.D * nwl * 8);
  o.acc = take((size_t)G * sizeof(wfp::PlanAcc));
  o.last = take(dm * 2);
  o.stamp = take(dm * 2);
  o.fin = take((size_t)G * sp.ring_size * tsz);
  o.wfm = take((size_t)G * std::max(1, h.W) * tsz);
  o.hstate = take(h.D > 64 ? 2 * 64 * sizeof(wfp::HState) : 0);
  o.hold = take(h.rcap.empty() ? 0 : (size_t)G * h.D * 8);
  // generated candidates: each one's changed sites (at most kPatchMaxMut
  // mutations)
  o.rows = take(search ? (size_t)G * wfp::kPatchWords * 4 : 0);
  o.bytes = (int)off;
  return o.bytes;
}

// How a window's times are carried: uint32 when no time of any plan can reach
// 2^32 (proven by the static bound below), uint32 with an fp64 rescoring of
// the plans that saturate when the bound is within kCheckedSpan of 2^32 (few
// plans get there), else fp64.
enum TimeMode { kTimeU32 = 0, kTimeF64 = 1, kTimeChecked = 2 };
constexpr int64_t kCheckedSpan = 8;

// Build the table image and choose LDS placement, plans per wave and waves per
// workgroup for this window, with uint32 (time64 = false) or fp64 times;
// *mode reports which time arithmetic the window needs.
wf_status plan_window(wf_plan_ctx* ctx, const HostWindow& h, bool time64_req, Image& img,
                      wfp::ScoreParams& sp, TimeMode* mode) {
  const int N = h.N, D = h.D, M = h.M, W = h.W;
  // time origin: earliest arrival or device free time
  int64_t origin = INT64_MAX;
  for (int32_t f = 0; f < W; ++f) origin = std::min(origin, h.arrival[f]);
  for (int32_t d = 0; d < D; ++d) origin = std::min(origin, h.free0[d]);
  if (origin == INT64_MAX) origin = 0;
  // largest relative time any plan can reach: latest arrival/free time plus
  // every activation's longest run and its model's longest load, in sequence
  int64_t t0 = 0;
  for (int32_t f = 0; f < W; ++f) t0 = std::max(t0, h.arrival[f] - origin);
  for (int32_t d = 0; d < D; ++d) t0 = std::max(t0, h.free0[d] - origin);
  int64_t bound = t0;
  std::vector<int64_t> maxlat((size_t)std::max(N, 1), 0);
  for (int32_t i = 0; i < N; ++i) {
    int64_t ml = 0, mload = 0;
    for (int32_t d = 0; d < D; ++d) {
      ml = std::max<int64_t>(ml, h.lat[(size_t)i * D + d]);
      mload = std::max<int64_t>(mload, h.load[(size_t)h.act_model[i] * D + d]);
    }
    maxlat[i] = ml;
    bound += ml + mload;
  }
  // a fused chain's summed run time is carried as uint32
  int64_t chain_max = 0;
  std::vector<int64_t> csum((size_t)std::max(N, 1), 0);
  for (int32_t i = N - 1; i >= 0; --i) {
    csum[i] = maxlat[i] + (h.chain_next[i] >= 0 ? csum[h.chain_next[i]] : 0);
    chain_max = std::max(chain_max, csum[i]);
  }
  if (chain_max >= (int64_t(1) << 32))
    return fail(&ctx->err, WF_EUNSUPPORTED, "a fusible chain may run for 2^32 us or more");
  const int64_t two32 = int64_t(1) << 32;
  *mode = bound < two32 ? kTimeU32
          : (t0 < two32 / 2 && bound < kCheckedSpan * two32) ? kTimeChecked : kTimeF64;
  const bool time64 = *mode == kTimeF64 || time64_req;
  const int tsz = time64 ? 8 : 4;

  // ---- table image ----
  std::vector<uint32_t> act((size_t)std::max(N, 1), 0);
  std::vector<uint16_t> cnext((size_t)std::max(N, 1), 0xffff);
  for (int32_t i = 0; i < N; ++i) {
    // ready work of the ranking key: no predecessor, arrived by time 0
    const bool ready = h.pred_off[i] == h.pred_off[i + 1] && h.arrival[h.act_wf[i]] <= 0;
    act[i] = (uint32_t)h.act_model[i] | ((uint32_t)h.fusible[i] << 6) | ((uint32_t)ready << 7) |
             ((uint32_t)h.wf_class[h.act_wf[i]] << 8) | ((uint32_t)h.act_wf[i] << 16);
    cnext[i] = h.chain_next[i] >= 0 ? (uint16_t)h.chain_next[i] : (uint16_t)0xffff;
  }
  const int32_t E = N > 0 ? h.pred_off[N] : 0;
  std::vector<uint32_t> edge((size_t)std::max(E, 1), 0);
  for (int32_t v = 0; v < N; ++v)
    for (int32_t k = h.pred_off[v]; k < h.pred_off[v + 1]; ++k)
      edge[k] = (uint32_t)h.pred_idx[k] | ((uint32_t)v << 16);
  std::vector<int32_t> eoff((size_t)h.n_levels + 1);
  for (int32_t l = 0; l <= h.n_levels; ++l) eoff[l] = N > 0 ? h.pred_off[h.level_off[l]] : 0;
  std::vector<unsigned char> arr((size_t)std::max(W, 1) * tsz, 0), fr((size_t)D * tsz, 0);
  for (int32_t f = 0; f < W; ++f) {
    const int64_t r = h.arrival[f] - origin;
    if (time64) { const double x = (double)r; std::memcpy(&arr[(size_t)f * 8], &x, 8); }
    else { const uint32_t x = (uint32_t)r; std::memcpy(&arr[(size_t)f * 4], &x, 4); }
  }
  for (int32_t d = 0; d < D; ++d) {
    const int64_t r = h.free0[d] - origin;
    if (time64) { const double x = (double)r; std::memcpy(&fr[(size_t)d * 8], &x, 8); }
    else { const uint32_t x = (uint32_t)r; std::memcpy(&fr[(size_t)d * 4], &x, 4); }
  }
  std::vector<uint32_t> alv((size_t)std::max(N, 1), 0);
  for (int32_t l = 0; l < h.n_levels; ++l)
    for (int32_t i = h.level_off[l]; i < h.level_off[l + 1]; ++i)
      alv[i] = (uint32_t)h.level_off[l] | ((uint32_t)(h.level_off[l + 1] - h.level_off[l]) << 16);
  // the walk's per-unit record: run time, memory and workflow arrival in one
  // 16-byte load
  std::vector<uint32_t> ud((size_t)std::max(N * D, 1) * 4, 0);
  for (int32_t i = 0; i < N; ++i)
    for (int32_t d = 0; d < D; ++d) {
      uint32_t* r = &ud[((size_t)i * D + d) * 4];
      r[0] = (uint32_t)h.lat[(size_t)i * D + d];
      r[1] = (uint32_t)h.mem[(size_t)i * D + d];
      std::memcpy(&r[2], &arr[(size_t)h.act_wf[i] * tsz], tsz);
      if (!time64) r[3] = act[i];  // the ranking-key mode reads it from here
    }
  wfp::TabOffsets& t = sp.t;
  t.act = img.put(act.data(), act.size() * 4);
  t.alv = img.put(alv.data(), alv.size() * 4);
  t.cnext = img.put(cnext.data(), cnext.size() * 2);
  t.edge = img.put(edge.data(), edge.size() * 4);
  t.eoff = img.put(eoff.data(), eoff.size() * 4);
  t.loff = img.put(h.level_off.data(), h.level_off.size() * 4);
  t.ud = img.put(ud.data(), ud.size() * 4);
  t.wmib = img.put(h.wmib.data(), h.wmib.size() * 4);
  std::vector<int32_t> lw((size_t)M * D * 2);
  for (int32_t m = 0; m < M; ++m)
    for (int32_t d = 0; d < D; ++d) {
      lw[((size_t)m * D + d) * 2] = h.load[(size_t)m * D + d];
      lw[((size_t)m * D + d) * 2 + 1] = h.wmib[m];
    }
  t.lw = img.put(lw.data(), lw.size() * 4);
  std::vector<uint64_t> elig((size_t)std::max(N, 1) * 2, 0);
  for (int32_t i = 0; i < N; ++i)
    for (int32_t d = 0; d < D; ++d)
      if (h.lat[(size_t)i * D + d] >= 0) elig[(size_t)i * 2 + d / 64] |= uint64_t(1) << (d % 64);
  t.elig = img.put(elig.data(), elig.size() * 8);
  t.batch = img.put(h.batch.data(), h.batch.size() * 4);
  t.rcap = img.put(h.rcap.data(), h.rcap.size() * 4);
  t.cap = img.put(h.cap.data(), h.cap.size() * 4);
  t.arr = img.put(arr.data(), arr.size());
  t.res0 = img.put(h.init_res.data(), h.init_res.size() * 8);
  t.free0 = img.put(fr.data(), fr.size());
  // activations with no successor in their own workflow: a workflow's
  // latest finish is reached at one of them
  std::vector<uint8_t> has_wf_succ((size_t)std::max(N, 1), 0);
  for (int32_t v = 0; v < N; ++v)
    for (int32_t k = h.pred_off[v]; k < h.pred_off[v + 1]; ++k)
      if (h.act_wf[h.pred_idx[k]] == h.act_wf[v]) has_wf_succ[h.pred_idx[k]] = 1;
  std::vector<uint32_t> sink;
  for (int32_t i = 0; i < N; ++i)
    if (!has_wf_succ[i]) sink.push_back((uint32_t)i | ((uint32_t)h.act_wf[i] << 16));
  const int32_t S = (int32_t)sink.size();
  if (sink.empty()) sink.push_back(0);
  t.sink = img.put(sink.data(), sink.size() * 4);
  // ring of recent levels (the scan reclamation modes, and the paper's
  // order, whose finishes alone may take it): a finish must stay from the
  // level where it is written -- a fused chain's members with the chain
  // head, up to ring_a levels early -- to the last level an edge reads it,
  // ring_b levels later
  const bool batched_w = std::any_of(h.batch.begin(), h.batch.end(), [](int32_t b) { return b > 1; });
  const bool ring_tables = h.victim_order == WF_VICTIM_PAPER || batched_w || M > 16 || !h.rcap.empty();
  sp.ring_ok = 0;
  if (ring_tables && N > 0) {
    std::vector<int32_t> lvl((size_t)N), wmin((size_t)N);
    for (int32_t l = 0; l < h.n_levels; ++l)
      for (int32_t i = h.level_off[l]; i < h.level_off[l + 1]; ++i) lvl[i] = l;
    int32_t ra = 0, rb = 0;
    for (int32_t v = 0; v < N; ++v) {
      wmin[v] = h.fusible[v] ? wmin[h.pred_idx[h.pred_off[v]]] : lvl[v];
      ra = std::max(ra, lvl[v] - wmin[v]);
      for (int32_t k = h.pred_off[v]; k < h.pred_off[v + 1]; ++k)
        rb = std::max(rb, lvl[v] - lvl[h.pred_idx[k]]);
    }
    // positions are activation indices mod the ring size: the most
    // activations held by levels lv - ring_b .. lv + ring_a for any lv
    int64_t size = 1;
    for (int32_t l = 0; l < h.n_levels; ++l) {
      const int32_t a0 = std::max(0, l - rb), a1 = std::min(h.n_levels, l + ra + 1);
      size = std::max<int64_t>(size, h.level_off[a1] - h.level_off[a0]);
    }
    if (size <= 65535) {
      sp.ring_ok = 1;
      sp.ring_size = (int)size;
      sp.ring_w = h.wmax;
      sp.ring_a = ra;
      sp.ring_b = rb;
      std::vector<uint16_t> rpos((size_t)N), rsnk((size_t)N);
      for (int32_t i = 0; i < N; ++i) {
        rpos[i] = (uint16_t)(i % size);
        rsnk[i] = has_wf_succ[i] ? (uint16_t)0xffff : (uint16_t)h.act_wf[i];
      }
      std::vector<uint32_t> redge((size_t)std::max(E, 1), 0);
      for (int32_t v = 0; v < N; ++v)
        for (int32_t k = h.pred_off[v]; k < h.pred_off[v + 1]; ++k)
          redge[k] = (uint32_t)rpos[h.pred_idx[k]] | ((uint32_t)rpos[v] << 16);
      t.rpos = img.put(rpos.data(), rpos.size() * 2);
      t.rsnk = img.put(rsnk.data(), rsnk.size() * 2);
      t.redge = img.put(redge.data(), redge.size() * 4);
    }
  }
  img.bytes.resize(align_up(img.bytes.size(), 16), 0);
  t.bytes = (int)img.bytes.size();

  sp.N = N;
  sp.W = W;
  sp.M = M;
  sp.D = D;
  sp.NB = (N + 3) / 4;
  sp.S = S;
  sp.n_levels = h.n_levels;
  sp.nwa = std::max(1, (N + 63) / 64);
  sp.origin = origin;
  sp.min_arrival = h.min_arrival;
  sp.w_mk = h.w_mk;
  sp.w_p95 = h.w_p95;
  sp.time64 = time64 ? 1 : 0;
  // with M <= 16 the resident set is a queue of 4-bit model ids; it fits in
  // 32 bits when no device can ever hold more than 8 models: a device holds
  // its initial set, or models whose weights sum to at most its capacity, or
  // (after a load that overflows) the one model just loaded
  // (with batch limits too: a load reclaims until the models, plus the
  // running units' memory, fit, or until nothing is left to reclaim)
  sp.nibble = 0;
  sp.queue = 0;
  sp.rcap = h.rcap.empty() ? 0 : 1;
  if (M <= 16) {
    std::vector<int32_t> w(h.wmib.begin(), h.wmib.begin() + M);
    std::sort(w.begin(), w.end());
    int qcap = 1;
    for (int32_t d = 0; d < D; ++d) {
      int k = 0;
      int64_t sum = 0;
      while (k < M && sum + w[k] <= h.cap[d]) sum += w[k++];
      qcap = std::max(qcap, std::max(k, __builtin_popcountll(h.init_res[d])));
    }
    sp.queue = qcap <= 8 ? 32 : 64;
  }
  const bool batched = std::any_of(h.batch.begin(), h.batch.end(), [](int32_t b) { return b > 1; });
  if (batched) {
    sp.nibble = h.victim_order == WF_VICTIM_PAPER ? -3 : -2;
  } else if (h.victim_order == WF_VICTIM_PAPER) {
    sp.nibble = -1;
  } else {
    // (with replica caps the queue modes keep the resident mask as well: the
    // per-level check reads it)
    sp.nibble = sp.queue;
  }
  sp.has_chains = 0;
  for (int32_t i = 0; i < N; ++i) sp.has_chains |= h.chain_next[i] >= 0 ? 1 : 0;

  return WF_OK;
}

// Plans per wave, waves per workgroup and table placement for one kernel
// mode (scoring rows from HBM, or scoring generated candidates).
wf_status plan_launch(wf_plan_ctx* ctx, const HostWindow& h, bool search, wfp::ScoreParams& sp,
                      bool ring_search = false) {
  const int D = h.D;
  const int tsz = sp.time64 ? 8 : 4;
  const int lds_cu = std::min(ctx->lds_per_cu, 160 * 1024);
  const int lds_blk = std::min(ctx->lds_per_block, lds_cu);
  const int gmax = std::max(1, 64 / D);
  // the workgroup's copies in LDS: every (model, device) load time (the
  // paper reclamation order) and every model's weights
  sp.wg_ld = ((sp.nibble == -1 || sp.nibble == -3) ? (int)align_up((size_t)h.M * D * 4, 16) : 0) +
             (int)align_up((size_t)h.M * 4, 16);
  double best = -1.0;
  for (int tl = 1; tl >= 0; --tl) {
    const int tab_lds = (tl ? sp.t.bytes : 0) + sp.wg_ld;
    for (int G = gmax; G >= 1; --G) {
      wfp::WaveOffsets o{};
      const int wb = wave_layout(h, G, tsz, sp.nwa, sp.nibble, search, o, false);
      int waves = std::min(8, (lds_blk - tab_lds) / std::max(wb, 1));
      if (waves < 1) continue;
      const int lds_wg = tab_lds + waves * wb;
      const int wg_per_cu = std::max(1, lds_cu / lds_wg);
      const int waves_cu = std::min(32, wg_per_cu * waves);
      // walk lanes in flight per CU (at most 8 waves: two per SIMD at the
      // kernel's register use); cached table reads cost about as much as
      // LDS reads, so the table stays in LDS only when that costs no wave
      const double score = (double)std::min(G * D, 64) * std::min(waves_cu, 8) * (tl ? 1.0 : 0.99);
      if (score > best) {
        best = score;
        sp.G = G;
        sp.waves = waves;
        sp.tab_in_lds = tl;
        sp.lds_bytes = lds_wg;
        sp.grid = ctx->n_cu * wg_per_cu;
        sp.wo = o;
      }
    }
  }
  sp.wave_global = 0;
  sp.scratch = nullptr;
  // per-wave regions in HBM (the small per-(device, model) arrays stay in
  // LDS): every lane of a wave busy and up to eight waves per CU, but each
  // per-activation access goes through the cache instead of LDS.  Taken
  // when no LDS layout fits, or when the LDS layout keeps too few walk lanes
  // in flight (deep or wide windows, whose per-plan state fills LDS with a
  // few plans per CU).  The cheaper a walk trip, the more the cache latency
  // of the HBM part shows, so the ratio needed depends on the reclamation
  // mode: 8 with a queue (whose last-slot table then lives in HBM too), 3
  // with a plain or batch-limited scan, 2.1 with the paper's order.
  // Measured on MI355X: paper-order scans at ratios 2.15-6.4 run 1.3-2.4x
  // faster in HBM; other scans at 3.3-6.4 run 1.2-1.7x faster, at 2.0-2.24
  // 1.3-1.5x slower; a queue at 1.6 runs 2.4x slower.
  wfp::WaveOffsets og{};
  const int Gg = gmax, waves_g = 4;
  const int64_t wb_g = wave_layout(h, Gg, tsz, sp.nwa, sp.nibble, search, og, true);
  const int64_t hbm_wave = wb_g - og.split;  // HBM bytes per wave
  const int lds_wg_g = sp.wg_ld + waves_g * og.split;
  // (up to three four-wave workgroups per CU run: the HBM layout's kernel
  // is built for three waves per SIMD; the choices below weigh the two per
  // CU their ratios were measured with)
  const int wgs_fit = lds_wg_g <= lds_blk ? std::max(1, lds_cu / std::max(lds_wg_g, 1)) : 0;
  const int wgs_per_cu = std::min(2, wgs_fit), wgs_run = std::min(3, wgs_fit);
  const double hbm_lanes = (double)std::min(Gg * D, 64) * waves_g * wgs_per_cu;
  if (best < 0 && wgs_per_cu == 0)
    return fail(&ctx->err, WF_EUNSUPPORTED, "window too large for LDS (N=%d, D=%d, M=%d)", h.N, D, h.M);
  const bool paper_scan = sp.nibble == -1 || sp.nibble == -3;
  const double min_ratio = sp.nibble > 0 ? 8.0 : paper_scan ? 2.1 : 3.0;
  if (wgs_per_cu > 0 && (best < 0 || best * min_ratio <= hbm_lanes)) {
    const int64_t cap_bytes = int64_t(1) << 30;
    const int G = Gg, waves = waves_g;
    const wfp::WaveOffsets o = og;
    int64_t wgs = std::min<int64_t>((int64_t)ctx->n_cu * wgs_run,
                                    cap_bytes / std::max<int64_t>(hbm_wave * waves, 1));
    if (wgs < 1 && best >= 0) return WF_OK;  // keep the LDS layout
    if (wgs < 1)
      return fail(&ctx->err, WF_EUNSUPPORTED, "window too large (N=%d, widest level %d, D=%d, M=%d)",
                  h.N, h.wmax, D, h.M);
    sp.G = G;
    sp.waves = waves;
    sp.tab_in_lds = 0;
    sp.wave_global = 1;
    sp.lds_bytes = lds_wg_g;
    sp.grid = (int)wgs;
    sp.wo = o;
  }
  // the ring of recent levels: per-plan state of the current level and the
  // levels a unit can still reach, all in LDS.  Taken over the HBM layout
  // when it keeps as many walk lanes in flight, and over the LDS layout
  // only when that keeps fewer than half as many: building the order level
  // by level costs more per plan than the LDS layout's one sweep.
  // Measured on MI355X: 4,096 activations in 128 levels 12.5 -> 2.55 ms
  // (against the HBM layout); 256 activations with batch limits or replica
  // caps 11.2 -> 13.0 and 8.4 -> 10.9 ms with the ring at 1.3x the LDS
  // layout's lanes.
  sp.ring = 0;
  const char* ring_env = std::getenv("WF_PLAN_RING");
  const bool ring_off = ring_env && std::strcmp(ring_env, "off") == 0;
  const bool ring_force = ring_env && std::strcmp(ring_env, "on") == 0;
  if ((!search || ring_search) && !ring_off && sp.ring_ok && (sp.nibble == 0 || sp.nibble == -2)) {
    const int nwl = (sp.ring_w + 63) / 64 + 1;
    const double cur = sp.wave_global ? hbm_lanes : best;
    double rbest = -1.0;
    int rG = 0, rwaves = 0, rlds = 0, rwgs = 0;
    wfp::WaveOffsets ro{};
    for (int G = gmax; G >= 1; --G) {
      wfp::WaveOffsets o{};
      const int wb = ring_layout(h, sp, G, tsz, nwl, search, o);
      const int waves = std::min(8, (lds_blk - sp.wg_ld) / std::max(wb, 1));
      if (waves < 1) continue;
      const int lds_wg = sp.wg_ld + waves * wb;
      const int wg_per_cu = std::max(1, lds_cu / lds_wg);
      const double score = (double)std::min(G * D, 64) * std::min(std::min(32, wg_per_cu * waves), 8);
      if (score > rbest) {
        rbest = score;
        rG = G;
        rwaves = waves;
        rlds = lds_wg;
        rwgs = wg_per_cu;
        ro = o;
      }
    }
    if (rbest > 0 && (ring_force || (sp.wave_global ? rbest >= cur : rbest >= 2.0 * cur))) {
      sp.ring = 1;
      sp.wave_global = 0;
      sp.tab_in_lds = 0;
      sp.G = rG;
      sp.waves = rwaves;
      sp.lds_bytes = rlds;
      sp.grid = ctx->n_cu * rwgs;
      sp.wo = ro;
      sp.nwa = nwl;
    }
  }
  // the paper's order in the HBM layout keeps its finishes in the ring of
  // recent levels (LDS): the order is built before the walk, as its next use
  // per slot needs every level's order, but the finishes and their atomics
  // stay out of HBM (sp.ring = 2)
  const bool paper_scan_mode = sp.nibble == -1 || sp.nibble == -3;
  if (paper_scan_mode && !search && !ring_off && sp.ring_ok && sp.wave_global && sp.ring == 0) {
    wfp::WaveOffsets o4{};
    const int64_t wb4 = wave_layout(h, sp.G, tsz, sp.nwa, sp.nibble, search, o4, true, sp.ring_size);
    const int lds4 = sp.wg_ld + sp.waves * o4.split;
    // (taken only where the ring keeps the HBM layout's waves per CU: a wide
    // level makes the ring as large as the window)
    const int wg_hbm = std::max(1, std::min(2, lds_cu / std::max(sp.lds_bytes, 1)));
    if (lds4 <= lds_blk && std::max(1, std::min(2, lds_cu / lds4)) >= wg_hbm) {
      const int wg_per_cu = std::max(1, std::min(2, lds_cu / lds4));
      const int64_t hw = std::max<int64_t>((wb4 - o4.split) * sp.waves, 1);
      const int64_t wgs = std::min<int64_t>((int64_t)ctx->n_cu * wg_per_cu, (int64_t(1) << 30) / hw);
      if (wgs >= 1) {
        sp.ring = 2;
        sp.lds_bytes = lds4;
        sp.grid = (int)wgs;
        sp.wo = o4;
      }
    }
  }
  return WF_OK;
}

// Per-wave LDS region of the lean kernel for G plans; returns its size.
int lean_layout(const HostWindow& h, int G, int nwa, wfp::LeanOffsets& o) {
  size_t off = 0;
  auto take = [&](size_t n) {
    const size_t at = off;
    off = align_up(off + std::max<size_t>(n, 1), 16);
    return (int)at;
  };
  const int NB = (h.N + 3) / 4;
  o = wfp::LeanOffsets{};
  o.flags = take((size_t)G * NB);
  o.rec = take((size_t)G * h.N * 2);
  o.mask = take((size_t)G * h.D * nwa * 8);
  const size_t last_bytes = (size_t)G * h.D * h.M * 4;
  const bool paper = h.victim_order == WF_VICTIM_PAPER;
  o.fin = take((size_t)G * h.N * 4);
  // the last slots are read before the walk starts, so they share the
  // finish region (after the candidates' changed sites) where they fit; the
  // paper's order keeps its per-model keys there during the walk
  const size_t patch_bytes = align_up((size_t)G * wfp::kPatchWords * 4, 16);
  if (!paper && patch_bytes + last_bytes <= (size_t)G * h.N * 4)
    o.last = o.fin + (int)patch_bytes;
  else
    o.last = take(last_bytes);
  o.wfm = take((size_t)G * std::max(1, h.W) * 4);
  o.acc = take((size_t)G * 48);
  o.hold = take(h.rcap.empty() && !paper ? 0 : (size_t)G * h.D * 2);
  // (next uses in one byte for at most 256 activations: no next use is 0,
  // as a device's first unit is nobody's next)
  o.nx = take(paper ? (size_t)G * h.N * (h.N <= 256 ? 1 : 2) : 0);
  o.bytes = (int)off;
  return o.bytes;
}


// Whether the lean kernel serves this window's plan scores, and its table
// image and launch plan: uint32 times (proven or checked), at most 16
// models, at most 512 activations (9-bit slot entries), and the tables plus
// the waves' regions in LDS.  Plans per wave: 64 / D; as many waves as LDS
// holds, at most 10 per workgroup for the queue variants (three per SIMD)
// and 8 for the paper's order (two per SIMD).
void plan_lean(wf_plan_ctx* ctx, const HostWindow& h, const wfp::ScoreParams& sp, bool checked,
               Image& img, wfp::LeanParams& lp) {
  lp = wfp::LeanParams{};
  const char* force = std::getenv("WF_PLAN_KERNEL");
  if (force && std::strcmp(force, "general") == 0) return;
  // (batch limits with the default order: the queue's order, passing over
  // leased copies; the paper's order over a resident mask; neither with
  // replica caps)
  const bool batch = sp.nibble == -2 && h.rcap.empty();
  const bool paper = sp.nibble == -1 && h.rcap.empty();
  if (sp.time64 || (sp.nibble != 32 && sp.nibble != 64 && !batch && !paper) || h.N < 1 ||
      h.N > 512 || h.M > 16 || h.D > 64)
    return;
  const int N = h.N, D = h.D, M = h.M, W = h.W;
  // ---- table image (same words as the general image where they coincide) ----
  int64_t origin = INT64_MAX;
  for (int32_t f = 0; f < W; ++f) origin = std::min(origin, h.arrival[f]);
  for (int32_t d = 0; d < D; ++d) origin = std::min(origin, h.free0[d]);
  if (origin == INT64_MAX) origin = 0;
  if (origin != sp.origin) return;
  std::vector<uint32_t> act((size_t)N), alv((size_t)N), aarr((size_t)N), arr((size_t)std::max(W, 1), 0);
  std::vector<uint16_t> cnext((size_t)N);
  for (int32_t f = 0; f < W; ++f) arr[f] = (uint32_t)(h.arrival[f] - origin);
  for (int32_t i = 0; i < N; ++i) {
    const bool ready = h.pred_off[i] == h.pred_off[i + 1] && h.arrival[h.act_wf[i]] <= 0;
    act[i] = (uint32_t)h.act_model[i] | ((uint32_t)h.fusible[i] << 6) | ((uint32_t)ready << 7) |
             ((uint32_t)h.wf_class[h.act_wf[i]] << 8) | ((uint32_t)h.act_wf[i] << 16);
    cnext[i] = h.chain_next[i] >= 0 ? (uint16_t)h.chain_next[i] : (uint16_t)0xffff;
    aarr[i] = arr[h.act_wf[i]];
  }
  for (int32_t l = 0; l < h.n_levels; ++l)
    for (int32_t i = h.level_off[l]; i < h.level_off[l + 1]; ++i)
      alv[i] = (uint32_t)h.level_off[l] | ((uint32_t)(h.level_off[l + 1] - h.level_off[l]) << 16);
  const int32_t E = h.pred_off[N];
  std::vector<uint32_t> edge((size_t)std::max(E, 1), 0);
  for (int32_t v = 0; v < N; ++v)
    for (int32_t k = h.pred_off[v]; k < h.pred_off[v + 1]; ++k)
      edge[k] = (uint32_t)h.pred_idx[k] | ((uint32_t)v << 16);
  std::vector<int32_t> eoff((size_t)h.n_levels + 1);
  for (int32_t l = 0; l <= h.n_levels; ++l) eoff[l] = h.pred_off[h.level_off[l]];
  // device-major: a device lane's rows are contiguous
  std::vector<int32_t> um((size_t)N * D * 2), lw((size_t)M * D * 4, 0);
  for (int32_t i = 0; i < N; ++i)
    for (int32_t d = 0; d < D; ++d) {
      um[((size_t)d * N + i) * 2] = h.lat[(size_t)i * D + d];
      um[((size_t)d * N + i) * 2 + 1] = h.mem[(size_t)i * D + d];
    }
  for (int32_t m = 0; m < M; ++m)
    for (int32_t d = 0; d < D; ++d) {
      int32_t* r = &lw[((size_t)d * M + m) * 4];
      r[0] = h.load[(size_t)m * D + d];
      r[1] = h.wmib[m];
      r[2] = (int32_t)((uint32_t)m * 0x11111111u);
    }
  std::vector<uint32_t> fr((size_t)D);
  for (int32_t d = 0; d < D; ++d) fr[d] = (uint32_t)(h.free0[d] - origin);
  std::vector<uint8_t> has_wf_succ((size_t)N, 0);
  for (int32_t v = 0; v < N; ++v)
    for (int32_t k = h.pred_off[v]; k < h.pred_off[v + 1]; ++k)
      if (h.act_wf[h.pred_idx[k]] == h.act_wf[v]) has_wf_succ[h.pred_idx[k]] = 1;
  std::vector<uint32_t> sink;
  for (int32_t i = 0; i < N; ++i)
    if (!has_wf_succ[i]) sink.push_back((uint32_t)i | ((uint32_t)h.act_wf[i] << 16));
  if ((int)sink.size() != sp.S) return;
  if (sink.empty()) sink.push_back(0);
  wfp::LeanTab& t = lp.t;
  t.lw = img.put(lw.data(), lw.size() * 4);
  t.wmib = img.put(h.wmib.data(), h.wmib.size() * 4);
  t.aarr = img.put(aarr.data(), aarr.size() * 4);
  t.rcap = img.put(h.rcap.data(), h.rcap.size() * 4);
  img.bytes.resize(align_up(img.bytes.size(), 16), 0);
  t.lds_bytes = (int)img.bytes.size();
  t.um = img.put(um.data(), um.size() * 4);
  t.act = img.put(act.data(), act.size() * 4);
  t.alv = img.put(alv.data(), alv.size() * 4);
  t.cnext = img.put(cnext.data(), cnext.size() * 2);
  t.edge = img.put(edge.data(), edge.size() * 4);
  t.eoff = img.put(eoff.data(), eoff.size() * 4);
  t.loff = img.put(h.level_off.data(), h.level_off.size() * 4);
  t.cap = img.put(h.cap.data(), h.cap.size() * 4);
  t.arr = img.put(arr.data(), arr.size() * 4);
  t.res0 = img.put(h.init_res.data(), h.init_res.size() * 8);
  t.free0 = img.put(fr.data(), fr.size() * 4);
  t.sink = img.put(sink.data(), sink.size() * 4);
  t.batch = img.put(h.batch.data(), h.batch.size() * 4);
  img.bytes.resize(align_up(img.bytes.size(), 16), 0);
  t.bytes = (int)img.bytes.size();
  // ---- launch plan ----
  const int lds_cu = std::min(ctx->lds_per_cu, 160 * 1024);
  const int lds_blk = std::min(ctx->lds_per_block, lds_cu);
  const int G = std::max(1, 64 / D);
  wfp::LeanOffsets o{};
  const int wb = lean_layout(h, G, sp.nwa, o);
  const int fit = (lds_blk - t.lds_bytes) / std::max(wb, 1);
  const int waves = std::min(wfp::kLeanWaves, fit);
  if (waves < 2) return;
  lp.G = G;
  lp.waves = waves;
  lp.lds_bytes = t.lds_bytes + waves * wb;
  lp.grid = ctx->n_cu * std::max(1, lds_cu / lp.lds_bytes);
  lp.xwaves = std::min(wfp::kLeanPlainWaves, fit);
  lp.xlds_bytes = t.lds_bytes + lp.xwaves * wb;
  lp.xgrid = ctx->n_cu * std::max(1, lds_cu / lp.xlds_bytes);
  lp.wo = o;
  lp.checked = checked ? 1 : 0;
  lp.qbits = paper ? -1 : sp.queue;
  lp.rcap = h.rcap.empty() ? 0 : 1;
  lp.batch = batch ? 1 : 0;
  lp.paper = paper ? 1 : 0;
  lp.ok = 1;
  // generated candidates: each plan's changed sites live in its finish
  // entries until the walk
  lp.search_ok = N >= 1 + 4 * wfp::kPatchMaxMut ? 1 : 0;
}

// The lean kernel's launch over n plans: the grid never exceeds the groups
// there are.
wfp::LeanParams lean_grid(wfp::LeanParams lp, int64_t n) {
  const int64_t groups = (n + lp.G - 1) / lp.G;
  const int64_t wgs = (groups + lp.waves - 1) / lp.waves;
  if (wgs < lp.grid) lp.grid = (int)wgs;
  return lp;
}

// Launch parameters of one pass over n plans: the grid never exceeds the
// groups there are.
wfp::ScoreParams fit_grid(wfp::ScoreParams sp, int64_t n) {
  const int64_t groups = (n + sp.G - 1) / sp.G;
  const int64_t wgs = (groups + sp.waves - 1) / sp.waves;
  if (wgs < sp.grid) sp.grid = (int)wgs;
  return sp;
}

// Run a scoring launch with the window's parameters, then, for a window
// whose uint32 times are not proven safe, the fp64 pass over the groups it
// flagged (same stream, so in order).  Generated candidates with more than
// kPatchMaxMut mutations take the layout that holds whole rows.
template <typename F>
hipError_t two_pass(const DeviceWindow& dw, bool search, int64_t n, F&& launch, int32_t n_mut = 0) {
  const wfp::ScoreParams& s =
      !search ? dw.sp : (n_mut <= wfp::kPatchMaxMut ? dw.sp_search : dw.sp_search_wide);
  hipError_t e = launch(fit_grid(s, n));
  if (e == hipSuccess && dw.checked) e = launch(fit_grid(search ? dw.sp64_search : dw.sp64, n));
  return e;
}

}  // namespace

extern "C" {

const char* wf_plan_version(void) { return "wf_plan 0.2 (gfx950)"; }

int wf_plan_time_bits(const wf_plan_ctx* ctx) {
  if (!ctx || !ctx->has_window) return 0;
  return ctx->dw.sp.time64 ? 64 : 32;
}

const char* wf_plan_score_kernel(const wf_plan_ctx* ctx) {
  if (!ctx || !ctx->has_window) return "";
  return ctx->dw.lean.ok ? "score_lean" : "score_plans";
}

const char* wf_plan_last_error(const wf_plan_ctx* ctx) {
  return ctx ? ctx->err.c_str() : g_thread_err.c_str();
}

wf_status wf_plan_validate_window(const wf_window_desc* w, char* err, size_t err_len) {
  std::string msg;
  const wf_status st = validate(w, &msg, nullptr);
  if (err && err_len) std::snprintf(err, err_len, "%s", st == WF_OK ? "" : msg.c_str());
  g_thread_err = st == WF_OK ? "" : msg;
  return st;
}

wf_status wf_plan_ctx_create(int hip_device, wf_plan_ctx** out) {
  if (!out) {
    g_thread_err = "out is NULL";
    return WF_EINVAL;
  }
  *out = nullptr;
  int n = 0;
  hipError_t e = hipGetDeviceCount(&n);
  if (e != hipSuccess || n <= 0) {
    g_thread_err = std::string("no HIP device: ") + hipGetErrorString(e);
    return WF_EHIP;
  }
  if (hip_device < 0 || hip_device >= n) {
    g_thread_err = "hip_device out of range";
    return WF_EINVAL;
  }
  wf_plan_ctx* ctx = new (std::nothrow) wf_plan_ctx();
  if (!ctx) {
    g_thread_err = "out of host memory";
    return WF_ENOMEM;
  }
  ctx->device = hip_device;
  int prev = 0;
  (void)hipGetDevice(&prev);
  e = hipSetDevice(hip_device);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&ctx->n_cu, hipDeviceAttributeMultiprocessorCount, hip_device);
  if (e == hipSuccess)
    e = hipDeviceGetAttribute(&ctx->lds_per_block, hipDeviceAttributeMaxSharedMemoryPerBlock, hip_device);
  if (e == hipSuccess)
    e = hipDeviceGetAttribute(&ctx->lds_per_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, hip_device);
  (void)hipSetDevice(prev);
  if (e != hipSuccess) {
    g_thread_err = std::string("device query failed: ") + hipGetErrorString(e);
    delete ctx;
    return WF_EHIP;
  }
  if (ctx->lds_per_cu <= 0) ctx->lds_per_cu = ctx->lds_per_block;
  (void)hipSetDevice(hip_device);
  e = hipMalloc(&ctx->key_work, (size_t)wfp::kArgminKeyBlocks * wfp::ARGMIN_KEY_WORK_BYTES);
  (void)hipSetDevice(prev);
  if (e != hipSuccess) {
    g_thread_err = std::string("work area allocation failed: ") + hipGetErrorString(e);
    delete ctx;
    return WF_ENOMEM;
  }
  *out = ctx;
  return WF_OK;
}

void wf_plan_ctx_destroy(wf_plan_ctx* ctx) {
  if (!ctx) return;
  int prev = 0;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(ctx->device);
  free_device_window(ctx->dw);
  if (ctx->key_work) (void)hipFree(ctx->key_work);
  (void)hipSetDevice(prev);
  delete ctx;
}

wf_status wf_plan_upload_window(wf_plan_ctx* ctx, const wf_window_desc* w) {
  if (!ctx) {
    g_thread_err = "ctx is NULL";
    return WF_EINVAL;
  }
  HostWindow h;
  wf_status st = validate(w, &ctx->err, &h);
  if (st != WF_OK) return st;
  Image img, img64;
  wfp::ScoreParams sp{}, sp64{};
  TimeMode mode;
  st = plan_window(ctx, h, false, img, sp, &mode);
  if (st != WF_OK) return st;
  wfp::ScoreParams sps = sp;
  st = plan_launch(ctx, h, false, sp);
  if (st != WF_OK) return st;
  const bool checked = mode == kTimeChecked;
  // generated candidates: the ring layout where it pays and the window needs
  // no fp64 rescoring pass (the changed sites hold at most kPatchMaxMut
  // mutations; sps_wide serves more)
  wfp::ScoreParams spsw = sps;
  st = plan_launch(ctx, h, true, spsw);
  if (st != WF_OK) return st;
  st = plan_launch(ctx, h, true, sps, !checked);
  if (st != WF_OK) return st;
  wfp::ScoreParams sps64{};
  if (checked) {
    st = plan_window(ctx, h, true, img64, sp64, &mode);
    if (st != WF_OK) return st;
    sps64 = sp64;
    st = plan_launch(ctx, h, false, sp64);
    if (st != WF_OK) return st;
    st = plan_launch(ctx, h, true, sps64);
    if (st != WF_OK) return st;
    sp64.rescore = 1;
    sps64.rescore = 1;
  }

  int prev = 0;
  (void)hipGetDevice(&prev);
  hipError_t e = hipSetDevice(ctx->device);
  if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
  DeviceWindow dw;
  e = hipMalloc(&dw.tab, img.bytes.size());
  if (e != hipSuccess) {
    (void)hipSetDevice(prev);
    ctx->err = "device allocation of the window failed";
    return WF_ENOMEM;
  }
  e = hipMemcpy(dw.tab, img.bytes.data(), img.bytes.size(), hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    free_device_window(dw);
    (void)hipSetDevice(prev);
    return hip_fail(ctx, e, "copying the window to the device");
  }
  if (checked) {
    e = hipMalloc(&dw.tab64, img64.bytes.size());
    if (e != hipSuccess) {
      free_device_window(dw);
      (void)hipSetDevice(prev);
      ctx->err = "device allocation of the window failed";
      return WF_ENOMEM;
    }
    e = hipMemcpy(dw.tab64, img64.bytes.data(), img64.bytes.size(), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      free_device_window(dw);
      (void)hipSetDevice(prev);
      return hip_fail(ctx, e, "copying the window to the device");
    }
  }
  size_t rule_best_at = 0;
  const std::vector<unsigned char> rimg = rule_image(h, &rule_best_at);
  e = hipMalloc(&dw.rules, rimg.size());
  if (e == hipSuccess) e = hipMemcpy(dw.rules, rimg.data(), rimg.size(), hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    free_device_window(dw);
    (void)hipSetDevice(prev);
    return hip_fail(ctx, e, "copying the rule tables to the device");
  }
  dw.rule_pf = static_cast<const unsigned long long*>(dw.rules);
  dw.rule_best = static_cast<const int8_t*>(dw.rules) + rule_best_at;
  // one scratch area serves every pass (they run in order on a stream)
  wfp::ScoreParams* all[5] = {&sp, &sps, &spsw, &sp64, &sps64};
  size_t need = 0;
  for (int i = 0; i < (checked ? 5 : 3); ++i)
    if (all[i]->wave_global)
      need = std::max(need, (size_t)all[i]->grid * all[i]->waves *
                                (size_t)(all[i]->wo.bytes - all[i]->wo.split));
  if (need) {
    e = hipMalloc(&dw.scratch, need);
    if (e != hipSuccess) {
      free_device_window(dw);
      (void)hipSetDevice(prev);
      ctx->err = "device allocation of the scoring scratch failed";
      return WF_ENOMEM;
    }
    for (int i = 0; i < 5; ++i)
      if (all[i]->wave_global) all[i]->scratch = static_cast<unsigned char*>(dw.scratch);
  }
  sp.tab = static_cast<const unsigned char*>(dw.tab);
  sps.tab = static_cast<const unsigned char*>(dw.tab);
  spsw.tab = static_cast<const unsigned char*>(dw.tab);
  Image limg;
  plan_lean(ctx, h, sp, checked, limg, dw.lean);
  if (dw.lean.ok) {
    e = hipMalloc(&dw.tab_lean, limg.bytes.size());
    if (e == hipSuccess)
      e = hipMemcpy(dw.tab_lean, limg.bytes.data(), limg.bytes.size(), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      free_device_window(dw);
      (void)hipSetDevice(prev);
      return hip_fail(ctx, e, "copying the lean kernel's tables to the device");
    }
    dw.lean.tab = static_cast<const unsigned char*>(dw.tab_lean);
  }
  dw.sp = sp;
  dw.sp_search = sps;
  dw.sp_search_wide = spsw;
  dw.checked = checked;
  if (checked) {
    sp64.tab = static_cast<const unsigned char*>(dw.tab64);
    sps64.tab = static_cast<const unsigned char*>(dw.tab64);
    dw.sp64 = sp64;
    dw.sp64_search = sps64;
  }
  if (std::getenv("WF_PLAN_VERBOSE"))
    std::fprintf(stderr,
                 "[wf_plan] N=%d W=%d D=%d M=%d levels=%d wmax=%d time=%s G=%d waves/wg=%d "
                 "grid=%d tables=%s(%d B) wave=%d B (lds part %d B) lds/wg=%d reclaim=%s\n",
                 sp.N, sp.W, sp.D, sp.M, sp.n_levels, h.wmax,
                 sp.time64 ? "fp64" : checked ? "u32+fp64" : "u32", sp.G,
                 sp.waves, sp.grid, sp.wave_global ? "hbm+scratch" : (sp.tab_in_lds ? "lds" : "hbm"),
                 sp.t.bytes, sp.wo.bytes, sp.wave_global ? sp.wo.split : sp.wo.bytes, sp.lds_bytes, sp.nibble == 32 ? "queue32" : sp.nibble == 64 ? "queue64" : sp.nibble == -1 ? "paper-scan" :
                 sp.nibble == -2 ? "batch-scan" : sp.nibble == -3 ? "batch-paper-scan" : "scan");
  if (std::getenv("WF_PLAN_VERBOSE") && sps.ring)
    std::fprintf(stderr, "[wf_plan] generated candidates: ring of recent levels (G=%d, waves/wg=%d), "
                 "changed sites for at most %d mutations\n", sps.G, sps.waves, wfp::kPatchMaxMut);
  if (std::getenv("WF_PLAN_VERBOSE") && sp.ring == 1)
    std::fprintf(stderr, "[wf_plan] ring of recent levels: %d positions (%d levels ahead, %d "
                 "behind), widest level %d, %d mask words per device\n", sp.ring_size, sp.ring_a,
                 sp.ring_b, sp.ring_w, sp.nwa);
  if (std::getenv("WF_PLAN_VERBOSE") && sp.ring == 2)
    std::fprintf(stderr, "[wf_plan] finishes in a ring of recent levels: %d positions (%d levels "
                 "ahead, %d behind); order and slot arrays in HBM\n", sp.ring_size, sp.ring_a,
                 sp.ring_b);
  if (std::getenv("WF_PLAN_VERBOSE") && dw.lean.ok)
    std::fprintf(stderr, "[wf_plan] lean kernel: G=%d waves/wg=%d (queue variants %d) grid=%d (%d) "
                 "tables=%d B wave=%d B lds/wg=%d (%d)\n",
                 dw.lean.G, dw.lean.waves, dw.lean.xwaves, dw.lean.grid, dw.lean.xgrid,
                 dw.lean.t.bytes, dw.lean.wo.bytes, dw.lean.lds_bytes, dw.lean.xlds_bytes);
  free_device_window(ctx->dw);
  ctx->dw = dw;
  ctx->host = std::move(h);
  ctx->has_window = true;
  (void)hipSetDevice(prev);
  ctx->err.clear();
  return WF_OK;
}

wf_status wf_plan_score_batch(wf_plan_ctx* ctx, const int8_t* dev, const uint16_t* prio,
                              const uint8_t* flags, int64_t n_plans, wf_plan_score* scores,
                              const wf_plan_sched* sched, void* hip_stream) {
  if (!ctx) {
    g_thread_err = "ctx is NULL";
    return WF_EINVAL;
  }
  if (!ctx->has_window) return fail(&ctx->err, WF_ENOWINDOW, "no window uploaded");
  if (n_plans < 0) return fail(&ctx->err, WF_EINVAL, "n_plans is negative");
  if (n_plans == 0) return WF_OK;
  if (!scores) return fail(&ctx->err, WF_EINVAL, "scores is NULL");
  if (ctx->host.N > 0 && (!dev || !prio || !flags))
    return fail(&ctx->err, WF_EINVAL, "a plan array (dev, prio, flags) is NULL");
  if (sched && (!sched->start_us || !sched->finish_us || !sched->load_start_us || !sched->peak_mib))
    return fail(&ctx->err, WF_EINVAL, "a schedule array is NULL");
  int prev = 0;
  (void)hipGetDevice(&prev);
  hipError_t e = hipSetDevice(ctx->device);
  if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
  const DeviceWindow& dw = ctx->dw;
  if (!sched && dw.lean.ok) {
    // the lean kernel, then (times not proven below 2^32) the general fp64
    // pass over the groups holding a plan whose times saturated
    wfp::LeanParams lp = dw.lean;
    const int64_t groups = (n_plans + lp.G - 1) / lp.G;
    const int64_t wgs = (groups + lp.waves - 1) / lp.waves;
    if (wgs < lp.grid) lp.grid = (int)wgs;
    e = wfp::launch_score_lean(dw.sp, lp, dev, prio, flags, n_plans, scores, nullptr, false,
                               static_cast<hipStream_t>(hip_stream));
    if (e == hipSuccess && dw.checked)
      e = wfp::launch_score(fit_grid(dw.sp64, n_plans), dev, prio, flags, n_plans, scores, nullptr,
                            nullptr, static_cast<hipStream_t>(hip_stream));
  } else {
    e = two_pass(dw, false, n_plans, [&](const wfp::ScoreParams& sp) {
      return wfp::launch_score(sp, dev, prio, flags, n_plans, scores, sched, nullptr,
                               static_cast<hipStream_t>(hip_stream));
    });
  }
  (void)hipSetDevice(prev);
  if (e != hipSuccess) return hip_fail(ctx, e, "launching the scoring kernel");
  return WF_OK;
}

// Shared argument checks of the candidate-generation calls.
static wf_status search_args(wf_plan_ctx* ctx, const int8_t* dev, const uint16_t* prio,
                             const uint8_t* flags, int32_t mode, int32_t n_mut, int64_t first,
                             int64_t n_candidates) {
  if (!ctx) {
    g_thread_err = "ctx is NULL";
    return WF_EINVAL;
  }
  if (!ctx->has_window) return fail(&ctx->err, WF_ENOWINDOW, "no window uploaded");
  if (mode != WF_SEARCH_UNIFORM && mode != WF_SEARCH_RULES)
    return fail(&ctx->err, WF_EINVAL, "mode = %d is not a WF_SEARCH_* value", (int)mode);
  if (n_mut < 0 || n_mut > WF_MAX_MUT)
    return fail(&ctx->err, WF_EINVAL, "n_mut must be in [0, %d]", WF_MAX_MUT);
  if (n_candidates < 0) return fail(&ctx->err, WF_EINVAL, "n_candidates is negative");
  if (first < 0 || first > (int64_t(1) << 62) - n_candidates)
    return fail(&ctx->err, WF_EINVAL, "candidates must lie in [0, 2^62)");
  if (ctx->host.N > 0 && (!dev || !prio || !flags))
    return fail(&ctx->err, WF_EINVAL, "an incumbent row (dev, prio, flags) is NULL");
  return WF_OK;
}

static wfp::SearchArgs search_params(const wf_plan_ctx* ctx, int32_t mode, uint64_t seed,
                                     int32_t n_mut, int64_t first) {
  return wfp::SearchArgs{seed, n_mut, mode, first, ctx->host.D, ctx->dw.rule_best,
                         ctx->dw.rule_pf,
                         reinterpret_cast<const unsigned long long*>(ctx->dw.sp.tab + ctx->dw.sp.t.elig)};
}

wf_status wf_plan_search_batch(wf_plan_ctx* ctx, const int8_t* dev, const uint16_t* prio,
                               const uint8_t* flags, int32_t mode, uint64_t seed, int32_t n_mut,
                               int64_t first, int64_t n_candidates, wf_plan_score* scores,
                               void* hip_stream) {
  wf_status st = search_args(ctx, dev, prio, flags, mode, n_mut, first, n_candidates);
  if (st != WF_OK) return st;
  if (n_candidates == 0) return WF_OK;
  if (!scores) return fail(&ctx->err, WF_EINVAL, "scores is NULL");
  int prev = 0;
  (void)hipGetDevice(&prev);
  hipError_t e = hipSetDevice(ctx->device);
  if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
  const wfp::SearchArgs sa = search_params(ctx, mode, seed, n_mut, first);
  const DeviceWindow& dw = ctx->dw;
  if (dw.lean.ok && !dw.lean.batch && !dw.lean.paper && dw.lean.search_ok &&
      n_mut <= wfp::kPatchMaxMut) {
    // the lean kernel generates the candidates as the incumbent plus their
    // changed sites; then (times not proven below 2^32) the general fp64
    // pass over the groups holding a candidate whose times saturated
    wfp::LeanParams lp = dw.lean;
    const int64_t groups = (n_candidates + lp.G - 1) / lp.G;
    const int64_t wgs = (groups + lp.waves - 1) / lp.waves;
    if (wgs < lp.grid) lp.grid = (int)wgs;
    e = wfp::launch_score_lean(dw.sp, lp, dev, prio, flags, n_candidates, scores, &sa, false,
                               static_cast<hipStream_t>(hip_stream));
    if (e == hipSuccess && dw.checked)
      e = wfp::launch_score(fit_grid(dw.sp64_search, n_candidates), dev, prio, flags, n_candidates,
                            scores, nullptr, &sa, static_cast<hipStream_t>(hip_stream));
  } else {
    e = two_pass(
        dw, true, n_candidates,
        [&](const wfp::ScoreParams& sp) {
          return wfp::launch_score(sp, dev, prio, flags, n_candidates, scores, nullptr, &sa,
                                   static_cast<hipStream_t>(hip_stream));
        },
        n_mut);
  }
  (void)hipSetDevice(prev);
  if (e != hipSuccess) return hip_fail(ctx, e, "launching the scoring kernel");
  return WF_OK;
}

wf_status wf_plan_search_rows(wf_plan_ctx* ctx, const int8_t* dev, const uint16_t* prio,
                              const uint8_t* flags, int32_t mode, uint64_t seed, int32_t n_mut,
                              int64_t first, int64_t n_candidates, int8_t* out_dev,
                              uint16_t* out_prio, uint8_t* out_flags, void* hip_stream) {
  wf_status st = search_args(ctx, dev, prio, flags, mode, n_mut, first, n_candidates);
  if (st != WF_OK) return st;
  if (n_candidates == 0 || ctx->host.N == 0) return WF_OK;
  if (!out_dev || !out_prio || !out_flags)
    return fail(&ctx->err, WF_EINVAL, "an output row array is NULL");
  if (n_candidates >= (int64_t(1) << 31))
    return fail(&ctx->err, WF_EINVAL, "n_candidates must be below 2^31");
  int prev = 0;
  (void)hipGetDevice(&prev);
  hipError_t e = hipSetDevice(ctx->device);
  if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
  const wfp::SearchArgs sa = search_params(ctx, mode, seed, n_mut, first);
  e = wfp::launch_search_rows(ctx->dw.sp_search, dev, prio, flags, sa, n_candidates, out_dev,
                              out_prio, out_flags, static_cast<hipStream_t>(hip_stream));
  (void)hipSetDevice(prev);
  if (e != hipSuccess) return hip_fail(ctx, e, "launching the candidate-row kernel");
  return WF_OK;
}

wf_status wf_plan_argmin(wf_plan_ctx* ctx, const wf_plan_score* scores, int64_t n_plans,
                         int64_t* out_index, void* hip_stream) {
  if (!ctx) {
    g_thread_err = "ctx is NULL";
    return WF_EINVAL;
  }
  if (!ctx->has_window) return fail(&ctx->err, WF_ENOWINDOW, "no window uploaded");
  if (n_plans < 0 || n_plans >= (int64_t(1) << 32))
    return fail(&ctx->err, WF_EINVAL, "n_plans must be in [0, 2^32)");
  if (!out_index) return fail(&ctx->err, WF_EINVAL, "out_index is NULL");
  if (n_plans > 0 && !scores) return fail(&ctx->err, WF_EINVAL, "scores is NULL");
  int prev = 0;
  (void)hipGetDevice(&prev);
  hipError_t e = hipSetDevice(ctx->device);
  if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
  e = wfp::launch_argmin(scores, n_plans, out_index, ctx->key_work,
                         static_cast<hipStream_t>(hip_stream));
  (void)hipSetDevice(prev);
  if (e != hipSuccess) return hip_fail(ctx, e, "launching the argmin kernels");
  return WF_OK;
}

wf_status wf_plan_argmin_noalloc(const wf_plan_score* scores, int64_t n_plans,
                                 int64_t* out_index, void* hip_stream) {
  if (n_plans < 0 || n_plans >= (int64_t(1) << 32)) {
    g_thread_err = "n_plans must be in [0, 2^32)";
    return WF_EINVAL;
  }
  if (!out_index) {
    g_thread_err = "out_index is NULL";
    return WF_EINVAL;
  }
  if (n_plans > 0 && !scores) {
    g_thread_err = "scores is NULL";
    return WF_EINVAL;
  }
  int device = 0;
  hipError_t e = hipGetDevice(&device);
  void* work = nullptr;
  if (e == hipSuccess) e = wfp::static_scratch(device, &work);
  if (e != hipSuccess) {
    g_thread_err = std::string("static work area of the current device: ") + hipGetErrorString(e);
    return WF_EHIP;
  }
  e = wfp::launch_argmin(scores, n_plans, out_index, work, static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) {
    g_thread_err = std::string("launching the argmin kernels: ") + hipGetErrorString(e);
    return WF_EHIP;
  }
  g_thread_err.clear();
  return WF_OK;
}

wf_status wf_plan_score_keys(wf_plan_ctx* ctx, const int8_t* dev, const uint16_t* prio,
                             const uint8_t* flags, int64_t n_plans, wf_plan_key* keys,
                             void* hip_stream) {
  if (!ctx) {
    g_thread_err = "ctx is NULL";
    return WF_EINVAL;
  }
  if (!ctx->has_window) return fail(&ctx->err, WF_ENOWINDOW, "no window uploaded");
  if (n_plans < 0) return fail(&ctx->err, WF_EINVAL, "n_plans is negative");
  if (n_plans == 0) return WF_OK;
  if (!keys) return fail(&ctx->err, WF_EINVAL, "keys is NULL");
  if (ctx->host.N > 0 && (!dev || !prio || !flags))
    return fail(&ctx->err, WF_EINVAL, "a plan array (dev, prio, flags) is NULL");
  int prev = 0;
  (void)hipGetDevice(&prev);
  hipError_t e = hipSetDevice(ctx->device);
  if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
  const DeviceWindow& dw = ctx->dw;
  if (dw.lean.ok && !dw.lean.batch && !dw.lean.paper) {
    // the lean kernel's key mode, then the general fp64 pass over the groups
    // holding a plan whose uint32 times saturated
    const wfp::LeanParams lp = lean_grid(dw.lean, n_plans);
    e = wfp::launch_score_lean(dw.sp, lp, dev, prio, flags, n_plans, keys, nullptr, true,
                               static_cast<hipStream_t>(hip_stream));
    if (e == hipSuccess && dw.checked)
      e = wfp::launch_score_keys(fit_grid(dw.sp64, n_plans), dev, prio, flags, n_plans, keys,
                                 nullptr, static_cast<hipStream_t>(hip_stream));
  } else {
    e = two_pass(dw, false, n_plans, [&](const wfp::ScoreParams& sp) {
      return wfp::launch_score_keys(sp, dev, prio, flags, n_plans, keys, nullptr,
                                    static_cast<hipStream_t>(hip_stream));
    });
  }
  (void)hipSetDevice(prev);
  if (e != hipSuccess) return hip_fail(ctx, e, "launching the ranking-key kernel");
  return WF_OK;
}

wf_status wf_plan_search_keys(wf_plan_ctx* ctx, const int8_t* dev, const uint16_t* prio,
                              const uint8_t* flags, int32_t mode, uint64_t seed, int32_t n_mut,
                              int64_t first, int64_t n_candidates, wf_plan_key* keys,
                              void* hip_stream) {
  wf_status st = search_args(ctx, dev, prio, flags, mode, n_mut, first, n_candidates);
  if (st != WF_OK) return st;
  if (n_candidates == 0) return WF_OK;
  if (!keys) return fail(&ctx->err, WF_EINVAL, "keys is NULL");
  int prev = 0;
  (void)hipGetDevice(&prev);
  hipError_t e = hipSetDevice(ctx->device);
  if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
  const wfp::SearchArgs sa = search_params(ctx, mode, seed, n_mut, first);
  const DeviceWindow& dw = ctx->dw;
  if (dw.lean.ok && !dw.lean.batch && !dw.lean.paper && dw.lean.search_ok &&
      n_mut <= wfp::kPatchMaxMut) {
    const wfp::LeanParams lp = lean_grid(dw.lean, n_candidates);
    e = wfp::launch_score_lean(dw.sp, lp, dev, prio, flags, n_candidates, keys, &sa, true,
                               static_cast<hipStream_t>(hip_stream));
    if (e == hipSuccess && dw.checked)
      e = wfp::launch_score_keys(fit_grid(dw.sp64_search, n_candidates), dev, prio, flags,
                                 n_candidates, keys, &sa, static_cast<hipStream_t>(hip_stream));
  } else {
    e = two_pass(
        dw, true, n_candidates,
        [&](const wfp::ScoreParams& sp) {
          return wfp::launch_score_keys(sp, dev, prio, flags, n_candidates, keys, &sa,
                                        static_cast<hipStream_t>(hip_stream));
        },
        n_mut);
  }
  (void)hipSetDevice(prev);
  if (e != hipSuccess) return hip_fail(ctx, e, "launching the ranking-key kernel");
  return WF_OK;
}

wf_status wf_plan_prefix(wf_plan_ctx* ctx, const int8_t* dev, const int64_t* start_us,
                         const int64_t* finish_us, const int64_t* load_start_us,
                         const uint64_t* reclaimed, uint8_t* commit, uint64_t* commit_reclaimed,
                         int64_t* t_next_us, void* hip_stream) {
  if (!ctx) {
    g_thread_err = "ctx is NULL";
    return WF_EINVAL;
  }
  if (!ctx->has_window) return fail(&ctx->err, WF_ENOWINDOW, "no window uploaded");
  if (!t_next_us) return fail(&ctx->err, WF_EINVAL, "t_next_us is NULL");
  if (ctx->host.N > 0 && (!dev || !start_us || !finish_us || !load_start_us || !reclaimed ||
                          !commit || !commit_reclaimed))
    return fail(&ctx->err, WF_EINVAL, "a plan, schedule or output array is NULL");
  // the earliest workflow arrival after the window time 0
  int64_t next_arrival = INT64_MAX;
  for (int32_t f = 0; f < ctx->host.W; ++f)
    if (ctx->host.arrival[f] > 0 && ctx->host.arrival[f] < next_arrival) next_arrival = ctx->host.arrival[f];
  int prev = 0;
  (void)hipGetDevice(&prev);
  hipError_t e = hipSetDevice(ctx->device);
  if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
  e = wfp::launch_prefix(ctx->dw.sp, next_arrival, dev, start_us, finish_us, load_start_us, reclaimed,
                         commit, commit_reclaimed, t_next_us, static_cast<hipStream_t>(hip_stream));
  (void)hipSetDevice(prev);
  if (e != hipSuccess) return hip_fail(ctx, e, "launching the prefix kernel");
  return WF_OK;
}

wf_status wf_plan_argmin_keys(wf_plan_ctx* ctx, const wf_plan_key* keys, int64_t n_plans,
                              int64_t* out_index, void* hip_stream) {
  if (!ctx) {
    g_thread_err = "ctx is NULL";
    return WF_EINVAL;
  }
  if (!ctx->has_window) return fail(&ctx->err, WF_ENOWINDOW, "no window uploaded");
  if (n_plans < 0 || n_plans > (int64_t(1) << 62))
    return fail(&ctx->err, WF_EINVAL, "n_plans must be in [0, 2^62]");
  if (!out_index) return fail(&ctx->err, WF_EINVAL, "out_index is NULL");
  if (n_plans > 0 && !keys) return fail(&ctx->err, WF_EINVAL, "keys is NULL");
  int prev = 0;
  (void)hipGetDevice(&prev);
  hipError_t e = hipSetDevice(ctx->device);
  if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
  e = wfp::launch_argmin_keys(keys, n_plans, out_index, ctx->key_work,
                              static_cast<hipStream_t>(hip_stream));
  (void)hipSetDevice(prev);
  if (e != hipSuccess) return hip_fail(ctx, e, "launching the ranking-key argmin kernels");
  return WF_OK;
}

}  // extern "C"

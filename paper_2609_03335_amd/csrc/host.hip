// Host side of the C ABI declared in include/wf_plan.h: contexts, window
// validation and derivation (levels, Eq. 3 fusibility, unique successors),
// the device copy of the window, launch geometry, and the two entry points
// that enqueue work.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
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
  float w_mk = 1.f, w_p95 = 0.f;
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
      return fail(err, WF_EINVAL, "wf_arrival_us[%lld] outside [0, 2^62]", (long long)f);
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
      return fail(err, WF_EINVAL, "dev_free0_us[%lld] outside [0, 2^62]", (long long)d);
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
  if (!out) return WF_OK;

  HostWindow& h = *out;
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
  void* blob = nullptr;
  size_t bytes = 0;
  wfp::WindowDev view{};
  wfp::ScoreLaunch launch{};
  int64_t* scratch = nullptr;  // big-mode finish times and workflow maxima
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
};

namespace {

wf_status hip_fail(wf_plan_ctx* ctx, hipError_t e, const char* what) {
  ctx->err = std::string(what) + ": " + hipGetErrorString(e);
  return WF_EHIP;
}

void free_device_window(DeviceWindow& dw) {
  if (dw.blob) (void)hipFree(dw.blob);
  if (dw.scratch) (void)hipFree(dw.scratch);
  dw = DeviceWindow{};
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Carve the scoring kernel's LDS for G plans per wave; returns total bytes.
int lds_layout(const HostWindow& h, int G, bool big, wfp::ScoreLaunch& L) {
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes, 16);
    return (int)o;
  };
  L.G = G;
  L.big = big ? 1 : 0;
  L.nwords = std::max(1, (h.wmax + 63) / 64);
  L.off_pos = take((size_t)G * std::max(1, h.wmax) * 2);
  L.off_claim = take((size_t)G * L.nwords * 8);
  L.off_mask = take((size_t)G * h.D * L.nwords * 8);
  L.off_cnt = take((size_t)G * h.D * h.M * 4);
  L.off_last = take((size_t)G * h.D * h.M * 4);
  L.off_acc = take((size_t)G * sizeof(wfp::PlanAcc));
  if (!big) {
    L.off_finish = take((size_t)G * std::max(1, h.N) * 8);
    L.off_wfmax = take((size_t)G * std::max(1, h.W) * 8);
    L.scratch_per_wave = 0;
  } else {
    L.off_finish = L.off_wfmax = 0;
    L.scratch_per_wave = (int64_t)G * (std::max(1, h.N) + std::max(1, h.W));
  }
  L.lds_bytes = (int)off;
  return L.lds_bytes;
}

wf_status plan_launch(wf_plan_ctx* ctx, const HostWindow& h, wfp::ScoreLaunch& L) {
  const int gmax = std::max(1, 64 / h.D);
  for (int pass = 0; pass < 2; ++pass) {
    const bool big = pass == 1;
    for (int G = gmax; G >= 1; --G) {
      if (lds_layout(h, G, big, L) <= ctx->lds_per_block) {
        const int per_cu = std::max(1, std::min(32, ctx->lds_per_cu / std::max(1, L.lds_bytes)));
        L.grid = ctx->n_cu * per_cu;
        return WF_OK;
      }
    }
  }
  return fail(&ctx->err, WF_EUNSUPPORTED,
              "window needs more LDS than a workgroup may use (widest level %d, %d devices, %d models)",
              h.wmax, h.D, h.M);
}

}  // namespace

extern "C" {

const char* wf_plan_version(void) { return "wf_plan 0.1 (gfx950)"; }

const char* wf_plan_last_error(const wf_plan_ctx* ctx) {
  return ctx ? ctx->err.c_str() : g_thread_err.c_str();
}

wf_status wf_plan_validate_window(const wf_window_desc* w, char* err, size_t err_len) {
  std::string msg;
  const wf_status st = validate(w, &msg, nullptr);
  if (err && err_len) {
    std::snprintf(err, err_len, "%s", st == WF_OK ? "" : msg.c_str());
  }
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
  *out = ctx;
  return WF_OK;
}

void wf_plan_ctx_destroy(wf_plan_ctx* ctx) {
  if (!ctx) return;
  int prev = 0;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(ctx->device);
  free_device_window(ctx->dw);
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
  wfp::ScoreLaunch L{};
  st = plan_launch(ctx, h, L);
  if (st != WF_OK) return st;

  // one device allocation holding every table
  std::vector<std::pair<const void*, size_t>> parts = {
      {h.act_model.data(), h.act_model.size() * 4}, {h.act_wf.data(), h.act_wf.size() * 4},
      {h.fusible.data(), h.fusible.size()},         {h.chain_next.data(), h.chain_next.size() * 4},
      {h.pred_off.data(), h.pred_off.size() * 4},   {h.pred_idx.data(), h.pred_idx.size() * 4},
      {h.lat.data(), h.lat.size() * 4},             {h.mem.data(), h.mem.size() * 4},
      {h.arrival.data(), h.arrival.size() * 8},     {h.cap.data(), h.cap.size() * 4},
      {h.wmib.data(), h.wmib.size() * 4},           {h.load.data(), h.load.size() * 4},
      {h.init_res.data(), h.init_res.size() * 8},   {h.free0.data(), h.free0.size() * 8},
      {h.level_off.data(), h.level_off.size() * 4}};
  std::vector<size_t> offs;
  size_t total = 0;
  for (auto& p : parts) {
    offs.push_back(total);
    total = align_up(total + p.second, 256);
  }
  std::vector<unsigned char> staging(total, 0);
  for (size_t i = 0; i < parts.size(); ++i)
    if (parts[i].second) std::memcpy(staging.data() + offs[i], parts[i].first, parts[i].second);

  int prev = 0;
  (void)hipGetDevice(&prev);
  hipError_t e = hipSetDevice(ctx->device);
  if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
  DeviceWindow dw;
  e = hipMalloc(&dw.blob, total);
  if (e != hipSuccess) {
    (void)hipSetDevice(prev);
    ctx->err = "device allocation of the window failed";
    return WF_ENOMEM;
  }
  if (L.big) {
    e = hipMalloc(&dw.scratch, (size_t)L.grid * (size_t)L.scratch_per_wave * 8);
    if (e != hipSuccess) {
      free_device_window(dw);
      (void)hipSetDevice(prev);
      ctx->err = "device allocation of the scoring scratch failed";
      return WF_ENOMEM;
    }
  }
  e = hipMemcpy(dw.blob, staging.data(), total, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    free_device_window(dw);
    (void)hipSetDevice(prev);
    return hip_fail(ctx, e, "copying the window to the device");
  }
  dw.bytes = total;
  unsigned char* b = static_cast<unsigned char*>(dw.blob);
  wfp::WindowDev& v = dw.view;
  v.N = h.N;
  v.W = h.W;
  v.M = h.M;
  v.D = h.D;
  v.NB = (h.N + 3) / 4;
  v.n_levels = h.n_levels;
  v.wmax = std::max(1, h.wmax);
  v.min_arrival = h.min_arrival;
  v.w_mk = h.w_mk;
  v.w_p95 = h.w_p95;
  v.act_model = reinterpret_cast<const int32_t*>(b + offs[0]);
  v.act_wf = reinterpret_cast<const int32_t*>(b + offs[1]);
  v.fusible = reinterpret_cast<const uint8_t*>(b + offs[2]);
  v.chain_next = reinterpret_cast<const int32_t*>(b + offs[3]);
  v.pred_off = reinterpret_cast<const int32_t*>(b + offs[4]);
  v.pred_idx = reinterpret_cast<const int32_t*>(b + offs[5]);
  v.lat = reinterpret_cast<const int32_t*>(b + offs[6]);
  v.mem = reinterpret_cast<const int32_t*>(b + offs[7]);
  v.arrival = reinterpret_cast<const int64_t*>(b + offs[8]);
  v.cap = reinterpret_cast<const int32_t*>(b + offs[9]);
  v.wmib = reinterpret_cast<const int32_t*>(b + offs[10]);
  v.load = reinterpret_cast<const int32_t*>(b + offs[11]);
  v.init_res = reinterpret_cast<const uint64_t*>(b + offs[12]);
  v.free0 = reinterpret_cast<const int64_t*>(b + offs[13]);
  v.level_off = reinterpret_cast<const int32_t*>(b + offs[14]);
  dw.launch = L;
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
  wfp::ScoreLaunch L = ctx->dw.launch;
  const int64_t groups = (n_plans + L.G - 1) / L.G;
  if (groups < L.grid) L.grid = (int)groups;
  e = wfp::launch_score(ctx->dw.view, L, ctx->dw.scratch, dev, prio, flags, n_plans, scores, sched,
                        static_cast<hipStream_t>(hip_stream));
  (void)hipSetDevice(prev);
  if (e != hipSuccess) return hip_fail(ctx, e, "launching the scoring kernel");
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
  e = wfp::launch_argmin(scores, n_plans, out_index, ctx->n_cu * 4, static_cast<hipStream_t>(hip_stream));
  (void)hipSetDevice(prev);
  if (e != hipSuccess) return hip_fail(ctx, e, "launching the argmin kernels");
  return WF_OK;
}

}  // extern "C"

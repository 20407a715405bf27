// extern "C" entry points of libfairserve.so (declared in include/fairserve.h):
// synchronous argument checks, workspace layout, and kernel sequencing.
#include <cmath>
#include <cstring>
#include <mutex>

#include "fs_device.h"
#include "fs_launch.h"

namespace fs {

// Workspace of fs_fairness_metrics_noalloc: one copy per GPU, held until the process
// ends.  Host code never passes this name to a kernel or a copy (on the host it is only
// a stand-in for the symbol): it uses the device address that hipGetSymbolAddress gives
// for the current GPU.
constexpr size_t kScratchBytes = size_t(32) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

__global__ void k_zero_i32(int32_t *p) {
  if (threadIdx.x == 0) *p = 0;
}

hipError_t launch_zero_i32(int32_t *p, hipStream_t stream) {
  hipLaunchKernelGGL(k_zero_i32, dim3(1), dim3(64), 0, stream, p);
  return hipGetLastError();
}

namespace {

constexpr size_t kAlign = 256;

bool aligned(const void *p) { return (reinterpret_cast<uintptr_t>(p) % kAlign) == 0; }

// Checks that need no device access: shapes, the host copy of the replica offsets,
// and which optional arrays are present.  A trace without requests may leave its
// per-request arrays NULL (an empty device tensor has no storage).
fs_status check_trace(const fs_trace *t, bool need_lengths) {
  if (!t || t->n_replicas < 1 || t->n_users < 1 || t->n_apps < 1 || t->n_apps > kMaxApps)
    return FS_E_ARG;
  if (!t->rep_off_h || !t->rep_off) return FS_E_ARG;
  if (t->rep_off_h[0] != 0) return FS_E_ARG;
  for (int32_t r = 0; r < t->n_replicas; ++r) {
    int64_t n = t->rep_off_h[r + 1] - t->rep_off_h[r];
    if (n < 0 || n > INT32_MAX - 64) return FS_E_ARG;
  }
  if (int64_t(t->n_replicas) * t->n_users > (int64_t(1) << 31)) return FS_E_ARG;
  if (t->rep_off_h[t->n_replicas] == 0) return FS_OK;
  if (!t->ts_us || !t->user || !t->app) return FS_E_ARG;
  bool any = t->call || t->head || t->prev;
  bool all = t->call && t->head && t->prev;
  if (any && !all) return FS_E_ARG;
  if (need_lengths && (!t->len_in || !t->len_out)) return FS_E_ARG;
  return FS_OK;
}

// Per-request array p is present, or not needed because the trace has no requests.
bool per_request(const fs_trace *t, const void *p) {
  return p != nullptr || t->rep_off_h[t->n_replicas] == 0;
}

fs_status check_weights(const fs_trace *t, const fs_weights *w) {
  if (!w || w->n_stages < 1 || w->n_stages > 4096 || !w->coef) return FS_E_ARG;
  int64_t table = int64_t(t->n_apps) * w->n_stages * 3;
  if (w->coef_rep_stride != 0 && w->coef_rep_stride != table) return FS_E_ARG;
  if (w->prio && w->prio_rep_stride != 0 && w->prio_rep_stride != t->n_users) return FS_E_ARG;
  return FS_OK;
}

fs_status check_limits(const fs_trace *t, const fs_limits *l) {
  if (!l || l->window_us <= 0 || l->t_user < 0 || !l->t_app_h || l->app_scope < 0 ||
      l->app_scope > 1)
    return FS_E_ARG;
  for (int32_t a = 0; a < t->n_apps; ++a)
    if (l->t_app_h[a] < 0) return FS_E_ARG;
  return FS_OK;
}

fs_status check_engine(const fs_engine *e) {
  if (!e || e->step_us <= 0 || e->cap_tokens <= 0 || e->cap_tokens > kCapLimit ||
      (e->flags &
       ~(FS_ENGINE_GLOBAL_ONLY | FS_ENGINE_FCFS | FS_ENGINE_BLIND | FS_ENGINE_LITERAL)))
    return FS_E_ARG;
  return FS_OK;
}

fs_status check_outputs(const fs_trace *t, const fs_outputs *o) {
  if (!o || !per_request(t, o->status) || !per_request(t, o->admit_step) || !o->counter ||
      !o->steps || !o->decisions || !o->max_gap || !o->err)
    return FS_E_ARG;
  return FS_OK;
}

fs_status hip_status(hipError_t e) { return e == hipSuccess ? FS_OK : FS_E_HIP; }

int64_t n_records(const fs_trace *t) { return t->rep_off_h[t->n_replicas]; }

size_t round_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// The device address of `scratch` on the current GPU, looked up once per device.
constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void *scratch_ptr[kMaxDevices] = {};

fs_status scratch_on_current_device(void **ptr) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return FS_E_HIP;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_ptr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return FS_E_HIP;
    scratch_ptr[dev] = p;
  }
  *ptr = scratch_ptr[dev];
  return FS_OK;
}

}  // namespace
}  // namespace fs

using namespace fs;

extern "C" {

const char *fs_status_string(fs_status s) {
  switch (s) {
    case FS_OK: return "ok";
    case FS_E_ARG: return "invalid argument";
    case FS_E_ORDER: return "arrival times decrease within a replica";
    case FS_E_RANGE: return "value out of range";
    case FS_E_OVERFLOW: return "fixed-point overflow (cost or counter reached 2^62)";
    case FS_E_WORKSPACE: return "workspace or state buffer too small";
    case FS_E_STATE: return "state buffer does not match this trace";
    case FS_E_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

fs_status fs_sync_status(hipStream_t stream, const int32_t *err) {
  if (!err) return FS_E_ARG;
  if (hipStreamSynchronize(stream) != hipSuccess) return FS_E_HIP;
  int32_t v = 0;
  if (hipMemcpy(&v, err, sizeof(v), hipMemcpyDeviceToHost) != hipSuccess) return FS_E_HIP;
  return fs_status(v);
}

fs_status fs_coef_from_expectations(int32_t n_apps, int32_t n_stages, const double *e_in_h,
                                    const double *e_sys_h, const double *e_out_h, int64_t K,
                                    int64_t *coef_h) {
  if (n_apps < 1 || n_stages < 1 || K < 1 || K > (int64_t(1) << 20) || !e_in_h || !e_sys_h ||
      !e_out_h || !coef_h)
    return FS_E_ARG;
  // alpha, beta, gamma: input, system and output token weights
  const int64_t weight[3] = {1, 2, 1};
  for (int64_t at = 0; at < int64_t(n_apps) * n_stages; ++at) {
    double w_aj = double(weight[0]) * e_in_h[at] + double(weight[1]) * e_sys_h[at] +
                  double(weight[2]) * e_out_h[at];
    if (!(w_aj > 0.0)) return FS_E_ARG;
    for (int x = 0; x < 3; ++x) {
      double scaled = double((int64_t(1) << 16) * K * weight[x]) / w_aj;
      double r = std::nearbyint(scaled);  // round half to even
      if (!(r >= 0.0) || r >= double(kCoefLimit)) return FS_E_RANGE;
      coef_h[at * 3 + x] = int64_t(r);
    }
  }
  return FS_OK;
}

size_t fs_history_workspace(const fs_trace *t, int32_t n_stages) {
  if (check_trace(t, false) != FS_OK || n_stages < 1 || n_stages > 4096) return 0;
  return history_workspace_bytes(t, n_stages);
}

fs_status fs_weights_from_history(const fs_trace *t, int32_t n_stages, int64_t K,
                                  int32_t base_limit, int64_t *stats, int64_t *coef,
                                  int32_t *t_app, void *ws, size_t ws_bytes, int32_t *err,
                                  hipStream_t stream) {
  fs_status s = check_trace(t, true);
  if (s != FS_OK) return s;
  if (n_stages < 1 || n_stages > 4096 || K < 1 || K > (int64_t(1) << 20) || base_limit < 0 ||
      !stats || !err || n_records(t) >= history_max_records())
    return FS_E_ARG;
  const size_t need = history_workspace_bytes(t, n_stages);
  if (need > 0 && (!ws || !aligned(ws) || ws_bytes < need)) return FS_E_WORKSPACE;
  // the first kernel clears err
  return hip_status(
      launch_history(t, n_stages, K, base_limit, stats, coef, t_app, ws, err, stream));
}

fs_status fs_cost(const fs_trace *t, const fs_weights *w, int64_t *cost, int32_t *err,
                  hipStream_t stream) {
  fs_status s = check_trace(t, true);
  if (s == FS_OK) s = check_weights(t, w);
  if (s != FS_OK) return s;
  if (!per_request(t, cost) || !err) return FS_E_ARG;
  if (launch_zero_i32(err, stream) != hipSuccess) return FS_E_HIP;
  return hip_status(launch_cost(t, w, cost, err, stream));
}

size_t fs_throttle_workspace(const fs_trace *t) {
  if (check_trace(t, false) != FS_OK || !throttle_shape_ok(t)) return 0;
  return throttle_workspace_bytes(t);
}

fs_status fs_throttle(const fs_trace *t, const fs_limits *lim, const uint8_t *overloaded,
                      uint32_t flags, uint32_t *bitmap, uint8_t *reason, int32_t *cnt_user,
                      int32_t *cnt_app, void *ws, size_t ws_bytes, int32_t *err,
                      hipStream_t stream) {
  fs_status s = check_trace(t, false);
  if (s == FS_OK) s = check_limits(t, lim);
  if (s != FS_OK) return s;
  if ((flags & ~FS_THROTTLE_RAW) || !per_request(t, bitmap) || !err || !throttle_shape_ok(t))
    return FS_E_ARG;
  if (!ws || !aligned(ws) || ws_bytes < throttle_workspace_bytes(t)) return FS_E_WORKSPACE;
  if (launch_zero_i32(err, stream) != hipSuccess) return FS_E_HIP;
  return hip_status(launch_throttle(t, lim, overloaded, flags, bitmap, reason, cnt_user, cnt_app,
                                    ws, err, stream));
}

size_t fs_state_bytes(const fs_trace *t) {
  if (check_trace(t, false) != FS_OK) return 0;
  return state_bytes(t);
}

fs_status fs_state_init(void *state, size_t bytes, const fs_trace *t, hipStream_t stream) {
  fs_status s = check_trace(t, false);
  if (s != FS_OK) return s;
  if (!state || !aligned(state) || bytes < state_bytes(t)) return FS_E_WORKSPACE;
  return hip_status(launch_state_init(state, t, stream));
}

fs_status fs_schedule_step(void *state, const fs_trace *t, const int64_t *cost,
                           const uint8_t *exceed_reason, const fs_engine *eng, fs_outputs *out,
                           int64_t n_steps, hipStream_t stream) {
  fs_status s = check_trace(t, true);
  if (s == FS_OK) s = check_engine(eng);
  if (s == FS_OK) s = check_outputs(t, out);
  if (s != FS_OK) return s;
  if (!state || !aligned(state) || !per_request(t, cost)) return FS_E_ARG;
  if (launch_zero_i32(out->err, stream) != hipSuccess) return FS_E_HIP;
  return hip_status(launch_schedule(state, t, cost, exceed_reason, eng, out, n_steps, stream));
}

size_t fs_run_trace_workspace(const fs_trace *t) {
  if (check_trace(t, false) != FS_OK || !throttle_shape_ok(t)) return 0;
  int64_t N = n_records(t);
  size_t b = round_up(size_t(N) * sizeof(int64_t));   // cost
  b += round_up(size_t(N));                           // raw reasons
  b += round_up(size_t((N + 31) / 32) * 4);           // exceed bitmap
  b += round_up(throttle_workspace_bytes(t));
  b += round_up(state_bytes(t));
  return b;
}

fs_status fs_run_trace(const fs_trace *t, const fs_weights *w, const fs_limits *lim,
                       const fs_engine *eng, fs_outputs *out, void *ws, size_t ws_bytes,
                       hipStream_t stream) {
  fs_status s = check_trace(t, true);
  if (s == FS_OK) s = check_weights(t, w);
  if (s == FS_OK) s = check_limits(t, lim);
  if (s == FS_OK) s = check_engine(eng);
  if (s == FS_OK) s = check_outputs(t, out);
  if (s != FS_OK) return s;
  if (!throttle_shape_ok(t)) return FS_E_ARG;
  if (!ws || !aligned(ws) || ws_bytes < fs_run_trace_workspace(t)) return FS_E_WORKSPACE;
  int64_t N = n_records(t);
  char *p = static_cast<char *>(ws);
  int64_t *cost = reinterpret_cast<int64_t *>(p);
  p += round_up(size_t(N) * sizeof(int64_t));
  uint8_t *reason = reinterpret_cast<uint8_t *>(p);
  p += round_up(size_t(N));
  uint32_t *bitmap = reinterpret_cast<uint32_t *>(p);
  p += round_up(size_t((N + 31) / 32) * 4);
  void *tws = p;
  p += round_up(throttle_workspace_bytes(t));
  void *state = p;
  if (launch_zero_i32(out->err, stream) != hipSuccess) return FS_E_HIP;
  hipError_t e = launch_cost(t, w, cost, out->err, stream);
  if (e == hipSuccess)
    e = launch_throttle(t, lim, nullptr, FS_THROTTLE_RAW, bitmap, reason, nullptr, nullptr, tws,
                        out->err, stream);
  if (e == hipSuccess) e = launch_state_init(state, t, stream);
  if (e == hipSuccess) e = launch_schedule(state, t, cost, reason, eng, out, -1, stream);
  return hip_status(e);
}

size_t fs_metrics_workspace(const fs_trace *t) {
  if (check_trace(t, false) != FS_OK) return 0;
  return metrics_workspace_bytes(t);
}

fs_status fs_fairness_metrics(const fs_trace *t, const int64_t *cost, const fs_outputs *out,
                              const fs_engine *eng, int32_t delay_steps, fs_metrics *m, void *ws,
                              size_t ws_bytes, hipStream_t stream) {
  fs_status s = check_trace(t, true);
  if (s == FS_OK) s = check_engine(eng);
  if (s != FS_OK) return s;
  if (!per_request(t, cost) || !out || !per_request(t, out->status) ||
      !per_request(t, out->admit_step) || !out->max_gap || !out->err || !m || delay_steps < 0)
    return FS_E_ARG;
  if (!m->jain || !m->max_gap_tokens || !m->svc_req_pct || !m->svc_int_pct ||
      !m->served_users_pct || !m->delayed_users_pct || !m->throttled || !m->aborted_midway ||
      !m->wasted_tokens)
    return FS_E_ARG;
  if (!ws || !aligned(ws) || ws_bytes < metrics_workspace_bytes(t)) return FS_E_WORKSPACE;
  if (launch_zero_i32(out->err, stream) != hipSuccess) return FS_E_HIP;
  return hip_status(launch_metrics(t, cost, out, eng, delay_steps, m, ws, stream));
}

size_t fs_workload_workspace(const fs_trace *t) {
  if (check_trace(t, false) != FS_OK) return 0;
  return workload_workspace_bytes(t);
}

fs_status fs_workload_stats(const fs_trace *t, int64_t minute_us, const fs_wstats *out, void *ws,
                            size_t ws_bytes, int32_t *err, hipStream_t stream) {
  fs_status s = check_trace(t, true);
  if (s != FS_OK) return s;
  if (minute_us <= 0 || !out || !err || !out->minutes || !out->user_req || !out->user_tok ||
      !out->rate_hist || !out->len_hist || !out->len_sum || !out->size_hist || !out->graph)
    return FS_E_ARG;
  if (!ws || !aligned(ws) || ws_bytes < workload_workspace_bytes(t)) return FS_E_WORKSPACE;
  if (launch_zero_i32(err, stream) != hipSuccess) return FS_E_HIP;
  return hip_status(launch_workload(t, minute_us, out, ws, err, stream));
}

size_t fs_metrics_noalloc_limit(void) { return kScratchBytes; }

fs_status fs_fairness_metrics_noalloc(const fs_trace *t, const int64_t *cost,
                                      const fs_outputs *out, const fs_engine *eng,
                                      int32_t delay_steps, fs_metrics *m, hipStream_t stream) {
  fs_status s = check_trace(t, true);
  if (s == FS_OK) s = check_engine(eng);
  if (s != FS_OK) return s;
  if (!per_request(t, cost) || !out || !per_request(t, out->status) ||
      !per_request(t, out->admit_step) || !out->max_gap || !out->err || !m || delay_steps < 0)
    return FS_E_ARG;
  if (!m->jain || !m->max_gap_tokens || !m->svc_req_pct || !m->svc_int_pct ||
      !m->served_users_pct || !m->delayed_users_pct || !m->throttled || !m->aborted_midway ||
      !m->wasted_tokens)
    return FS_E_ARG;
  if (metrics_workspace_bytes(t) > kScratchBytes) return FS_E_WORKSPACE;
  void *ws = nullptr;
  s = scratch_on_current_device(&ws);
  if (s != FS_OK) return s;
  if (launch_zero_i32(out->err, stream) != hipSuccess) return FS_E_HIP;
  // the first kernel clears every part of the workspace the others accumulate into
  return hip_status(launch_metrics(t, cost, out, eng, delay_steps, m, ws, stream));
}

}  // extern "C"

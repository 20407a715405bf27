// Host-side launchers of the libfairserve kernels (internal).
#pragma once
#include <hip/hip_runtime.h>

#include "../../include/fairserve.h"

namespace fs {

hipError_t launch_cost(const fs_trace *t, const fs_weights *w, int64_t *cost, int32_t *err,
                       hipStream_t stream);

size_t throttle_workspace_bytes(const fs_trace *t);
bool throttle_shape_ok(const fs_trace *t);
hipError_t launch_throttle(const fs_trace *t, const fs_limits *lim, const uint8_t *overloaded,
                           uint32_t flags, uint32_t *bitmap, uint8_t *reason, int32_t *cnt_user,
                           int32_t *cnt_app, void *ws, int32_t *err, hipStream_t stream);

size_t state_bytes(const fs_trace *t);
hipError_t launch_state_init(void *state, const fs_trace *t, hipStream_t stream);
hipError_t launch_schedule(void *state, const fs_trace *t, const int64_t *cost,
                           const uint8_t *reason, const fs_engine *eng, fs_outputs *out,
                           int64_t n_steps, hipStream_t stream);

hipError_t launch_metrics(const fs_trace *t, const int64_t *cost, const fs_outputs *out,
                          const fs_engine *eng, int32_t delay_steps, fs_metrics *m, void *ws,
                          hipStream_t stream);
size_t metrics_workspace_bytes(const fs_trace *t);

size_t history_workspace_bytes(const fs_trace *t, int32_t n_stages);
hipError_t launch_history(const fs_trace *t, int32_t n_stages, int64_t K, int32_t base_limit,
                          int64_t *stats, int64_t *coef, int32_t *t_app, void *ws, int32_t *err,
                          hipStream_t stream);
int64_t history_max_records();

size_t workload_workspace_bytes(const fs_trace *t);
hipError_t launch_workload(const fs_trace *t, int64_t minute_us, const fs_wstats *out, void *ws,
                           int32_t *err, hipStream_t stream);

hipError_t launch_zero_i32(int32_t *p, hipStream_t stream);

// Device-wide exclusive prefix sum of n uint32 values in place; `part` needs
// scan_partials_bytes(n) bytes of scratch.
size_t scan_partials_bytes(int64_t n);
hipError_t exclusive_scan(uint32_t *data, int64_t n, uint32_t *part, hipStream_t stream);

}  // namespace fs

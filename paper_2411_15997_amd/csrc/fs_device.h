// Internal device-side definitions shared by the libfairserve kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/fairserve.h"

namespace fs {

constexpr int64_t kLenLimit = int64_t(1) << 24;    // token counts are in [0, 2^24)
constexpr int64_t kCoefLimit = int64_t(1) << 36;   // Q16 coefficients are in [0, 2^36)
constexpr int64_t kPrioLimit = int64_t(1) << 16;   // Q8 priorities are in [0, 2^16)
constexpr int64_t kValueLimit = int64_t(1) << 62;  // costs and counters stay below 2^62
constexpr int64_t kCapLimit = int64_t(1) << 40;    // engine capacity per step
constexpr int kMaxApps = 1024;

// Plain-pointer view of fs_trace passed to kernels by value.
struct DevTrace {
  int32_t R, U, A;
  const int64_t *rep_off;
  const int64_t *ts;
  const int32_t *user, *app, *call, *head, *prev;
  const int32_t *len_in, *len_sys, *len_out;
  int64_t N;
};

inline DevTrace dev_trace(const fs_trace *t) {
  DevTrace d;
  d.R = t->n_replicas;
  d.U = t->n_users;
  d.A = t->n_apps;
  d.rep_off = t->rep_off;
  d.ts = t->ts_us;
  d.user = t->user;
  d.app = t->app;
  d.call = t->call;
  d.head = t->head;
  d.prev = t->prev;
  d.len_in = t->len_in;
  d.len_sys = t->len_sys;
  d.len_out = t->len_out;
  d.N = t->rep_off_h[t->n_replicas];
  return d;
}

// Records the largest error code seen (deterministic under any interleaving).
__device__ inline void raise_err(int32_t *err, int32_t code) {
  if (code) atomicMax(err, code);
}

// Replica containing global record g: last r with rep_off[r] <= g (and g < rep_off[R]).
__device__ inline int32_t replica_of(const int64_t *rep_off, int32_t R, int64_t g) {
  int32_t lo = 0, hi = R - 1;
  while (lo < hi) {
    int32_t mid = (lo + hi + 1) >> 1;
    if (__ldg(rep_off + mid) <= g)
      lo = mid;
    else
      hi = mid - 1;
  }
  return lo;
}

__device__ inline int64_t tokens_of(const DevTrace &t, int64_t g) {
  int64_t v = int64_t(t.len_in[g]) + int64_t(t.len_out[g]);
  if (t.len_sys) v += t.len_sys[g];
  return v;
}

__device__ inline bool len_ok(int32_t x) { return x >= 0 && int64_t(x) < kLenLimit; }

// Wave-level helpers (wavefront = 64 lanes on gfx950).
__device__ inline int lane_id() { return __lane_id(); }

template <class T>
__device__ inline T wave_bcast(T v, int src_lane) {
  return __shfl(v, src_lane, 64);
}

}  // namespace fs

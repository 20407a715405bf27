// Scheduler state blob, kernel arguments and wavefront helpers shared by the two
// scheduler kernels (on-chip: fs_sched_onchip.hip; global memory: fs_sched.hip).
//
// The state blob (fs_state_bytes) is what lets fs_schedule_step stop after n steps
// and resume later, and what lets the on-chip kernel hand a replica over to the
// global-memory kernel when an on-chip capacity would overflow.  It holds the
// per-replica scalars, the service counters of every user and the fate of every
// request; the waiting queue itself is rebuilt on resume from the requests that
// have arrived and are still undecided, in stream order.
#pragma once
#include "fs_device.h"
#include "fs_launch.h"

namespace fs {
namespace sched {

constexpr uint64_t kMagic = 0x32535652'49414646ull;
constexpr int32_t kVersion = 5;
constexpr uint64_t kTierShift = 62;
constexpr uint64_t kValMask = (uint64_t(1) << 62) - 1;
constexpr uint64_t kEmptyKey = ~uint64_t(0);

// Per-replica scalars.  `mid` = 1 when a launch stopped inside the admissions of
// step s (an on-chip capacity would have overflowed there); `mid_budget` is the
// budget that step still has.  Literal engine: `n_run` calls are running (their
// records and finish steps in run_rec / run_fin, in admission order), holding
// `kv_used` tokens of KV cache.
struct RepState {
  int64_t s, nxt, debt, backlog, seq, gap, last_exit_u, low, s_end;
  int32_t last_exit, done, overflow, mid;
  int64_t mid_budget;
  int64_t kv_used, n_run;
  int64_t pad2[2];
};
static_assert(sizeof(RepState) == 128, "RepState layout");

struct Header {
  uint64_t magic;
  int32_t version, R, U, pad;
  int64_t N;
  int64_t pad2[4];
};

inline size_t up256(size_t x) { return (x + 255) / 256 * 256; }

struct StateLayout {
  size_t hdr, reps, u_all, xslot_all, fate, succ, seg_start, seg_part, seg_rec, seg_tok, seg_cost,
      seg_succ, seg_pk;
  // global-memory scheduler structures (n_r + 1 entries per replica, at rep_off[r] + r)
  size_t xkey, xuser, xq, xfh, xft, xhh, xht, xsb, xrh, xrdy;
  size_t e_all, e_free;
  size_t emap;  // per record: the pool entry it last occupied (checked before use)
  size_t run_rec, run_fin;  // literal engine: running calls (n_r + 1 per replica)
  size_t total;
};

inline StateLayout state_layout(int32_t R, int32_t U, int64_t N) {
  StateLayout L;
  size_t n = size_t(N > 0 ? N : 1), ru = size_t(R) * size_t(U);
  size_t nr = size_t(N) + size_t(R) + 1;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o += up256(bytes);
    return at;
  };
  L.hdr = take(sizeof(Header));
  L.reps = take(sizeof(RepState) * size_t(R));
  L.u_all = take(ru * 8);
  L.xslot_all = take(ru * 4);
  L.fate = take(n);
  L.succ = take(n * 4);
  L.seg_start = take((ru + 1) * 4);
  L.seg_part = take(scan_partials_bytes(int64_t(ru + 1)));
  L.seg_rec = take(n * 4);
  L.seg_tok = take(n * 4);
  L.seg_cost = take(n * 8);
  L.seg_succ = take(n * 4);
  L.seg_pk = take(n * 16);
  L.xkey = take(nr * 8);
  L.xuser = take(nr * 4);
  L.xq = take(nr * 4);
  L.xfh = take(nr * 4);
  L.xft = take(nr * 4);
  L.xhh = take(nr * 4);
  L.xht = take(nr * 4);
  L.xsb = take(nr * 4);
  L.xrh = take(nr * 4);
  L.xrdy = take(nr * 4);
  L.e_all = take(nr * 48);
  L.e_free = take(nr * 4);
  L.emap = take(n * 4);
  L.run_rec = take(nr * 4);
  L.run_fin = take(nr * 4);
  L.total = o;
  return L;
}

// LDS layout of the on-chip kernel (sizes chosen on the host from the replica
// count, so that enough work-groups fit on a CU).
struct OnchipCfg {
  int32_t ring;       // first calls kept on chip per backlogged user (power of two)
  int32_t cache;      // recent arrivals whose data stays on chip (power of two)
  int32_t users_lds;  // 1: counters of idle users in LDS, 0: in the state buffer
  int32_t batch;      // literal engine: running calls kept on chip (power of two), else 0
  int32_t user_tab;   // entries (power of two) of the per-user tables for a batch of arrivals
  int32_t glds;       // global-memory kernel: 1 = its user table and counters in LDS
  int32_t hblk;       // global-memory kernel: block minima of X kept in LDS (0: none)
  int32_t inl_glds;   // the same two, for the global-memory pass that an on-chip
  int32_t inl_hblk;   // instance continues with, within its own LDS allocation
  size_t lds_bytes;
};

struct SchedArgs {
  DevTrace t;
  const int64_t *cost;
  const uint8_t *reason;
  int64_t tau, cap, theta;
  int64_t n_steps;
  bool global_only;
  bool fcfs;   // first come, first served (FS_ENGINE_FCFS)
  bool blind;  // interaction-blind limits (FS_ENGINE_BLIND)
  bool literal;  // the literal engine (FS_ENGINE_LITERAL): charge at finish, KV capacity
  int8_t *status;
  int32_t *admit_step, *admit_seq;
  int64_t *counter_after, *counter_on_arrival, *counter, *steps, *decisions, *max_gap;
  int32_t *err;
  char *state;
  StateLayout L;
  OnchipCfg oc;
};

// A condition that is rarely true (laid out off the straight-line path).
#define FS_RARE(x) __builtin_expect(!!(x), 0)

// ------------------------------------------------------------- wave helpers

__device__ inline int32_t rdl(int32_t v, int l) { return __builtin_amdgcn_readlane(v, l); }
__device__ inline uint32_t rdlu(uint32_t v, int l) {
  return uint32_t(__builtin_amdgcn_readlane(int32_t(v), l));
}
__device__ inline int64_t rdl64(int64_t v, int l) {
  uint32_t lo = __builtin_amdgcn_readlane(uint32_t(uint64_t(v)), l);
  uint32_t hi = __builtin_amdgcn_readlane(uint32_t(uint64_t(v) >> 32), l);
  return int64_t((uint64_t(hi) << 32) | lo);
}
__device__ inline int32_t uni(int32_t v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ inline int64_t uni64(int64_t v) { return rdl64(v, 0); }

// Every structure of a replica is read and written by that replica's single wave,
// so work-group scope is enough for a load to see the wave's own earlier stores.
template <class T>
__device__ inline T ld_fresh(const T *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ inline void wave_fence() { __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront"); }

// DPP moves for a full-wave reduction (result in lane 63): swap within pairs, swap
// pairs, mirror within 8, mirror within 16, then broadcast row ends to later rows.
template <int CTRL, int ROWS>
__device__ inline uint32_t dpp(uint32_t v) {
  return uint32_t(__builtin_amdgcn_update_dpp(int(v), int(v), CTRL, ROWS, 0xF, false));
}

template <int CTRL, int ROWS>
__device__ inline void argmin_step(uint64_t &k, uint32_t &us, uint32_t &x) {
  const uint32_t lo = dpp<CTRL, ROWS>(uint32_t(k)), hi = dpp<CTRL, ROWS>(uint32_t(k >> 32));
  const uint32_t ous = dpp<CTRL, ROWS>(us), ox = dpp<CTRL, ROWS>(x);
  const uint64_t ok = (uint64_t(hi) << 32) | lo;
  const bool take = ok < k || (ok == k && ous < us);
  k = take ? ok : k;
  us = take ? ous : us;
  x = take ? ox : x;
}

__device__ inline void wave_argmin(uint64_t &k, uint32_t &us, uint32_t &x) {
  argmin_step<0xB1, 0xF>(k, us, x);
  argmin_step<0x4E, 0xF>(k, us, x);
  argmin_step<0x141, 0xF>(k, us, x);
  argmin_step<0x140, 0xF>(k, us, x);
  argmin_step<0x142, 0xA>(k, us, x);
  argmin_step<0x143, 0xC>(k, us, x);
}

template <int CTRL, int ROWS>
__device__ inline void minmax_step(uint64_t &lo, uint64_t &hi) {
  const uint64_t a = (uint64_t(dpp<CTRL, ROWS>(uint32_t(lo >> 32))) << 32) |
                     dpp<CTRL, ROWS>(uint32_t(lo));
  const uint64_t b = (uint64_t(dpp<CTRL, ROWS>(uint32_t(hi >> 32))) << 32) |
                     dpp<CTRL, ROWS>(uint32_t(hi));
  lo = a < lo ? a : lo;
  hi = b > hi ? b : hi;
}

__device__ inline void wave_minmax(uint64_t &lo, uint64_t &hi) {
  minmax_step<0xB1, 0xF>(lo, hi);
  minmax_step<0x4E, 0xF>(lo, hi);
  minmax_step<0x141, 0xF>(lo, hi);
  minmax_step<0x140, 0xF>(lo, hi);
  minmax_step<0x142, 0xA>(lo, hi);
  minmax_step<0x143, 0xC>(lo, hi);
}

// 32-bit wave minimum / maximum, left in every lane.  Four DPP steps leave each
// 16-lane row's extreme in every lane of the row (with the identity as the DPP "old"
// value the compiler fuses each move into the min/max instruction); swapping halves
// and then rows (gfx950 permlane swaps) combines the four rows.
template <int CTRL>
__device__ inline uint32_t dpp_id(uint32_t id, uint32_t v) {
  return uint32_t(__builtin_amdgcn_update_dpp(int(id), int(v), CTRL, 0xF, 0xF, false));
}
__device__ inline uint32_t vmin(uint32_t a, uint32_t b) { return a < b ? a : b; }
__device__ inline uint32_t vmax(uint32_t a, uint32_t b) { return a > b ? a : b; }
__device__ inline uint32_t wave_min32v(uint32_t v) {
  v = vmin(v, dpp_id<0xB1>(~0u, v));
  v = vmin(v, dpp_id<0x4E>(~0u, v));
  v = vmin(v, dpp_id<0x141>(~0u, v));
  v = vmin(v, dpp_id<0x140>(~0u, v));
  const auto h = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  v = vmin(h[0], h[1]);
  const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return vmin(r[0], r[1]);
}
__device__ inline uint32_t wave_max32v(uint32_t v) {
  v = vmax(v, dpp_id<0xB1>(0u, v));
  v = vmax(v, dpp_id<0x4E>(0u, v));
  v = vmax(v, dpp_id<0x141>(0u, v));
  v = vmax(v, dpp_id<0x140>(0u, v));
  const auto h = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  v = vmax(h[0], h[1]);
  const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return vmax(r[0], r[1]);
}
// Both at once, the two chains interleaved step by step (each fills the other's wait
// states between dependent DPP moves).
__device__ inline void wave_minmax32v(uint32_t &mn, uint32_t &mx) {
  mn = vmin(mn, dpp_id<0xB1>(~0u, mn));
  mx = vmax(mx, dpp_id<0xB1>(0u, mx));
  mn = vmin(mn, dpp_id<0x4E>(~0u, mn));
  mx = vmax(mx, dpp_id<0x4E>(0u, mx));
  mn = vmin(mn, dpp_id<0x141>(~0u, mn));
  mx = vmax(mx, dpp_id<0x141>(0u, mx));
  mn = vmin(mn, dpp_id<0x140>(~0u, mn));
  mx = vmax(mx, dpp_id<0x140>(0u, mx));
  const auto h = __builtin_amdgcn_permlane32_swap(mn, mn, false, false);
  const auto g = __builtin_amdgcn_permlane32_swap(mx, mx, false, false);
  mn = vmin(h[0], h[1]);
  mx = vmax(g[0], g[1]);
  const auto r = __builtin_amdgcn_permlane16_swap(mn, mn, false, false);
  const auto q = __builtin_amdgcn_permlane16_swap(mx, mx, false, false);
  mn = vmin(r[0], r[1]);
  mx = vmax(q[0], q[1]);
}
// The same, returned in a scalar register.
__device__ inline uint32_t wave_min32(uint32_t v) { return uint32_t(uni(int32_t(wave_min32v(v)))); }
__device__ inline uint32_t wave_max32(uint32_t v) { return uint32_t(uni(int32_t(wave_max32v(v)))); }

// Wave sum of 32-bit values, returned in a scalar register.
__device__ inline uint32_t wave_sum32(uint32_t v) {
  v += dpp_id<0xB1>(0u, v);
  v += dpp_id<0x4E>(0u, v);
  v += dpp_id<0x141>(0u, v);
  v += dpp_id<0x140>(0u, v);
  return rdlu(v, 15) + rdlu(v, 31) + rdlu(v, 47) + rdlu(v, 63);
}

// Inclusive prefix sum over the wave (lane order): shifts of 1, 2, 4 and 8 within
// each 16-lane row, then each row's total is carried into the rows after it.
template <int CTRL, int ROWS>
__device__ inline uint32_t dpp0(uint32_t v) {
  return uint32_t(__builtin_amdgcn_update_dpp(0, int(v), CTRL, ROWS, 0xF, false));
}
__device__ inline uint32_t wave_incl_scan32(uint32_t v) {
  v += dpp0<0x111, 0xF>(v);
  v += dpp0<0x112, 0xF>(v);
  v += dpp0<0x114, 0xF>(v);
  v += dpp0<0x118, 0xF>(v);
  v += dpp0<0x142, 0xA>(v);
  v += dpp0<0x143, 0xC>(v);
  return v;
}

__device__ inline bool state_header_ok(const SchedArgs &a) {
  const Header *h = reinterpret_cast<const Header *>(a.state + a.L.hdr);
  return h->magic == kMagic && h->version == kVersion && h->R == a.t.R && h->U == a.t.U &&
         h->N == a.t.N;
}

// A replica already drained by an earlier call: republish its results.
__device__ inline bool finish_if_done(const SchedArgs &a, int32_t r) {
  RepState *rs = reinterpret_cast<RepState *>(a.state + a.L.reps) + r;
  if (!rs->done) return false;
  if (threadIdx.x == 0) {
    a.steps[r] = rs->s;
    a.decisions[r] = rs->seq;
    a.max_gap[r] = rs->gap;
  }
  const int64_t *u_all =
      reinterpret_cast<const int64_t *>(a.state + a.L.u_all) + int64_t(r) * a.t.U;
  for (int32_t k = threadIdx.x; k < a.t.U; k += 64) a.counter[int64_t(r) * a.t.U + k] = u_all[k];
  return true;
}

// Host side: the on-chip kernel's LDS layout for this launch and its launcher.
OnchipCfg onchip_config(int32_t R, int32_t U, bool literal);
void launch_onchip(const SchedArgs &a, hipStream_t s);

}  // namespace sched
}  // namespace fs

// WSC scheduler steps (Alg. 1, monitoring and execution streams) under the
// token-budget step engine, one wavefront per trace replica.
//
// Per replica the state is the paper's: service counters u_i, the waiting queue Q
// (a dictionary from user to queued requests), the last user to leave Q, and the
// overload measure (tokens queued).  The wave keeps the hot part on chip:
//   X table   compact slots [0, nX) of users with something queued: user id, a key
//             (tier << 62 | u) whose tier is 0 while the user has a ready later call of
//             an incomplete interaction, its first-call FIFO (pool entries) and counts.
//             The argmin over (key, user id) is a lane-parallel scan plus a wave
//             reduction: tier 0 first, then least counter, then lowest user id.
//   pool      queued requests (record, cost, tokens, next call, FIFO link).
//   CL        queued later calls: ready (previous call admitted) or pending.
//   window    the next 64 records in registers (one per lane) with the user's slot,
//             idle counter, "previous call admitted" and "first call throttled" flags
//             prefetched; every state change patches the lanes it affects, so the
//             arrival loop never waits on memory.
// Counters of idle users live in LDS when they fit, else in the state buffer.  If
// an on-chip capacity overflows, the wave saves its state and the same code resumes
// with every structure in global memory (second launch, same stream).
#include "fs_device.h"
#include "fs_launch.h"

namespace fs {
namespace {

constexpr uint64_t kMagic = 0x31535652'49414646ull;  // "FFAIRVS1"
constexpr int32_t kVersion = 1;
constexpr uint64_t kTierShift = 62;
constexpr uint64_t kValMask = (uint64_t(1) << 62) - 1;
constexpr uint64_t kEmptyKey = ~uint64_t(0);
constexpr int kUsersLdsMax = 1024;   // per-user arrays on chip up to this many users
constexpr int kXCap = 128;            // on-chip backlogged-user slots
constexpr int kCLCap = 256;           // on-chip queued later calls

struct RepState {
  int64_t s, nxt, debt, backlog, seq, gap, last_exit_u, nq, s_end;
  int32_t last_exit, done, overflow, pad;
  int64_t pad2[5];
};
static_assert(sizeof(RepState) == 128, "RepState layout");

struct Header {
  uint64_t magic;
  int32_t version, R, U, pad;
  int64_t N;
  int64_t pad2[4];
};

size_t up(size_t x) { return (x + 255) / 256 * 256; }

struct StateLayout {
  size_t hdr, reps, u_all, xslot_all, fate, succ, qsave;
  // global-mode scratch (capacity n_r per replica, offset rep_off[r])
  size_t xkey, xuser, xq, xfh, xft, xrdy, p_cost, p_rec, p_tok, p_succ, p_next, p_free, cl_rec,
      cl_prev, cl_user, cl_e, cl_rdy;
  size_t total;
};

StateLayout state_layout(int32_t R, int32_t U, int64_t N) {
  StateLayout L;
  size_t n = size_t(N > 0 ? N : 1), ru = size_t(R) * size_t(U);
  size_t nr = size_t(N) + size_t(R) + 1;  // global-mode scratch: n_r + 1 entries per replica
  size_t o = 0;
  L.hdr = o; o += up(sizeof(Header));
  L.reps = o; o += up(sizeof(RepState) * size_t(R));
  L.u_all = o; o += up(ru * 8);
  L.xslot_all = o; o += up(ru * 4);
  L.fate = o; o += up(n);
  L.succ = o; o += up(n * 4);
  L.qsave = o; o += up(n * 4);
  L.xkey = o; o += up(nr * 8);
  L.xuser = o; o += up(nr * 4);
  L.xq = o; o += up(nr * 4);
  L.xfh = o; o += up(nr * 4);
  L.xft = o; o += up(nr * 4);
  L.xrdy = o; o += up(nr * 4);
  L.p_cost = o; o += up(nr * 8);
  L.p_rec = o; o += up(nr * 4);
  L.p_tok = o; o += up(nr * 4);
  L.p_succ = o; o += up(nr * 4);
  L.p_next = o; o += up(nr * 4);
  L.p_free = o; o += up(nr * 4);
  L.cl_rec = o; o += up(nr * 4);
  L.cl_prev = o; o += up(nr * 4);
  L.cl_user = o; o += up(nr * 4);
  L.cl_e = o; o += up(nr * 4);
  L.cl_rdy = o; o += up(nr * 4);
  L.total = o;
  return L;
}

struct SchedArgs {
  DevTrace t;
  const int64_t *cost;
  const uint8_t *reason;
  int64_t tau, cap, theta;
  int64_t n_steps;
  bool global_only;
  // outputs
  int8_t *status;
  int32_t *admit_step, *admit_seq;
  int64_t *counter_after, *counter_on_arrival, *counter, *steps, *decisions, *max_gap;
  int32_t *err;
  // state
  char *state;
  StateLayout L;
  int32_t pcap;   // on-chip pool entries
};

// -------------------------------------------------------------- small wave helpers

__device__ inline int32_t rdl(int32_t v, int l) { return __builtin_amdgcn_readlane(v, l); }
__device__ inline int64_t rdl64(int64_t v, int l) {
  uint32_t lo = __builtin_amdgcn_readlane(uint32_t(uint64_t(v)), l);
  uint32_t hi = __builtin_amdgcn_readlane(uint32_t(uint64_t(v) >> 32), l);
  return int64_t((uint64_t(hi) << 32) | lo);
}
__device__ inline int32_t uni(int32_t v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ inline int64_t uni64(int64_t v) { return rdl64(v, 0); }

__device__ inline uint64_t shfl_xor64(uint64_t v, int m) {
  uint32_t lo = __shfl_xor(uint32_t(v), m, 64);
  uint32_t hi = __shfl_xor(uint32_t(v >> 32), m, 64);
  return (uint64_t(hi) << 32) | lo;
}

template <class T>
__device__ inline T ld_fresh(const T *p) {  // global load that sees this wave's own stores
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Reads of the scheduler structures: plain for LDS, coherent for global memory.
template <bool G, class T>
__device__ inline T RD(const T *p) {
  if constexpr (G)
    return ld_fresh(p);
  else
    return *p;
}

// Storage of the scheduler structures: LDS (on chip) or the state buffer (global).
struct Store {
  // per-user (for the replica)
  int64_t *u;
  int32_t *xslot;
  // X table
  uint64_t *xkey;
  int32_t *xuser, *xq, *xfh, *xft, *xrdy;
  // pool of queued requests
  int64_t *p_cost;
  int32_t *p_rec, *p_tok, *p_succ, *p_next, *p_free;
  // queued later calls
  int32_t *cl_rec, *cl_prev, *cl_user, *cl_e, *cl_rdy;
  int32_t xcap, pcap, clcap;
  bool users_global;  // u / xslot in global memory (coherent loads needed)
};

// ---------------------------------------------------------------------------
// The scheduler body.  All control flow is wave-uniform; per-record work of the
// arrival window is held one record per lane.
// ---------------------------------------------------------------------------
template <bool G>
__device__ void run_replica(const SchedArgs &a, Store &S, int32_t r, bool onchip) {
  const int lane = threadIdx.x;
  const DevTrace &t = a.t;
  const int64_t base = t.rep_off[r];
  const int64_t n = t.rep_off[r + 1] - base;
  const int32_t U = t.U;
  RepState *rs = reinterpret_cast<RepState *>(a.state + a.L.reps) + r;
  int8_t *fate = reinterpret_cast<int8_t *>(a.state + a.L.fate) + base;
  const int32_t *succ = reinterpret_cast<const int32_t *>(a.state + a.L.succ) + base;
  int32_t *qsave = reinterpret_cast<int32_t *>(a.state + a.L.qsave) + base;
  int64_t *u_all = reinterpret_cast<int64_t *>(a.state + a.L.u_all) + int64_t(r) * U;

  // ---- scalar state
  int64_t s = uni64(rs->s), nxt = uni64(rs->nxt), debt = uni64(rs->debt);
  int64_t backlog = uni64(rs->backlog), seq = uni64(rs->seq), gap = uni64(rs->gap);
  int64_t last_exit_u = uni64(rs->last_exit_u), nq = uni64(rs->nq);
  int32_t last_exit = uni(rs->last_exit);
  int64_t s_end;
  if (onchip || !rs->overflow) {
    s_end = a.n_steps < 0 ? INT64_MAX : s + a.n_steps;
  } else {
    s_end = uni64(rs->s_end);  // resuming a launch that overflowed on chip
  }
  const int64_t tau = a.tau, C = a.cap, theta = a.theta;

  // ---- per-user arrays
  if (!S.users_global) {
    for (int32_t k = lane; k < U; k += 64) {
      S.u[k] = u_all[k];
      S.xslot[k] = -1;
    }
  }
  // pool free stack
  for (int32_t e = lane; e < S.pcap; e += 64) S.p_free[e] = S.pcap - 1 - e;
  int32_t nfree = S.pcap, nX = 0, ncl = 0;
  int32_t code = 0;
  bool overflow = false;
  __syncthreads();

  auto get_u = [&](int32_t k) -> int64_t {
    return S.users_global ? ld_fresh(S.u + k) : S.u[k];
  };
  auto get_xslot = [&](int32_t k) -> int32_t {
    return S.users_global ? ld_fresh(S.xslot + k) : S.xslot[k];
  };
  auto key_of = [&](int32_t x, int64_t uval) -> uint64_t {
    return (uint64_t(RD<G>(&S.xrdy[x]) > 0 ? 0 : 1) << kTierShift) | uint64_t(uval);
  };

  // ---- window of upcoming records (one per lane)
  int64_t wbase = nxt;
  int64_t w_ts = 0, w_cost = 0, c_u = 0;
  int32_t w_user = 0, w_call = 0, w_head = 0, w_prev = -1, w_succ = -1, w_tok = 0, w_reason = 0;
  int32_t c_xslot = -1, c_prev_adm = 0, c_head_blk = 0;
  auto load_window = [&]() {
    __threadfence();
    int64_t i = wbase + lane;
    if (i < n) {
      int64_t g = base + i;
      w_ts = t.ts[g];
      w_user = t.user[g];
      w_call = t.call ? t.call[g] : 0;
      w_head = t.call ? t.head[g] : int32_t(i);
      w_prev = t.call ? t.prev[g] : -1;
      w_succ = succ[i];
      w_tok = t.len_in[g] + t.len_out[g] + (t.len_sys ? t.len_sys[g] : 0);
      w_cost = a.cost[g];
      w_reason = a.reason ? a.reason[g] : 0;
      c_xslot = get_xslot(w_user);
      c_u = get_u(w_user);
      c_prev_adm = (w_call > 0) ? (ld_fresh(fate + w_prev) == 0) : 0;
      int8_t hf = (w_call > 0) ? ld_fresh(fate + w_head) : int8_t(-1);
      c_head_blk = (hf == 1 || hf == 2) ? 1 : 0;
    } else {
      w_user = -1;
      w_call = 0;
      w_head = -1;
      w_prev = -1;
    }
  };

  // ---- structure operations (wave-uniform arguments)
  auto fifo_push = [&](int32_t x, int32_t e) {
    if (lane == 0) {
      S.p_next[e] = -1;
      int32_t tl = RD<G>(&S.xft[x]);
      if (tl < 0) S.xfh[x] = e; else S.p_next[tl] = e;
      S.xft[x] = e;
    }
  };
  auto join_x = [&](int32_t k, int64_t uval) -> int32_t {
    int32_t x = nX++;
    if (lane == 0) {
      S.xuser[x] = k;
      S.xq[x] = 0;
      S.xfh[x] = -1;
      S.xft[x] = -1;
      S.xrdy[x] = 0;
      S.xkey[x] = (uint64_t(1) << kTierShift) | uint64_t(uval);
      S.xslot[k] = x;
    }
    if (w_user == k) c_xslot = x;
    return x;
  };
  // Remove slot x (its user leaves Q with counter uval): swap the last slot into x.
  auto leave_x = [&](int32_t x, int32_t k, int64_t uval) {
    int32_t last = nX - 1;
    if (lane == 0) {
      S.u[k] = uval;
      S.xslot[k] = -1;
    }
    if (w_user == k) {
      c_xslot = -1;
      c_u = uval;
    }
    if (x != last) {
      int32_t k2 = uni(RD<G>(&S.xuser[last]));
      if (lane == 0) {
        S.xuser[x] = k2;
        S.xq[x] = RD<G>(&S.xq[last]);
        S.xfh[x] = RD<G>(&S.xfh[last]);
        S.xft[x] = RD<G>(&S.xft[last]);
        S.xrdy[x] = RD<G>(&S.xrdy[last]);
        S.xkey[x] = RD<G>(&S.xkey[last]);
        S.xslot[k2] = x;
      }
      if (w_user == k2) c_xslot = x;
    }
    nX = last;
  };
  // argmin over X of (key, user id); returns slot
  auto argmin_x = [&](uint64_t &bk, int32_t &bu) -> int32_t {
    uint64_t k = kEmptyKey;
    int32_t us = INT32_MAX, bx = -1;
    for (int32_t x = lane; x < nX; x += 64) {
      uint64_t kk = RD<G>(&S.xkey[x]);
      int32_t uu = RD<G>(&S.xuser[x]);
      if (kk < k || (kk == k && uu < us)) {
        k = kk;
        us = uu;
        bx = x;
      }
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      uint64_t k2 = shfl_xor64(k, m);
      int32_t u2 = __shfl_xor(us, m, 64);
      int32_t x2 = __shfl_xor(bx, m, 64);
      if (k2 < k || (k2 == k && u2 < us)) {
        k = k2;
        us = u2;
        bx = x2;
      }
    }
    bk = uni64(int64_t(k));
    bu = uni(us);
    return uni(bx);
  };
  auto minmax_x = [&](int64_t &mn, int64_t &mx) {
    uint64_t lo = kEmptyKey, hi = 0;
    for (int32_t x = lane; x < nX; x += 64) {
      uint64_t v = RD<G>(&S.xkey[x]) & kValMask;
      lo = v < lo ? v : lo;
      hi = v > hi ? v : hi;
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      uint64_t l2 = shfl_xor64(lo, m), h2 = shfl_xor64(hi, m);
      lo = l2 < lo ? l2 : lo;
      hi = h2 > hi ? h2 : hi;
    }
    mn = uni64(int64_t(lo));
    mx = uni64(int64_t(hi));
  };
  // the user's lowest-index ready later call: CL position
  auto cl_ready_min = [&](int32_t k) -> int32_t {
    int32_t best = INT32_MAX, bc = -1;
    for (int32_t c = lane; c < ncl; c += 64) {
      const int32_t rec_c = RD<G>(&S.cl_rec[c]);
      if (RD<G>(&S.cl_rdy[c]) && RD<G>(&S.cl_user[c]) == k && rec_c < best) {
        best = rec_c;
        bc = c;
      }
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      int32_t b2 = __shfl_xor(best, m, 64), c2 = __shfl_xor(bc, m, 64);
      if (b2 < best) {
        best = b2;
        bc = c2;
      }
    }
    return uni(bc);
  };
  auto cl_find_pending = [&](int32_t prev_rec) -> int32_t {
    int32_t found = -1;
    for (int32_t c = lane; c < ncl; c += 64)
      if (!RD<G>(&S.cl_rdy[c]) && RD<G>(&S.cl_prev[c]) == prev_rec) found = c;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      int32_t f2 = __shfl_xor(found, m, 64);
      found = f2 > found ? f2 : found;
    }
    return uni(found);
  };
  auto cl_remove = [&](int32_t c) {
    int32_t last = ncl - 1;
    if (lane == 0 && c != last) {
      S.cl_rec[c] = RD<G>(&S.cl_rec[last]);
      S.cl_prev[c] = RD<G>(&S.cl_prev[last]);
      S.cl_user[c] = RD<G>(&S.cl_user[last]);
      S.cl_e[c] = RD<G>(&S.cl_e[last]);
      S.cl_rdy[c] = RD<G>(&S.cl_rdy[last]);
    }
    ncl = last;
  };
  auto cl_add = [&](int32_t rec, int32_t prev_rec, int32_t k, int32_t e, int32_t rdy) {
    int32_t c = ncl++;
    if (lane == 0) {
      S.cl_rec[c] = rec;
      S.cl_prev[c] = prev_rec;
      S.cl_user[c] = k;
      S.cl_e[c] = e;
      S.cl_rdy[c] = rdy;
    }
  };
  auto set_key = [&](int32_t x, int64_t uval) {
    if (lane == 0) S.xkey[x] = key_of(x, uval);
  };
  // Put one queued record (already counted in backlog) into the structures.
  // Returns false if an on-chip capacity would overflow (nothing changed then).
  auto enqueue = [&](int32_t rec, int32_t k, int32_t call, int32_t prev_rec, int32_t sc,
                     int32_t tok, int64_t cst, int32_t xs, int64_t uval, bool prev_adm) -> bool {
    if ((xs < 0 && nX >= S.xcap) || nfree == 0 || (call > 0 && ncl >= S.clcap)) return false;
    int32_t x = xs >= 0 ? xs : join_x(k, uval);
    int32_t e = uni(RD<G>(&S.p_free[--nfree]));
    if (lane == 0) {
      S.p_rec[e] = rec;
      S.p_cost[e] = cst;
      S.p_tok[e] = tok;
      S.p_succ[e] = sc;
      S.xq[x] = RD<G>(&S.xq[x]) + 1;
    }
    if (call == 0) {
      fifo_push(x, e);
    } else {
      cl_add(rec, prev_rec, k, e, prev_adm ? 1 : 0);
      if (prev_adm) {
        if (lane == 0) S.xrdy[x] = RD<G>(&S.xrdy[x]) + 1;
        set_key(x, uval);
      }
    }
    return true;
  };

  // ---- rebuild the queue saved by a previous call
  for (int64_t q = 0; q < nq && !overflow; ++q) {
    int32_t rec = uni(qsave[q]);
    int64_t g = base + rec;
    int32_t k = uni(t.user[g]);
    int32_t call = t.call ? uni(t.call[g]) : 0;
    int32_t prev_rec = t.call ? uni(t.prev[g]) : -1;
    int32_t tok = uni(t.len_in[g] + t.len_out[g] + (t.len_sys ? t.len_sys[g] : 0));
    int64_t cst = uni64(a.cost[g]);
    int32_t xs = uni(get_xslot(k));
    int64_t uval = xs >= 0 ? int64_t(uni64(int64_t(RD<G>(&S.xkey[xs]))) & int64_t(kValMask)) : uni64(get_u(k));
    bool prev_adm = call > 0 && ld_fresh(fate + prev_rec) == 0;
    if (!enqueue(rec, k, call, prev_rec, succ[rec], tok, cst, xs, uval, prev_adm)) overflow = true;
  }
  if (overflow) {
    // leave the saved state untouched for the global-memory pass
    for (int32_t x = 0; x < nX; ++x) {
      int32_t k = uni(RD<G>(&S.xuser[x]));
      if (lane == 0) S.xslot[k] = -1;
    }
    if (lane == 0) {
      rs->overflow = 1;
      rs->s_end = s_end;
    }
    return;
  }
  int64_t minX = 0;
  if (nX > 0) {
    int64_t mx;
    minmax_x(minX, mx);
  }
  load_window();

  // ---- steps
  while (!overflow && code == 0) {
    if (s >= s_end) break;
    if (nxt == n && nX == 0) break;
    if (nxt < n && nxt - wbase >= 64) {
      wbase = nxt;
      load_window();
    }
    if (nX == 0 && nxt < n) {
      // nothing queued: the steps before the next arrival only pay back debt
      int64_t target = rdl64(w_ts, int(nxt - wbase)) / tau;
      if (target > s_end) target = s_end;
      if (target > s) {
        int64_t k = target - s;
        debt = (k >= (-debt + C - 1) / C) ? 0 : debt + k * C;
        s = target;
        if (s >= s_end) break;
      }
    }
    if (s >= INT32_MAX) {
      code = FS_E_OVERFLOW;
      break;
    }

    // monitoring stream: arrivals of step s in stream order
    while (nxt < n) {
      if (nxt - wbase == 64) {
        wbase = nxt;
        load_window();
      }
      const int j = int(nxt - wbase);
      if (rdl64(w_ts, j) / tau > s) break;
      const int32_t rec = int32_t(nxt);
      const int32_t k = rdl(w_user, j);
      const int32_t call = rdl(w_call, j);
      const int32_t xs = rdl(c_xslot, j);
      const bool in_x = xs >= 0;
      int64_t uk = in_x ? int64_t(uni64(int64_t(RD<G>(&S.xkey[xs]))) & int64_t(kValMask)) : rdl64(c_u, j);
      const int64_t u_before = uk;
      if (!in_x) {  // counter lift for a user with nothing queued
        if (nX == 0) {
          if (last_exit >= 0) uk = uk > last_exit_u ? uk : last_exit_u;
        } else {
          uk = uk > minX ? uk : minX;
        }
      }
      bool blocked;
      int8_t why;
      if (call > 0) {
        blocked = rdl(c_head_blk, j) != 0;
        why = 3;
      } else {
        why = int8_t(rdl(w_reason, j));
        blocked = backlog > theta && why != 0;
      }
      const int32_t tok = rdl(w_tok, j);
      if (!blocked) {
        const bool prev_adm = rdl(c_prev_adm, j) != 0;
        if (!enqueue(rec, k, call, rdl(w_prev, j), rdl(w_succ, j), tok, rdl64(w_cost, j), xs, uk,
                     prev_adm)) {
          overflow = true;  // state is as before this arrival
          break;
        }
        if (!in_x && nX == 1) minX = uk;
        backlog += tok;
      } else {
        if (lane == 0) fate[rec] = why;
        if (!in_x && uk != u_before) {
          if (lane == 0) S.u[k] = uk;
          if (w_user == k) c_u = uk;
        }
        if (call == 0 && w_head == rec && w_call > 0) c_head_blk = 1;
        if (lane == 0) {
          int64_t g = base + rec;
          a.status[g] = why;
          a.admit_step[g] = -1;
          if (a.admit_seq) a.admit_seq[g] = -1;
          if (a.counter_after) a.counter_after[g] = -1;
        }
      }
      if (lane == 0 && a.counter_on_arrival) a.counter_on_arrival[base + rec] = uk;
      ++nxt;
    }
    if (overflow) break;

    // execution stream: admit while the step has budget
    int64_t budget = C + debt;
    while (budget > 0 && nX > 0) {
      uint64_t bk;
      int32_t k;
      const int32_t x = argmin_x(bk, k);
      const int64_t uk = int64_t(bk & kValMask);
      int32_t e;
      if (x < 0 || x >= nX) {
        code = FS_E_STATE;  // internal bookkeeping error: stop instead of reading out of bounds
        break;
      }
      if ((bk >> kTierShift) == 0) {
        const int32_t c = cl_ready_min(k);
        if (c < 0) {
          code = FS_E_STATE;
          break;
        }
        e = uni(RD<G>(&S.cl_e[c]));
        cl_remove(c);
        if (lane == 0) S.xrdy[x] = RD<G>(&S.xrdy[x]) - 1;
      } else {
        e = uni(RD<G>(&S.xfh[x]));
        if (e < 0 || e >= S.pcap) {
          code = FS_E_STATE;
          break;
        }
        const int32_t nx = uni(RD<G>(&S.p_next[e]));
        if (lane == 0) {
          S.xfh[x] = nx;
          if (nx < 0) S.xft[x] = -1;
        }
      }
      const int32_t rec = uni(RD<G>(&S.p_rec[e]));
      const int64_t cst = uni64(RD<G>(&S.p_cost[e]));
      const int32_t tok = uni(RD<G>(&S.p_tok[e]));
      const int32_t sc = uni(RD<G>(&S.p_succ[e]));
      const int32_t left = uni(RD<G>(&S.xq[x])) - 1;
      if (lane == 0) {
        S.p_free[nfree] = e;
        S.xq[x] = left;
      }
      ++nfree;
      budget -= tok;
      backlog -= tok;
      const int64_t unew = uk + cst;
      if (unew >= kValueLimit) {
        code = FS_E_OVERFLOW;
        break;
      }
      if (lane == 0) {
        int64_t g = base + rec;
        fate[rec] = 0;
        a.status[g] = 0;
        a.admit_step[g] = int32_t(s);
        if (a.admit_seq) a.admit_seq[g] = int32_t(seq);
        if (a.counter_after) a.counter_after[g] = unew;
      }
      ++seq;
      if (w_prev == rec) c_prev_adm = 1;
      if (sc >= 0 && sc < nxt) {
        // the next call arrived while this one was queued: it becomes ready now
        const int32_t c = cl_find_pending(rec);
        if (c >= 0) {
          if (lane == 0) {
            S.cl_rdy[c] = 1;
            S.xrdy[x] = RD<G>(&S.xrdy[x]) + 1;
          }
        }
      }
      if (left == 0) {
        last_exit = k;
        last_exit_u = unew;
        leave_x(x, k, unew);
      } else {
        set_key(x, unew);
      }
    }
    if (code) break;
    debt = budget < 0 ? budget : 0;
    if (nX > 0) {
      int64_t mn, mx;
      minmax_x(mn, mx);
      gap = mx - mn > gap ? mx - mn : gap;
      minX = mn;
    }
    ++s;
  }

  if (code) raise_err(a.err, code);

  // ---- save: counters of queued users back to u, queue contents to qsave
  int64_t q = 0;
  for (int32_t x = 0; x < nX; ++x) {
    const int32_t k = uni(RD<G>(&S.xuser[x]));
    const int64_t uval = int64_t(uni64(int64_t(RD<G>(&S.xkey[x]))) & int64_t(kValMask));
    if (lane == 0) {
      S.u[k] = uval;
      S.xslot[k] = -1;
    }
    int32_t walked = 0;
    for (int32_t e = uni(RD<G>(&S.xfh[x])); e >= 0 && e < S.pcap && walked < S.pcap;
         e = uni(RD<G>(&S.p_next[e])), ++walked) {
      if (lane == 0) qsave[q] = RD<G>(&S.p_rec[e]);
      ++q;
    }
  }
  for (int32_t c = 0; c < ncl; ++c) {
    if (lane == 0) qsave[q] = RD<G>(&S.cl_rec[c]);
    ++q;
  }
  __syncthreads();
  if (!S.users_global) {
    for (int32_t k = lane; k < U; k += 64) u_all[k] = S.u[k];
  }
  const bool drained = nxt == n && nX == 0;
  if (lane == 0) {
    rs->s = s;
    rs->nxt = nxt;
    rs->debt = debt;
    rs->backlog = backlog;
    rs->seq = seq;
    rs->gap = gap;
    rs->last_exit_u = last_exit_u;
    rs->nq = q;
    rs->last_exit = last_exit;
    rs->done = drained ? 1 : 0;
    rs->overflow = overflow ? 1 : 0;
    rs->s_end = s_end;
    if (!overflow) {
      a.steps[r] = s;
      a.decisions[r] = seq;
      a.max_gap[r] = gap;
    }
  }
  __threadfence();
  if (!overflow) {
    for (int32_t k = lane; k < U; k += 64)
      a.counter[int64_t(r) * U + k] = S.users_global ? ld_fresh(u_all + k) : u_all[k];
  }
}

__device__ inline bool state_header_ok(const SchedArgs &a) {
  const Header *h = reinterpret_cast<const Header *>(a.state + a.L.hdr);
  return h->magic == kMagic && h->version == kVersion && h->R == a.t.R && h->U == a.t.U &&
         h->N == a.t.N;
}

// On-chip pass: LDS holds the X table, pool, CL (and the counters when U is small).
template <bool USERS_LDS>
__global__ void __launch_bounds__(64) k_schedule_onchip(SchedArgs a) {
  extern __shared__ __align__(16) char smem[];
  const int32_t r = blockIdx.x;
  if (*a.err) return;
  if (!state_header_ok(a)) return;
  RepState *rs = reinterpret_cast<RepState *>(a.state + a.L.reps) + r;
  if (rs->done) {
    if (threadIdx.x == 0) {
      a.steps[r] = rs->s;
      a.decisions[r] = rs->seq;
      a.max_gap[r] = rs->gap;
    }
    const int64_t *u_all = reinterpret_cast<const int64_t *>(a.state + a.L.u_all) + int64_t(r) * a.t.U;
    for (int32_t k = threadIdx.x; k < a.t.U; k += 64) a.counter[int64_t(r) * a.t.U + k] = u_all[k];
    return;
  }
  Store S;
  char *p = smem;
  auto take = [&](size_t bytes) {
    char *q = p;
    p += (bytes + 15) & ~size_t(15);
    return q;
  };
  S.xcap = kXCap;
  S.pcap = a.pcap;
  S.clcap = kCLCap;
  S.xkey = reinterpret_cast<uint64_t *>(take(8 * kXCap));
  S.p_cost = reinterpret_cast<int64_t *>(take(8 * size_t(a.pcap)));
  S.xuser = reinterpret_cast<int32_t *>(take(4 * kXCap));
  S.xq = reinterpret_cast<int32_t *>(take(4 * kXCap));
  S.xfh = reinterpret_cast<int32_t *>(take(4 * kXCap));
  S.xft = reinterpret_cast<int32_t *>(take(4 * kXCap));
  S.xrdy = reinterpret_cast<int32_t *>(take(4 * kXCap));
  S.p_rec = reinterpret_cast<int32_t *>(take(4 * size_t(a.pcap)));
  S.p_tok = reinterpret_cast<int32_t *>(take(4 * size_t(a.pcap)));
  S.p_succ = reinterpret_cast<int32_t *>(take(4 * size_t(a.pcap)));
  S.p_next = reinterpret_cast<int32_t *>(take(4 * size_t(a.pcap)));
  S.p_free = reinterpret_cast<int32_t *>(take(4 * size_t(a.pcap)));
  S.cl_rec = reinterpret_cast<int32_t *>(take(4 * kCLCap));
  S.cl_prev = reinterpret_cast<int32_t *>(take(4 * kCLCap));
  S.cl_user = reinterpret_cast<int32_t *>(take(4 * kCLCap));
  S.cl_e = reinterpret_cast<int32_t *>(take(4 * kCLCap));
  S.cl_rdy = reinterpret_cast<int32_t *>(take(4 * kCLCap));
  if (USERS_LDS) {
    S.u = reinterpret_cast<int64_t *>(take(8 * size_t(a.t.U)));
    S.xslot = reinterpret_cast<int32_t *>(take(4 * size_t(a.t.U)));
    S.users_global = false;
  } else {
    S.u = reinterpret_cast<int64_t *>(a.state + a.L.u_all) + int64_t(r) * a.t.U;
    S.xslot = reinterpret_cast<int32_t *>(a.state + a.L.xslot_all) + int64_t(r) * a.t.U;
    S.users_global = true;
  }
  run_replica<false>(a, S, r, true);
}

// Global-memory pass: resumes replicas that overflowed on chip (or all replicas
// when the engine asks for global memory only).
__global__ void __launch_bounds__(64) k_schedule_global(SchedArgs a) {
  const int32_t r = blockIdx.x;
  if (*a.err) return;
  if (!state_header_ok(a)) return;
  RepState *rs = reinterpret_cast<RepState *>(a.state + a.L.reps) + r;
  if (!a.global_only && !rs->overflow) return;
  if (rs->done) {
    if (threadIdx.x == 0) {
      a.steps[r] = rs->s;
      a.decisions[r] = rs->seq;
      a.max_gap[r] = rs->gap;
    }
    const int64_t *u_all = reinterpret_cast<const int64_t *>(a.state + a.L.u_all) + int64_t(r) * a.t.U;
    for (int32_t k = threadIdx.x; k < a.t.U; k += 64) a.counter[int64_t(r) * a.t.U + k] = u_all[k];
    return;
  }
  const int64_t base = a.t.rep_off[r];
  const int32_t cap = int32_t(a.t.rep_off[r + 1] - base) + 1;
  Store S;
  char *st = a.state;
  S.xcap = cap;
  S.pcap = cap;
  S.clcap = cap;
  S.xkey = reinterpret_cast<uint64_t *>(st + a.L.xkey) + base + r;
  S.xuser = reinterpret_cast<int32_t *>(st + a.L.xuser) + base + r;
  S.xq = reinterpret_cast<int32_t *>(st + a.L.xq) + base + r;
  S.xfh = reinterpret_cast<int32_t *>(st + a.L.xfh) + base + r;
  S.xft = reinterpret_cast<int32_t *>(st + a.L.xft) + base + r;
  S.xrdy = reinterpret_cast<int32_t *>(st + a.L.xrdy) + base + r;
  S.p_cost = reinterpret_cast<int64_t *>(st + a.L.p_cost) + base + r;
  S.p_rec = reinterpret_cast<int32_t *>(st + a.L.p_rec) + base + r;
  S.p_tok = reinterpret_cast<int32_t *>(st + a.L.p_tok) + base + r;
  S.p_succ = reinterpret_cast<int32_t *>(st + a.L.p_succ) + base + r;
  S.p_next = reinterpret_cast<int32_t *>(st + a.L.p_next) + base + r;
  S.p_free = reinterpret_cast<int32_t *>(st + a.L.p_free) + base + r;
  S.cl_rec = reinterpret_cast<int32_t *>(st + a.L.cl_rec) + base + r;
  S.cl_prev = reinterpret_cast<int32_t *>(st + a.L.cl_prev) + base + r;
  S.cl_user = reinterpret_cast<int32_t *>(st + a.L.cl_user) + base + r;
  S.cl_e = reinterpret_cast<int32_t *>(st + a.L.cl_e) + base + r;
  S.cl_rdy = reinterpret_cast<int32_t *>(st + a.L.cl_rdy) + base + r;
  S.u = reinterpret_cast<int64_t *>(st + a.L.u_all) + int64_t(r) * a.t.U;
  S.xslot = reinterpret_cast<int32_t *>(st + a.L.xslot_all) + int64_t(r) * a.t.U;
  S.users_global = true;
  run_replica<true>(a, S, r, false);
  if (threadIdx.x == 0) rs->overflow = 0;
}

// ---------------------------------------------------------------- init and checks

__global__ void k_state_header(char *state, StateLayout L, int32_t R, int32_t U, int64_t N) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    Header *h = reinterpret_cast<Header *>(state + L.hdr);
    h->magic = kMagic;
    h->version = kVersion;
    h->R = R;
    h->U = U;
    h->N = N;
  }
}

__global__ void k_state_reps(char *state, StateLayout L, int32_t R) {
  int32_t r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r < R) {
    RepState *rs = reinterpret_cast<RepState *>(state + L.reps) + r;
    RepState z = {};
    z.last_exit = -1;
    *rs = z;
  }
}

__global__ void k_state_users(char *state, StateLayout L, int64_t RU) {
  for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < RU;
       i += int64_t(gridDim.x) * blockDim.x) {
    reinterpret_cast<int64_t *>(state + L.u_all)[i] = 0;
    reinterpret_cast<int32_t *>(state + L.xslot_all)[i] = -1;
  }
}

__global__ void k_state_records(char *state, StateLayout L, int64_t N) {
  for (int64_t g = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; g < N;
       g += int64_t(gridDim.x) * blockDim.x) {
    reinterpret_cast<int8_t *>(state + L.fate)[g] = -1;
    reinterpret_cast<int32_t *>(state + L.succ)[g] = -1;
  }
}

// next-call links: succ[prev] = i within each replica (prev is validated by the
// scheduler's checks before use; invalid links are skipped here)
__global__ void k_state_succ(char *state, StateLayout L, DevTrace t) {
  if (!t.call) return;
  for (int64_t g = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; g < t.N;
       g += int64_t(gridDim.x) * blockDim.x) {
    int32_t c = t.call[g];
    if (c <= 0) continue;
    int32_t r = replica_of(t.rep_off, t.R, g);
    int64_t base = t.rep_off[r], i = g - base;
    int32_t p = t.prev[g];
    if (p >= 0 && p < i) reinterpret_cast<int32_t *>(state + L.succ)[base + p] = int32_t(i);
  }
}

struct CheckArgs {
  DevTrace t;
  const int64_t *cost;
  const uint8_t *reason;
  const char *state;
  StateLayout L;
  int32_t *err;
};

__global__ void __launch_bounds__(256) k_sched_check(CheckArgs a) {
  const DevTrace &t = a.t;
  int32_t code = 0;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    const Header *h = reinterpret_cast<const Header *>(a.state + a.L.hdr);
    if (!(h->magic == kMagic && h->version == kVersion && h->R == t.R && h->U == t.U &&
          h->N == t.N))
      code = FS_E_STATE;
  }
  for (int64_t g = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; g < t.N;
       g += int64_t(gridDim.x) * blockDim.x) {
    int32_t r = replica_of(t.rep_off, t.R, g);
    int64_t base = t.rep_off[r], i = g - base;
    int32_t u = t.user[g], ap = t.app[g];
    int64_t ts = t.ts[g];
    if (u < 0 || u >= t.U || ap < 0 || ap >= t.A) code = max(code, int32_t(FS_E_RANGE));
    if (ts < 0) code = max(code, int32_t(FS_E_RANGE));
    if (g > base && t.ts[g - 1] > ts) code = max(code, int32_t(FS_E_ORDER));
    if (!len_ok(t.len_in[g]) || !len_ok(t.len_out[g]) || (t.len_sys && !len_ok(t.len_sys[g])))
      code = max(code, int32_t(FS_E_RANGE));
    if (t.call) {
      int32_t c = t.call[g], h = t.head[g], p = t.prev[g];
      bool ok;
      if (c == 0) {
        ok = h == i && p == -1;
      } else {
        ok = c > 0 && p >= 0 && p < i;
        if (ok) {
          int64_t gp = base + p;
          ok = t.call[gp] == c - 1 && t.user[gp] == u && t.head[gp] == h;
        }
      }
      if (!ok) code = max(code, int32_t(FS_E_RANGE));
    }
    int64_t cst = a.cost[g];
    if (cst < 0 || cst >= kValueLimit) code = max(code, int32_t(FS_E_RANGE));
    if (a.reason && a.reason[g] > 2) code = max(code, int32_t(FS_E_RANGE));
  }
  if (code) raise_err(a.err, code);
}

int grid_for(int64_t n, int threads) {
  int64_t b = (n + threads - 1) / threads;
  if (b < 1) b = 1;
  if (b > 65536) b = 65536;
  return int(b);
}

size_t onchip_lds_bytes(int32_t pcap, int32_t U, bool users_lds) {
  size_t b = 0;
  auto add = [&](size_t x) { b += (x + 15) & ~size_t(15); };
  add(8 * kXCap);
  add(8 * size_t(pcap));
  for (int i = 0; i < 5; ++i) add(4 * kXCap);
  for (int i = 0; i < 5; ++i) add(4 * size_t(pcap));
  for (int i = 0; i < 5; ++i) add(4 * kCLCap);
  if (users_lds) {
    add(8 * size_t(U));
    add(4 * size_t(U));
  }
  return b;
}

}  // namespace

size_t state_bytes(const fs_trace *t) {
  return state_layout(t->n_replicas, t->n_users, t->rep_off_h[t->n_replicas]).total;
}

hipError_t launch_state_init(void *state, const fs_trace *t, hipStream_t s) {
  const int64_t N = t->rep_off_h[t->n_replicas];
  StateLayout L = state_layout(t->n_replicas, t->n_users, N);
  char *st = static_cast<char *>(state);
  hipLaunchKernelGGL(k_state_header, dim3(1), dim3(64), 0, s, st, L, t->n_replicas, t->n_users, N);
  hipLaunchKernelGGL(k_state_reps, dim3((t->n_replicas + 255) / 256), dim3(256), 0, s, st, L,
                     t->n_replicas);
  const int64_t RU = int64_t(t->n_replicas) * t->n_users;
  hipLaunchKernelGGL(k_state_users, dim3(grid_for(RU, 256)), dim3(256), 0, s, st, L, RU);
  if (N > 0) {
    hipLaunchKernelGGL(k_state_records, dim3(grid_for(N, 256)), dim3(256), 0, s, st, L, N);
    hipLaunchKernelGGL(k_state_succ, dim3(grid_for(N, 256)), dim3(256), 0, s, st, L, dev_trace(t));
  }
  return hipGetLastError();
}

hipError_t launch_schedule(void *state, const fs_trace *t, const int64_t *cost,
                           const uint8_t *reason, const fs_engine *eng, fs_outputs *out,
                           int64_t n_steps, hipStream_t s) {
  const int64_t N = t->rep_off_h[t->n_replicas];
  SchedArgs a;
  a.t = dev_trace(t);
  a.cost = cost;
  a.reason = reason;
  a.tau = eng->step_us;
  a.cap = eng->cap_tokens;
  a.theta = eng->overload_tokens;
  a.n_steps = n_steps;
  a.global_only = (eng->flags & FS_ENGINE_GLOBAL_ONLY) != 0;
  a.status = out->status;
  a.admit_step = out->admit_step;
  a.admit_seq = out->admit_seq;
  a.counter_after = out->counter_after;
  a.counter_on_arrival = out->counter_on_arrival;
  a.counter = out->counter;
  a.steps = out->steps;
  a.decisions = out->decisions;
  a.max_gap = out->max_gap;
  a.err = out->err;
  a.state = static_cast<char *>(state);
  a.L = state_layout(t->n_replicas, t->n_users, N);
  const bool users_lds = t->n_users <= kUsersLdsMax;
  a.pcap = t->n_users > 512 ? 512 : 1024;

  CheckArgs ca{a.t, cost, reason, a.state, a.L, a.err};
  hipLaunchKernelGGL(k_sched_check, dim3(grid_for(N > 0 ? N : 1, 256)), dim3(256), 0, s, ca);
  const dim3 grid(t->n_replicas), block(64);
  if (!a.global_only) {
    size_t lds = onchip_lds_bytes(a.pcap, t->n_users, users_lds);
    if (users_lds)
      hipLaunchKernelGGL(k_schedule_onchip<true>, grid, block, lds, s, a);
    else
      hipLaunchKernelGGL(k_schedule_onchip<false>, grid, block, lds, s, a);
  }
  hipLaunchKernelGGL(k_schedule_global, grid, block, 0, s, a);
  return hipGetLastError();
}

}  // namespace fs

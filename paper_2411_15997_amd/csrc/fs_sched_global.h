// WSC scheduler steps in global memory: the pass over one replica that the
// global-memory kernel runs (and that an on-chip instance continues with).
//
// The on-chip kernel (fs_sched_onchip.hip) runs every replica whose backlogged users,
// queued first calls and ready later calls fit its LDS and register tables.  A
// replica that would overflow them is handed over here: this pass keeps the same
// state as the on-chip one -- service counters u_i, the waiting queue Q (a
// dictionary from user to queued requests), the last user to leave Q, the overload
// measure -- with every structure in the state buffer, so its capacities are the
// trace's own sizes.  It rebuilds the queue from the requests that have arrived and
// are still undecided and continues exactly where the on-chip kernel stopped,
// including inside a step's admissions.
//   X table   slots [0, nX) of users with something queued: key (tier << 62 | u),
//             whose tier is 0 while the user has a ready later call of an incomplete
//             interaction, a FIFO of queued first calls and a list of ready later calls.
//   pool      entries of queued requests: record, cost, tokens, next call, link, and
//             the next call's data when that call has already arrived.
//   segments  first calls beyond the pool go to a per-user segment (sized by the
//             user's number of first calls) and are refilled 64 at a time.
//   window    the next 64 records, one per lane, with their step and the user's
//             state prefetched; every state change patches the lanes it affects.
#pragma once

#include "fs_sched_common.h"

namespace fs {
namespace {

using namespace sched;

constexpr int kReserve = 32;  // pool entries first calls leave for later calls

template <bool G, class T>
__device__ inline T RD(const T *p) {
  if constexpr (G)
    return ld_fresh(p);
  else
    return *p;
}

// A queued request in the pool: three 16-byte words.
struct Entry {
  int32_t rec, tok, succ, next;  // record, tokens, its next call (-1: none), list link
  int64_t cost, scost;           // its cost; the staged cost of its next call
  int32_t sv, stok, ssucc, pad;  // staged next call: present, its tokens, its own next call
};
static_assert(sizeof(Entry) == 48, "Entry layout");

// Storage of the pool and per-user arrays: LDS (on chip) or the state buffer (global).
struct Store {
  Entry *e;         // pool entries
  int32_t *e_free;  // stack of free entries
  int64_t *u;       // counters of the replica's users (current for users not in X)
  int32_t *xslot;   // user -> X slot (global-memory table only)
  int32_t pcap;
  bool users_global;
};

template <bool G>
__device__ inline Entry ld_entry(const Entry *p) {
  Entry v;
  if constexpr (G) {
    v.rec = ld_fresh(&p->rec);
    v.tok = ld_fresh(&p->tok);
    v.succ = ld_fresh(&p->succ);
    v.next = ld_fresh(&p->next);
    v.cost = ld_fresh(&p->cost);
    v.scost = ld_fresh(&p->scost);
    v.sv = ld_fresh(&p->sv);
    v.stok = ld_fresh(&p->stok);
    v.ssucc = ld_fresh(&p->ssucc);
  } else {
    v = *p;
  }
  v.rec = uni(v.rec);
  v.tok = uni(v.tok);
  v.succ = uni(v.succ);
  v.next = uni(v.next);
  v.cost = uni64(v.cost);
  v.scost = uni64(v.scost);
  v.sv = uni(v.sv);
  v.stok = uni(v.stok);
  v.ssucc = uni(v.ssucc);
  v.pad = 0;
  return v;
}

// The same table in global memory (after an on-chip overflow): slots [0, nX) packed,
// capacity n_r + 1, with the user -> slot table S.xslot.
struct XMem {
  uint64_t *k;
  int32_t *user, *q, *fh, *ft, *hh, *ht, *sb, *rh, *rdy;
  int32_t cap;
  __device__ void init() {}
  __device__ uint64_t key(int32_t x) const { return uint64_t(uni64(int64_t(ld_fresh(k + x)))); }
  __device__ void set_key(int32_t x, uint64_t v) {
    if (threadIdx.x == 0) k[x] = v;
  }
#define FS_XMEM_FIELD(f)                                                          \
  __device__ int32_t get_##f(int32_t x) const { return uni(ld_fresh(f + x)); } \
  __device__ void set_##f(int32_t x, int32_t v) {                                 \
    if (threadIdx.x == 0) f[x] = v;                                               \
  }
  FS_XMEM_FIELD(user)
  FS_XMEM_FIELD(q)
  FS_XMEM_FIELD(fh)
  FS_XMEM_FIELD(ft)
  FS_XMEM_FIELD(hh)
  FS_XMEM_FIELD(ht)
  FS_XMEM_FIELD(sb)
  FS_XMEM_FIELD(rh)
  FS_XMEM_FIELD(rdy)
#undef FS_XMEM_FIELD
  __device__ void copy(int32_t from, int32_t to) {
    set_key(to, key(from));
    set_user(to, get_user(from));
    set_q(to, get_q(from));
    set_fh(to, get_fh(from));
    set_ft(to, get_ft(from));
    set_hh(to, get_hh(from));
    set_ht(to, get_ht(from));
    set_sb(to, get_sb(from));
    set_rh(to, get_rh(from));
    set_rdy(to, get_rdy(from));
  }
  __device__ int32_t find(int32_t kk, const Store &S) const { return uni(ld_fresh(S.xslot + kk)); }
  __device__ int32_t alloc(int32_t kk, int32_t nX, const Store &S) {
    if (threadIdx.x == 0) S.xslot[kk] = nX;
    return nX;
  }
  // Moves the last slot into the freed one.
  __device__ void release(int32_t x, int32_t kk, int32_t nX, const Store &S) {
    const int32_t last = nX - 1;
    if (threadIdx.x == 0) S.xslot[kk] = -1;
    if (x != last) {
      const int32_t k2 = get_user(last);
      copy(last, x);
      if (threadIdx.x == 0) S.xslot[k2] = x;
    }
    set_key(last, kEmptyKey);
  }
  __device__ int32_t slot(int32_t i, int32_t) const { return i; }
  // one slot per lane (not wave-uniform)
  __device__ uint64_t key_at(int32_t x) const { return ld_fresh(k + x); }
  __device__ uint32_t user_at(int32_t x) const { return uint32_t(ld_fresh(user + x)); }
  __device__ int32_t argmin(int32_t nX, uint64_t &bk, int32_t &bu) const {
    uint64_t kk = kEmptyKey;
    uint32_t us = 0xffffffffu, bx = 0xffffffffu;
    for (int32_t x0 = threadIdx.x; x0 < nX; x0 += 256) {  // four slots a lane, loads together
      uint64_t a[4];
      uint32_t b[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int32_t x = x0 + 64 * j;
        a[j] = x < nX ? ld_fresh(k + x) : kEmptyKey;
        b[j] = x < nX ? uint32_t(ld_fresh(user + x)) : 0xffffffffu;
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bool take = a[j] < kk || (a[j] == kk && b[j] < us);
        kk = take ? a[j] : kk;
        us = take ? b[j] : us;
        bx = take ? uint32_t(x0 + 64 * j) : bx;
      }
    }
    wave_argmin(kk, us, bx);
    bk = uint64_t(rdl64(int64_t(kk), 63));
    bu = rdl(int32_t(us), 63);
    return rdl(int32_t(bx), 63);
  }
  __device__ void minmax(int32_t nX, int64_t &mn, int64_t &mx) const {
    uint64_t lo = kEmptyKey, hi = 0;
    for (int32_t x0 = threadIdx.x; x0 < nX; x0 += 256) {
      uint64_t v[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int32_t x = x0 + 64 * j;
        v[j] = x < nX ? ld_fresh(k + x) & kValMask : kEmptyKey;
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int32_t x = x0 + 64 * j;
        lo = v[j] < lo ? v[j] : lo;
        hi = x < nX && v[j] > hi ? v[j] : hi;
      }
    }
    wave_minmax(lo, hi);
    mn = rdl64(int64_t(lo), 63);
    mx = rdl64(int64_t(hi), 63);
  }
};

// The same table in LDS when the replica's users fit (one slot per user, so capacity U),
// with its own user -> slot table: every read of a decision's bookkeeping then stays
// on chip and only the pool of queued requests is in global memory.
struct XLds {
  uint64_t *k;
  int32_t *user, *q, *fh, *ft, *hh, *ht, *sb, *rh, *rdy, *xs;
  int32_t cap;
  __device__ void init() {
    for (int32_t i = threadIdx.x; i < cap; i += 64) {
      xs[i] = -1;
      k[i] = kEmptyKey;
    }
  }
  __device__ uint64_t key(int32_t x) const { return uint64_t(uni64(int64_t(k[x]))); }
  __device__ void set_key(int32_t x, uint64_t v) {
    if (threadIdx.x == 0) k[x] = v;
  }
#define FS_XLDS_FIELD(f)                                                 \
  __device__ int32_t get_##f(int32_t x) const { return uni(f[x]); } \
  __device__ void set_##f(int32_t x, int32_t v) {                        \
    if (threadIdx.x == 0) f[x] = v;                                      \
  }
  FS_XLDS_FIELD(user)
  FS_XLDS_FIELD(q)
  FS_XLDS_FIELD(fh)
  FS_XLDS_FIELD(ft)
  FS_XLDS_FIELD(hh)
  FS_XLDS_FIELD(ht)
  FS_XLDS_FIELD(sb)
  FS_XLDS_FIELD(rh)
  FS_XLDS_FIELD(rdy)
#undef FS_XLDS_FIELD
  __device__ void copy(int32_t from, int32_t to) {
    set_key(to, key(from));
    set_user(to, get_user(from));
    set_q(to, get_q(from));
    set_fh(to, get_fh(from));
    set_ft(to, get_ft(from));
    set_hh(to, get_hh(from));
    set_ht(to, get_ht(from));
    set_sb(to, get_sb(from));
    set_rh(to, get_rh(from));
    set_rdy(to, get_rdy(from));
  }
  __device__ int32_t find(int32_t kk, const Store &) const { return uni(xs[kk]); }
  __device__ int32_t alloc(int32_t kk, int32_t nX, const Store &) {
    if (threadIdx.x == 0) xs[kk] = nX;
    return nX;
  }
  // Moves the last slot into the freed one.
  __device__ void release(int32_t x, int32_t kk, int32_t nX, const Store &) {
    const int32_t last = nX - 1;
    if (threadIdx.x == 0) xs[kk] = -1;
    if (x != last) {
      const int32_t k2 = get_user(last);
      copy(last, x);
      if (threadIdx.x == 0) xs[k2] = x;
    }
    set_key(last, kEmptyKey);
  }
  __device__ int32_t slot(int32_t i, int32_t) const { return i; }
  // one slot per lane (not wave-uniform)
  __device__ uint64_t key_at(int32_t x) const { return k[x]; }
  __device__ uint32_t user_at(int32_t x) const { return uint32_t(user[x]); }
  __device__ int32_t argmin(int32_t nX, uint64_t &bk, int32_t &bu) const {
    uint64_t kk = kEmptyKey;
    uint32_t us = 0xffffffffu, bx = 0xffffffffu;
    for (int32_t x0 = threadIdx.x; x0 < nX; x0 += 256) {  // four slots a lane, loads together
      uint64_t a[4];
      uint32_t b[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int32_t x = x0 + 64 * j;
        a[j] = x < nX ? k[x] : kEmptyKey;
        b[j] = x < nX ? uint32_t(user[x]) : 0xffffffffu;
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bool take = a[j] < kk || (a[j] == kk && b[j] < us);
        kk = take ? a[j] : kk;
        us = take ? b[j] : us;
        bx = take ? uint32_t(x0 + 64 * j) : bx;
      }
    }
    wave_argmin(kk, us, bx);
    bk = uint64_t(rdl64(int64_t(kk), 63));
    bu = rdl(int32_t(us), 63);
    return rdl(int32_t(bx), 63);
  }
  __device__ void minmax(int32_t nX, int64_t &mn, int64_t &mx) const {
    uint64_t lo = kEmptyKey, hi = 0;
    for (int32_t x0 = threadIdx.x; x0 < nX; x0 += 256) {
      uint64_t v[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int32_t x = x0 + 64 * j;
        v[j] = x < nX ? k[x] & kValMask : kEmptyKey;
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int32_t x = x0 + 64 * j;
        lo = v[j] < lo ? v[j] : lo;
        hi = x < nX && v[j] > hi ? v[j] : hi;
      }
    }
    wave_minmax(lo, hi);
    mn = rdl64(int64_t(lo), 63);
    mx = rdl64(int64_t(hi), 63);
  }
};
constexpr size_t kXLdsBytesPerUser = 8 + 8 + 10 * 4;  // counter, key, nine fields and xs

// Per block of 64 X slots, in LDS: the least (key, user).  The argmin then reads the
// block minima and one block instead of every slot.  Kept while many users are
// backlogged (more than kHierOn; dropped at kHierOff or fewer, and while their blocks
// fit, cap); rebuilt from X when that starts.  Below that a flat scan of X, four slots
// a lane with their loads issued together, costs less than keeping the minima.
struct XBlocks {
  uint64_t *k;
  uint32_t *u;
  int32_t cap;  // blocks that fit (0: single-level scans only)
};
constexpr size_t kXBlockBytes = 8 + 4;
constexpr int32_t kHierOn = 512, kHierOff = 256;

// ---------------------------------------------------------------------------
// The scheduler body.  All control flow is wave-uniform; the arrival window holds
// one record per lane.  Per-record outputs are collected in registers and written
// with one store per field for up to 64 records: arrival outcomes by window lane,
// admissions by admission order.
// ---------------------------------------------------------------------------
// Inlined into the kernel for each table kind: as a called function its argument
// structs would live in scratch memory and every field read would go through it.
// EF >= 0: the engine flags fixed at compile time (1 first come first served, 2
// interaction-blind, 4 literal), else read from the arguments.
template <bool G, class XT, int EF = -1>
__device__ __forceinline__ void run_replica(const SchedArgs &a, Store &S, XT &X, const XBlocks &XB, int32_t r,
                            bool onchip) {
  const int lane = threadIdx.x;
  const DevTrace &t = a.t;
  const int64_t base = t.rep_off[r];
  const int64_t n = t.rep_off[r + 1] - base;
  const int32_t U = t.U;
  RepState *rs = reinterpret_cast<RepState *>(a.state + a.L.reps) + r;
  int8_t *fate = reinterpret_cast<int8_t *>(a.state + a.L.fate) + base;
  const int32_t *succ = reinterpret_cast<const int32_t *>(a.state + a.L.succ) + base;
  int32_t *emap = reinterpret_cast<int32_t *>(a.state + a.L.emap) + base;
  const uint32_t *seg_start = reinterpret_cast<const uint32_t *>(a.state + a.L.seg_start);
  int32_t *seg_rec = reinterpret_cast<int32_t *>(a.state + a.L.seg_rec);
  int32_t *seg_tok = reinterpret_cast<int32_t *>(a.state + a.L.seg_tok);
  int64_t *seg_cost = reinterpret_cast<int64_t *>(a.state + a.L.seg_cost);
  int32_t *seg_succ = reinterpret_cast<int32_t *>(a.state + a.L.seg_succ);
  int64_t *u_all = reinterpret_cast<int64_t *>(a.state + a.L.u_all) + int64_t(r) * U;
  int32_t *run_rec = reinterpret_cast<int32_t *>(a.state + a.L.run_rec) + base + r;
  int32_t *run_fin = reinterpret_cast<int32_t *>(a.state + a.L.run_fin) + base + r;

  // ---- scalar state
  int64_t s = uni64(rs->s), nxt = uni64(rs->nxt), debt = uni64(rs->debt);
  int64_t backlog = uni64(rs->backlog), seq = uni64(rs->seq), gap = uni64(rs->gap);
  int64_t last_exit_u = uni64(rs->last_exit_u), low = uni64(rs->low);
  int32_t last_exit = uni(rs->last_exit);
  int64_t s_end;
  if (onchip || !rs->overflow)
    s_end = a.n_steps < 0 ? INT64_MAX : s + a.n_steps;
  else
    s_end = uni64(rs->s_end);  // resuming a launch that overflowed on chip
  const int64_t tau = a.tau, C = a.cap, theta = a.theta;
  // resuming inside step s: its arrivals are done and its budget is partly spent
  bool mid = !onchip && uni(rs->mid) != 0;
  int64_t fcfs_lo = low;  // every record below is decided (first-come choice)
  const int64_t mid_budget = uni64(rs->mid_budget);
  // literal engine: the running batch (admission order) and the KV tokens it holds
  const bool literal = EF >= 0 ? (EF & 4) != 0 : a.literal;
  const bool e_fcfs = EF >= 0 ? (EF & 1) != 0 : a.fcfs;
  const bool e_blind = EF >= 0 ? (EF & 2) != 0 : a.blind;
  int64_t kv_used = uni64(rs->kv_used), n_run = uni64(rs->n_run);

  if (!S.users_global)
    for (int32_t k = lane; k < U; k += 64) S.u[k] = u_all[k];
  for (int32_t e = lane; e < S.pcap; e += 64) S.e_free[e] = S.pcap - 1 - e;
  X.init();
  int32_t nfree = S.pcap, nX = 0;
  int32_t code = 0;
  bool overflow = false;
  __syncthreads();

  auto get_u = [&](int32_t k) -> int64_t { return S.users_global ? ld_fresh(S.u + k) : S.u[k]; };
  auto slot_u = [&](int32_t x) -> int64_t { return int64_t(X.key(x) & kValMask); };

  // Literal engine: the choice whose call did not fit in the free KV cache, kept while
  // it stays the least (key, user): keys only grow under charges, so it is dropped
  // only when its own key changes or users join, leave or gain a ready call.  A step
  // that retries after a finish then tests the fit without a scan of X.
  int32_t st_x = -1, st_user = 0, st_tok = 0;
  uint64_t st_key = 0;
  // The least and largest counter in X as of the last gap sample, reused while no key
  // of X has changed since (steps of finishes that charge only idle users).
  bool x_dirty = true;
  int64_t x_mn = 0, x_mx = 0;

  // ---- two-level argmin over X (block minima of 64 slots) while nX > 64
  bool hier = false;
  auto blk_set = [&](int32_t b) {  // block b's least (key, user)
    const int32_t sx = b * 64 + lane;
    uint64_t kk = kEmptyKey;
    uint32_t us = 0xffffffffu, bx = 0xffffffffu;
    if (sx < nX) {
      kk = X.key_at(sx);
      us = X.user_at(sx);
      bx = uint32_t(sx);
    }
    wave_argmin(kk, us, bx);
    if (lane == 63) {
      XB.k[b] = kk;
      XB.u[b] = us;
    }
  };
  auto blk_touch = [&](int32_t x) {  // slot x changed (key, or moved / freed)
    if (!hier) return;
    wave_fence();
    blk_set(x >> 6);
  };
  auto blk_sync = [&]() {  // nX changed: start or stop keeping the block minima
    const bool fits = ((nX + 63) >> 6) <= XB.cap;
    if (!hier && nX > kHierOn && fits) {
      hier = true;
      wave_fence();
      for (int32_t b = 0; b * 64 < nX; ++b) blk_set(b);
    } else if (hier && (nX <= kHierOff || !fits)) {
      hier = false;
    }
  };
  // least (key, user) among the backlogged users: its slot, key and user
  auto argmin_x = [&](uint64_t &bk, int32_t &bu) -> int32_t {
    if (!hier) return X.argmin(nX, bk, bu);
    wave_fence();
    const int32_t nb = (nX + 63) >> 6;
    uint64_t kk = kEmptyKey;
    uint32_t us = 0xffffffffu, bx = 0xffffffffu;
    for (int32_t b = lane; b < nb; b += 64) {
      const uint64_t v = XB.k[b];
      const uint32_t w = XB.u[b];
      const bool take = v < kk || (v == kk && w < us);
      kk = take ? v : kk;
      us = take ? w : us;
      bx = take ? uint32_t(b) : bx;
    }
    wave_argmin(kk, us, bx);
    const int32_t b = rdl(int32_t(bx), 63);
    const int32_t sx = b * 64 + lane;
    uint64_t k2 = kEmptyKey;
    uint32_t u2 = 0xffffffffu, x2 = 0xffffffffu;
    if (sx < nX) {
      k2 = X.key_at(sx);
      u2 = X.user_at(sx);
      x2 = uint32_t(sx);
    }
    wave_argmin(k2, u2, x2);
    bk = uint64_t(rdl64(int64_t(k2), 63));
    bu = rdl(int32_t(u2), 63);
    return rdl(int32_t(x2), 63);
  };
  // least and largest counter among the backlogged users (nX > 0; once a step)
  auto minmax_x = [&](int64_t &mn, int64_t &mx) { X.minmax(nX, mn, mx); };
  auto set_key = [&](int32_t x, int64_t uval) {
    if (x == st_x) st_x = -1;
    x_dirty = true;
    X.set_key(x, (uint64_t(X.get_rdy(x) > 0 ? 0 : 1) << kTierShift) | uint64_t(uval));
    blk_touch(x);
  };
  auto tokens_at = [&](int64_t i) -> int32_t {
    const int64_t g = base + i;
    return t.len_in[g] + t.len_out[g] + (t.len_sys ? t.len_sys[g] : 0);
  };

  // ---- admissions waiting to be written: lane i holds the i-th of nd
  int32_t d_rec = 0, d_step = 0, nd = 0;
  int64_t d_cnt = 0;
  auto flush_decisions = [&]() {
    if (nd == 0) return;
    if (lane < nd) {
      const int64_t g = base + d_rec;
      fate[d_rec] = 0;
      a.status[g] = 0;
      a.admit_step[g] = d_step;
      if (a.admit_seq) a.admit_seq[g] = int32_t(seq - nd + lane);
      // (the literal engine writes counter_after when the call finishes)
      if (a.counter_after && !literal) a.counter_after[g] = d_cnt;
    }
    nd = 0;
  };

  // ---- window of upcoming records (one per lane), branch-free so it stays in registers
  int64_t wbase = nxt;
  int64_t w_cost = 0, c_u = 0, o_coa = 0;
  int32_t w_step = 0, w_user = -1, w_call = 0, w_head = -1, w_prev = -1, w_succ = -1, w_tok = 0,
          w_reason = 0, w_seg = 0, c_prev_adm = 0, c_head_blk = 0, c_prev_drop = 0, c_pe = -1,
          o_st = 0;
  // Arrival outcomes of the window's processed lanes: throttled ones get their status
  // and fate, every one its counter on arrival.
  auto flush_window = [&]() {
    const int64_t done = nxt - wbase;
    if (lane < done) {
      const int64_t i = wbase + lane, g = base + i;
      if (o_st > 0) {
        fate[i] = int8_t(o_st);
        a.status[g] = int8_t(o_st);
        a.admit_step[g] = -1;
        if (a.admit_seq) a.admit_seq[g] = -1;
        if (a.counter_after) a.counter_after[g] = -1;
      }
      if (a.counter_on_arrival) a.counter_on_arrival[g] = o_coa;
    }
    o_st = 0;
  };
  auto load_window = [&]() {
    wave_fence();
    const int64_t i = wbase + lane;
    const bool valid = i < n;
    const int64_t li = valid ? i : 0;
    const int64_t g = base + li;
    const int32_t call = (valid && t.call) ? t.call[g] : 0;
    const int32_t usr = valid ? t.user[g] : 0;
    const int32_t hd = (valid && t.call) ? t.head[g] : int32_t(li);
    const int32_t pv = (valid && t.call) ? t.prev[g] : -1;
    const int64_t ts = valid ? t.ts[g] : 0;
    w_step = int32_t(ts / tau);
    w_user = valid ? usr : -1;
    w_call = call;
    w_head = valid ? hd : -1;
    w_prev = pv;
    w_succ = valid ? succ[li] : -1;
    w_tok = valid ? tokens_at(li) : 0;
    w_cost = valid ? a.cost[g] : 0;
    w_reason = (valid && a.reason) ? a.reason[g] : 0;
    w_seg = int32_t(seg_start[int64_t(r) * U + usr]);
    const int64_t uu = get_u(usr);
    c_u = valid ? uu : 0;
    const int8_t pf = call > 0 ? ld_fresh(fate + pv) : int8_t(-1);
    const int8_t hf = call > 0 ? ld_fresh(fate + hd) : int8_t(-1);
    const int32_t pe = call > 0 ? ld_fresh(emap + pv) : -1;
    c_prev_adm = (call > 0 && pf == 0) ? 1 : 0;
    c_head_blk = (call > 0 && (hf == 1 || hf == 2)) ? 1 : 0;
    c_prev_drop = (call > 0 && pf > 0) ? 1 : 0;
    c_pe = pe;
    o_st = 0;
  };
  auto advance_window = [&]() {
    flush_window();
    flush_decisions();
    wbase = nxt;
    load_window();
  };

  // ---- backlogged users
  auto join_x = [&](int32_t k, int64_t uval, int32_t segb) -> int32_t {
    st_x = -1;
    x_dirty = true;
    const int32_t x = X.alloc(k, nX, S);
    ++nX;
    X.set_user(x, k);
    X.set_q(x, 0);
    X.set_fh(x, -1);
    X.set_ft(x, -1);
    X.set_hh(x, 0);
    X.set_ht(x, 0);
    X.set_sb(x, segb);
    X.set_rh(x, -1);
    X.set_rdy(x, 0);
    X.set_key(x, (uint64_t(1) << kTierShift) | uint64_t(uval));
    if (hier) blk_touch(x);
    blk_sync();
    return x;
  };
  auto leave_x = [&](int32_t x, int32_t k, int64_t uval) {
    st_x = -1;
    x_dirty = true;
    if (lane == 0) S.u[k] = uval;
    c_u = (w_user == k) ? uval : c_u;
    X.release(x, k, nX, S);
    --nX;
    // the last slot moved into x, and the old last slot (now nX) is free
    if (hier && (nX >> 6) != (x >> 6)) blk_touch(nX);
    blk_touch(x);
    blk_sync();
  };

  // ---- pool
  auto alloc_e = [&]() -> int32_t { return uni(RD<G>(&S.e_free[--nfree])); };
  auto free_e = [&](int32_t e) {
    if (lane == 0) S.e_free[nfree] = e;
    ++nfree;
  };
  // A record entered the pool at entry e: remember it for its next call's arrival.
  auto note_pool = [&](int32_t rec, int32_t e) {
    if (lane == 0) emap[rec] = e;
    c_pe = (w_prev == rec) ? e : c_pe;
  };
  auto put_entry = [&](int32_t e, int32_t rec, int32_t tok, int64_t cst, int32_t sc, int32_t sv,
                       int64_t scost, int32_t stok, int32_t ssucc) {
    if (lane == 0) {
      Entry v;
      v.rec = rec;
      v.tok = tok;
      v.succ = sc;
      v.next = -1;
      v.cost = cst;
      v.scost = scost;
      v.sv = sv;
      v.stok = stok;
      v.ssucc = ssucc;
      v.pad = 0;
      S.e[e] = v;
    }
    note_pool(rec, e);
  };
  // Data of record i (an arrived later call) read from the inputs.
  auto load_record = [&](int32_t i, int64_t &cst, int32_t &tok, int32_t &sc) {
    cst = uni64(a.cost[base + i]);
    tok = uni(tokens_at(i));
    sc = uni(succ[i]);
  };
  auto fifo_append = [&](int32_t x, int32_t e) {
    const int32_t tl = X.get_ft(x);
    if (tl < 0)
      X.set_fh(x, e);
    else if (lane == 0)
      S.e[tl].next = e;
    X.set_ft(x, e);
  };
  auto ready_push = [&](int32_t x, int32_t e) {
    st_x = -1;  // (its user's key drops to the ready tier)
    if (lane == 0) S.e[e].next = X.get_rh(x);
    X.set_rh(x, e);
    X.set_rdy(x, X.get_rdy(x) + 1);
  };
  // A first call joins its user's FIFO: in the pool while the user has nothing in its
  // HBM segment and the pool has room, else at the segment's tail.
  auto enqueue_first = [&](int32_t x, int32_t rec, int32_t tok, int64_t cst, int32_t sc) -> bool {
    const int32_t hh = X.get_hh(x), ht = X.get_ht(x);
    if (ht == hh && nfree > kReserve) {
      const int32_t e = alloc_e();
      put_entry(e, rec, tok, cst, sc, 0, 0, 0, -1);
      fifo_append(x, e);
      return true;
    }
    const int32_t k = X.get_user(x);
    const int64_t at = int64_t(X.get_sb(x)) + ht;
    const int64_t cap_end = int64_t(seg_start[int64_t(r) * U + k + 1]);
    if (at >= cap_end) return false;  // cannot happen: a segment holds all the user's first calls
    if (lane == 0) {
      seg_rec[at] = rec;
      seg_tok[at] = tok;
      seg_cost[at] = cst;
      seg_succ[at] = sc;
    }
    X.set_ht(x, ht + 1);
    return true;
  };
  // Refill the user's pool FIFO from its HBM segment (up to 64 entries, one load).
  auto refill = [&](int32_t x) -> bool {
    const int32_t hh = X.get_hh(x), ht = X.get_ht(x);
    int32_t m = ht - hh;
    if (m > 64) m = 64;
    if (m > nfree) m = nfree;
    if (m <= 0) return false;
    wave_fence();
    const int64_t at = int64_t(X.get_sb(x)) + hh + lane;
    const bool mine = lane < m;
    int32_t e = -1, rec = -1, sc = -1;
    if (mine) {
      rec = ld_fresh(seg_rec + at);
      const int32_t tok = ld_fresh(seg_tok + at);
      const int64_t cst = ld_fresh(seg_cost + at);
      sc = ld_fresh(seg_succ + at);
      int32_t sv = 0, stok = 0, ssucc = -1;
      int64_t scost = 0;
      if (sc >= 0 && sc < nxt) {  // its next call has already arrived: stage its data
        sv = 1;
        scost = a.cost[base + sc];
        stok = tokens_at(sc);
        ssucc = succ[sc];
      }
      e = RD<G>(&S.e_free[nfree - 1 - lane]);
      const int32_t en = lane + 1 < m ? RD<G>(&S.e_free[nfree - 2 - lane]) : -1;
      Entry v;
      v.rec = rec;
      v.tok = tok;
      v.succ = sc;
      v.next = en;
      v.cost = cst;
      v.scost = scost;
      v.sv = sv;
      v.stok = stok;
      v.ssucc = ssucc;
      v.pad = 0;
      S.e[e] = v;
      emap[rec] = e;
    }
    // next calls in the current window that have not arrived yet: point them at the entry
    uint64_t hit = __ballot(mine && sc >= nxt && sc < wbase + 64);
    while (hit) {
      const int l = __ffsll((long long)hit) - 1;
      hit &= hit - 1;
      const int32_t j = rdl(sc, l) - int32_t(wbase);
      c_pe = lane == j ? rdl(e, l) : c_pe;
    }
    X.set_fh(x, rdl(e, 0));
    X.set_ft(x, rdl(e, m - 1));
    X.set_hh(x, hh + m);
    nfree -= m;
    return true;
  };
  // Stage an arrived later call's data in its previous call's pool entry, if there.
  auto stage_in_prev = [&](int32_t prev_rec, int32_t pe, int64_t cst, int32_t tok, int32_t sc) {
    if (pe < 0 || pe >= S.pcap) return;
    if (uni(RD<G>(&S.e[pe].rec)) != prev_rec) return;
    if (lane == 0) {
      S.e[pe].sv = 1;
      S.e[pe].scost = cst;
      S.e[pe].stok = tok;
      S.e[pe].ssucc = sc;
    }
  };

  // Queue one arrived, unthrottled record (counted in backlog by the caller).
  // Returns false when an on-chip capacity would overflow (nothing changed then).
  auto enqueue = [&](int32_t rec, int32_t k, int32_t call, int32_t prev_rec, int32_t sc,
                     int32_t tok, int64_t cst, int32_t xs, int64_t uval, bool prev_adm,
                     int32_t segb, int32_t pe) -> bool {
    if (xs < 0 && nX >= X.cap) return false;
    if (call > 0 && prev_adm && nfree == 0) return false;
    const int32_t x = xs >= 0 ? xs : join_x(k, uval, segb);
    X.set_q(x, X.get_q(x) + 1);
    if (call == 0) {
      if (!enqueue_first(x, rec, tok, cst, sc)) code = FS_E_STATE;
    } else if (prev_adm) {
      const int32_t e = alloc_e();
      put_entry(e, rec, tok, cst, sc, 0, 0, 0, -1);
      ready_push(x, e);
      set_key(x, uval);
    } else {
      stage_in_prev(prev_rec, pe, cst, tok, sc);
    }
    return true;
  };

  // ---- rebuild the queue of a previous call: every arrived record still undecided
  for (int64_t b0 = low; b0 < nxt && !overflow && code == 0; b0 += 64) {
    const int64_t i = b0 + lane;
    const bool q = i < nxt && ld_fresh(fate + i) == -1;
    uint64_t m = __ballot(q);
    while (m && !overflow && code == 0) {
      const int l = __ffsll((long long)m) - 1;
      m &= m - 1;
      const int32_t rec = int32_t(b0 + l);
      const int64_t g = base + rec;
      const int32_t k = uni(t.user[g]);
      const int32_t call = t.call ? uni(t.call[g]) : 0;
      const int32_t prev_rec = t.call ? uni(t.prev[g]) : -1;
      int64_t cst;
      int32_t tok, sc;
      load_record(rec, cst, tok, sc);
      const int32_t xs = X.find(k, S);
      const int64_t uval = xs >= 0 ? slot_u(xs) : uni64(get_u(k));
      const bool prev_adm = call > 0 && ld_fresh(fate + prev_rec) == 0;
      const int32_t segb = int32_t(seg_start[int64_t(r) * U + k]);
      const int32_t pe = call > 0 ? uni(ld_fresh(emap + prev_rec)) : -1;
      if (!enqueue(rec, k, call, prev_rec, sc, tok, cst, xs, uval, prev_adm, segb, pe))
        overflow = true;
      // a ready later call whose own next call already arrived: stage that call's data
      if (!overflow && code == 0 && call > 0 && prev_adm && sc >= 0 && sc < nxt) {
        const int32_t xx = X.find(k, S);
        const int32_t e = X.get_rh(xx);
        int64_t c2;
        int32_t t2, s2;
        load_record(sc, c2, t2, s2);
        if (lane == 0) {
          S.e[e].sv = 1;
          S.e[e].scost = c2;
          S.e[e].stok = t2;
          S.e[e].ssucc = s2;
        }
      }
    }
  }
  if (overflow) {
    if (lane == 0) {
      rs->overflow = 1;
      rs->s_end = s_end;
    }
    return;
  }
  int64_t minX = 0;
  if (nX > 0) {
    int64_t mx;
    X.minmax(nX, minX, mx);
  }
  load_window();

  // literal engine: the earliest finish step of the running batch
  auto batch_min_fin = [&]() -> int64_t {
    uint32_t mf = 0xffffffffu;
    for (int64_t b0 = 0; b0 < n_run; b0 += 64) {
      const int64_t i = b0 + lane;
      const uint32_t f = i < n_run ? uint32_t(ld_fresh(run_fin + i)) : 0xffffffffu;
      mf = f < mf ? f : mf;
    }
    return n_run > 0 ? int64_t(wave_min32(mf)) : INT64_MAX;
  };
  int64_t min_fin = batch_min_fin();
  // Chunk mode (while the batch has at most kChunkCap entries): finished entries become
  // dead marks and lane c holds the least live finish step of entries [64c, 64c + 64),
  // so a step visits only the chunks with a finish due; the array is compacted when it
  // fills or is saved.  Otherwise every finish pass scans and compacts the whole batch.
  constexpr uint32_t kDeadFin = 0x7fffffffu;
  constexpr int64_t kChunkCap = 64 * 64;
  uint32_t cmin = 0xffffffffu;
  int64_t n_live = n_run;
  bool cm = false;
  // least live finish step of chunk c, into lane c
  auto chunk_min = [&](int64_t c) {
    const int64_t i = c * 64 + lane;
    const uint32_t f = i < n_run ? uint32_t(ld_fresh(run_fin + i)) : 0xffffffffu;
    const uint32_t m = wave_min32(f == kDeadFin ? 0xffffffffu : f);
    if (lane == c) cmin = m;
  };
  // removes the dead entries, keeping the admission order, and rebuilds the minima
  auto compact = [&]() {
    wave_fence();
    int64_t kept = 0;
    for (int64_t b0 = 0; b0 < n_run; b0 += 64) {
      const int64_t i = b0 + lane;
      const bool valid = i < n_run;
      const int32_t rr = valid ? ld_fresh(run_rec + i) : -1;
      const int32_t ff = valid ? ld_fresh(run_fin + i) : int32_t(kDeadFin);
      const bool live = valid && uint32_t(ff) != kDeadFin;
      const uint64_t km = __ballot(live);
      if (live) {
        const int64_t to = kept + __popcll(km & ((uint64_t(1) << lane) - 1));
        run_rec[to] = rr;
        run_fin[to] = ff;
      }
      kept += __popcll(km);
    }
    n_run = kept;
    wave_fence();
    cmin = 0xffffffffu;
    if (cm)
      for (int64_t c = 0; c * 64 < n_run; ++c) chunk_min(c);
  };
  if (literal && n_run <= kChunkCap / 2) {
    cm = true;
    wave_fence();
    for (int64_t c = 0; c * 64 < n_run; ++c) chunk_min(c);
  }
  // literal engine: the last admission attempt found the chosen call too large for the
  // free KV cache and nothing has changed since (no arrival, no finish): every step
  // until the next arrival or finish would repeat it, so those steps are skipped
  bool stalled = false;
  // Calls whose last output token is decoded in step s finish, in admission order: each
  // user is charged its call's cost (Eq. 2) and the call's KV tokens are freed; the
  // batch is compacted in place.
  // Charges one finishing call (record rec): its user pays its cost (Eq. 2) and its KV
  // tokens are freed.
  auto charge_finish = [&](int32_t rec) -> bool {
    const int64_t g = base + rec;
    const int32_t k = uni(t.user[g]);
    const int64_t cst = uni64(a.cost[g]);
    const int32_t xs = X.find(k, S);
    int64_t unew;
    if (xs >= 0) {
      unew = slot_u(xs) + cst;
      if (unew < kValueLimit) set_key(xs, unew);
    } else {
      unew = uni64(get_u(k)) + cst;
      if (unew < kValueLimit) {
        if (lane == 0) S.u[k] = unew;
        c_u = (w_user == k) ? unew : c_u;
      }
    }
    if (unew >= kValueLimit) {
      code = FS_E_OVERFLOW;
      return false;
    }
    if (k == last_exit) last_exit_u = unew;
    if (lane == 0 && a.counter_after) a.counter_after[g] = unew;
    kv_used -= uni(tokens_at(rec));
    return true;
  };
  // Chunk mode: the calls whose last output token falls in step s, chunk by chunk in
  // admission order, charged and marked dead.
  auto finish_chunks = [&]() {
    wave_fence();
    for (uint64_t due = __ballot(cmin <= uint32_t(s)); due && code == 0; due &= due - 1) {
      const int64_t c = __ffsll((long long)due) - 1;
      const int64_t i = c * 64 + lane;
      const bool valid = i < n_run;
      const int32_t rr = valid ? ld_fresh(run_rec + i) : -1;
      const int32_t ff = valid ? ld_fresh(run_fin + i) : int32_t(kDeadFin);
      const bool done = valid && int64_t(ff) == s;
      if (done) run_fin[i] = int32_t(kDeadFin);
      uint64_t dm = __ballot(done);
      n_live -= __popcll(dm);
      while (dm) {
        const int l = __ffsll((long long)dm) - 1;
        dm &= dm - 1;
        if (!charge_finish(rdl(rr, l))) break;
      }
      const uint32_t m = wave_min32((valid && !done && uint32_t(ff) != kDeadFin) ? uint32_t(ff)
                                                                                : 0xffffffffu);
      if (lane == c) cmin = m;
    }
    if (n_live == 0) {  // nothing runs: start the array afresh
      n_run = 0;
      cmin = 0xffffffffu;
    }
    const uint32_t mf = wave_min32(cmin);
    min_fin = mf == 0xffffffffu ? INT64_MAX : int64_t(mf);
  };
  auto finish_calls = [&]() {
    wave_fence();
    int64_t kept = 0;
    uint32_t mf = 0xffffffffu;
    for (int64_t b0 = 0; b0 < n_run && code == 0; b0 += 64) {
      const int64_t i = b0 + lane;
      const bool valid = i < n_run;
      const int32_t rr = valid ? ld_fresh(run_rec + i) : -1;
      const int32_t ff = valid ? ld_fresh(run_fin + i) : 0;
      const bool fin = valid && int64_t(ff) == s;
      uint64_t dm = __ballot(fin);
      const uint64_t km = __ballot(valid && !fin);
      if (valid && !fin) {
        const int64_t to = kept + __popcll(km & ((uint64_t(1) << lane) - 1));
        run_rec[to] = rr;
        run_fin[to] = ff;
        mf = uint32_t(ff) < mf ? uint32_t(ff) : mf;
      }
      kept += __popcll(km);
      while (dm) {
        const int l = __ffsll((long long)dm) - 1;
        dm &= dm - 1;
        const int32_t rec = rdl(rr, l);
        const int64_t g = base + rec;
        const int32_t k = uni(t.user[g]);
        const int64_t cst = uni64(a.cost[g]);
        const int32_t xs = X.find(k, S);
        int64_t unew;
        if (xs >= 0) {
          unew = slot_u(xs) + cst;
          if (unew < kValueLimit) set_key(xs, unew);
        } else {
          unew = uni64(get_u(k)) + cst;
          if (unew < kValueLimit) {
            if (lane == 0) S.u[k] = unew;
            c_u = (w_user == k) ? unew : c_u;
          }
        }
        if (unew >= kValueLimit) {
          code = FS_E_OVERFLOW;
          break;
        }
        if (k == last_exit) last_exit_u = unew;
        if (lane == 0 && a.counter_after) a.counter_after[g] = unew;
        kv_used -= uni(tokens_at(rec));
      }
    }
    n_run = kept;
    n_live = kept;
    min_fin = n_run > 0 ? int64_t(wave_min32(mf)) : INT64_MAX;
  };

  // ---- steps
  while (!overflow && code == 0) {
    if (s >= s_end) break;
    if (nxt == n && nX == 0 && n_live == 0) break;
    if (nxt < n && nxt - wbase >= 64) advance_window();
    if (literal && (nX == 0 || stalled)) {
      // nothing queued, or the queue waits for KV: nothing happens before the next
      // arrival or the next finish
      int64_t target = nxt < n ? int64_t(rdl(w_step, int(nxt - wbase))) : INT64_MAX;
      if (min_fin < target) target = min_fin;
      if (target > s_end) target = s_end;
      if (target > s) {
        s = target;
        if (s >= s_end) break;
      }
    } else if (nX == 0 && nxt < n) {
      // nothing queued: the steps before the next arrival only pay back debt
      int64_t target = rdl(w_step, int(nxt - wbase));
      if (target > s_end) target = s_end;
      if (target > s) {
        const int64_t k = target - s;
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
      if (nxt - wbase == 64) advance_window();
      const int j = int(nxt - wbase);
      if (rdl(w_step, j) > s) break;
      stalled = false;
      const int32_t rec = int32_t(nxt);
      const int32_t k = rdl(w_user, j);
      const int32_t call = rdl(w_call, j);
      const int32_t xs = X.find(k, S);
      const bool in_x = xs >= 0;
      int64_t uk = in_x ? slot_u(xs) : rdl64(c_u, j);
      const int64_t u_before = uk;
      if (!in_x) {  // counter lift for a user with nothing queued
        if (nX == 0) {
          if (last_exit >= 0) uk = uk > last_exit_u ? uk : last_exit_u;
        } else {
          uk = uk > minX ? uk : minX;
        }
      }
      bool blocked;
      int32_t why;
      if (call > 0 && !e_blind) {
        blocked = rdl(c_head_blk, j) != 0;
        why = 3;
      } else if (call > 0 && rdl(c_prev_drop, j) != 0) {
        blocked = true;  // interaction-blind limits: an earlier call of it was dropped
        why = 3;
      } else {
        why = rdl(w_reason, j);
        blocked = backlog > theta && why != 0;
      }
      const int32_t tok = rdl(w_tok, j);
      if (!blocked) {
        if (!enqueue(rec, k, call, rdl(w_prev, j), rdl(w_succ, j), tok, rdl64(w_cost, j), xs, uk,
                     rdl(c_prev_adm, j) != 0, rdl(w_seg, j), rdl(c_pe, j))) {
          overflow = true;  // state is as before this arrival
          break;
        }
        if (code) break;
        if (!in_x && nX == 1) minX = uk;
        backlog += tok;
      } else {
        o_st = lane == j ? why : o_st;
        if (!in_x && uk != u_before) {
          if (lane == 0) S.u[k] = uk;
          c_u = (w_user == k) ? uk : c_u;
        }
        c_head_blk = (call == 0 && w_head == rec && w_call > 0) ? 1 : c_head_blk;
        c_prev_drop = (w_prev == rec) ? 1 : c_prev_drop;
        if (lane == 0) fate[rec] = int8_t(why);  // read by the first-come choice
      }
      o_coa = lane == j ? uk : o_coa;
      ++nxt;
    }
    if (overflow || code) break;

    // execution stream: admit while the step has budget (literal engine: while the
    // chosen request fits in the free KV cache, or nothing runs)
    int64_t budget = mid ? mid_budget : C + debt;
    mid = false;
    while ((literal || budget > 0) && nX > 0) {
      uint64_t bk;
      int32_t k;
      int32_t x;
      if (!e_fcfs) {
        if (literal && st_x >= 0) {  // the call that did not fit is still the least
          x = st_x;
          bk = st_key;
          k = st_user;
          if (n_live > 0 && kv_used + st_tok > C) {
            stalled = true;
            break;
          }
        } else {
          x = argmin_x(bk, k);
        }
      } else {
        // the earliest queued request: the first arrived record still undecided (a
        // later call waiting for its previous call cannot be it); its user's FIFO head
        // or, for a later call, the user's earliest ready call
        wave_fence();
        int32_t rec = -1;
        while (fcfs_lo < nxt) {
          const int64_t i = fcfs_lo + lane;
          const uint64_t m = __ballot(i < nxt && ld_fresh(fate + i) == -1);
          if (m) {
            rec = int32_t(fcfs_lo + __ffsll((long long)m) - 1);
            fcfs_lo = rec;
            break;
          }
          fcfs_lo += 64;
        }
        if (rec < 0) {
          code = FS_E_STATE;
          break;
        }
        k = uni(t.user[base + rec]);
        x = X.find(k, S);
        if (x < 0) {
          code = FS_E_STATE;
          break;
        }
        const bool later = t.call && uni(t.call[base + rec]) > 0;
        bk = (uint64_t(later ? 0 : 1) << kTierShift) | uint64_t(slot_u(x));
      }
      if (x < 0 || x >= X.cap) {
        code = FS_E_STATE;  // internal bookkeeping error: stop rather than read out of bounds
        break;
      }
      const int64_t uk = int64_t(bk & kValMask);
      int32_t e;
      if ((bk >> kTierShift) == 0) {
        // the user's ready later call with the lowest record index
        int32_t best = INT32_MAX, be = -1, bprev = -1, prevp = -1;
        int32_t walked = 0;
        for (int32_t c = X.get_rh(x); c >= 0 && walked < S.pcap;
             c = uni(RD<G>(&S.e[c].next)), ++walked) {
          const int32_t rc = uni(RD<G>(&S.e[c].rec));
          if (rc < best) {
            best = rc;
            be = c;
            bprev = prevp;
          }
          prevp = c;
        }
        if (be < 0) {
          code = FS_E_STATE;
          break;
        }
        if (literal && n_live > 0) {
          const int32_t tk = uni(RD<G>(&S.e[be].tok));
          if (kv_used + tk > C) {
            stalled = true;
            if (!e_fcfs) {
              st_x = x;
              st_key = bk;
              st_user = k;
              st_tok = tk;
            }
            break;
          }
        }
        e = be;
        const int32_t nx = uni(RD<G>(&S.e[e].next));
        if (bprev < 0)
          X.set_rh(x, nx);
        else if (lane == 0)
          S.e[bprev].next = nx;
        X.set_rdy(x, X.get_rdy(x) - 1);
      } else {
        if (X.get_fh(x) < 0) {
          if (nfree == 0) {
            overflow = true;  // nothing modified for this decision yet
            break;
          }
          if (!refill(x)) {
            code = FS_E_STATE;
            break;
          }
        }
        e = X.get_fh(x);
        if (e < 0 || e >= S.pcap) {
          code = FS_E_STATE;
          break;
        }
        if (literal && n_live > 0) {
          const int32_t tk = uni(RD<G>(&S.e[e].tok));
          if (kv_used + tk > C) {
            stalled = true;
            if (!e_fcfs) {
              st_x = x;
              st_key = bk;
              st_user = k;
              st_tok = tk;
            }
            break;
          }
        }
        const int32_t nx = uni(RD<G>(&S.e[e].next));
        X.set_fh(x, nx);
        if (nx < 0) X.set_ft(x, -1);
      }
      const Entry v = ld_entry<G>(&S.e[e]);
      st_x = -1;  // admitted
      const int32_t left = X.get_q(x) - 1;
      free_e(e);
      X.set_q(x, left);
      budget -= v.tok;
      backlog -= v.tok;
      // literal engine: no charge now; the call runs until its last output token
      const int64_t unew = literal ? uk : uk + v.cost;
      if (unew >= kValueLimit) {
        code = FS_E_OVERFLOW;
        break;
      }
      if (literal) {
        const int32_t lo = uni(t.len_out[base + v.rec]);
        const int64_t fin = s + (lo > 1 ? lo : 1) - 1;
        if (fin >= INT32_MAX) {  // the step count would overflow before it finishes
          code = FS_E_OVERFLOW;
          break;
        }
        if (cm && n_run == kChunkCap) {  // full: drop the dead marks
          compact();
          if (n_run > kChunkCap / 2) {  // too many running for chunk mode
            cm = false;
            cmin = 0xffffffffu;
          }
        }
        if (lane == 0) {
          run_rec[n_run] = v.rec;
          run_fin[n_run] = int32_t(fin);
          if (a.counter_after) a.counter_after[base + v.rec] = -1;  // until it finishes
        }
        if (cm && lane == (n_run >> 6)) cmin = uint32_t(fin) < cmin ? uint32_t(fin) : cmin;
        ++n_run;
        ++n_live;
        kv_used += v.tok;
        min_fin = fin < min_fin ? fin : min_fin;
      }
      ++seq;
      if (lane == 0) fate[v.rec] = 0;  // read by the first-come choice
      d_rec = lane == nd ? v.rec : d_rec;
      d_step = lane == nd ? int32_t(s) : d_step;
      d_cnt = lane == nd ? unew : d_cnt;
      if (++nd == 64) flush_decisions();
      c_prev_adm = (w_prev == v.rec) ? 1 : c_prev_adm;
      int32_t sc = v.succ;
      if (e_blind && sc >= 0 && sc < nxt) {  // interaction-blind limits may have dropped it
        wave_fence();
        if (ld_fresh(fate + sc) > 0) sc = -1;
      }
      if (sc >= 0 && sc < nxt) {
        // the next call arrived while this one was queued: it becomes ready now
        int64_t c1 = v.scost;
        int32_t t1 = v.stok, s1 = v.ssucc;
        if (!v.sv) load_record(sc, c1, t1, s1);
        int32_t sv2 = 0, t2 = 0, s2 = -1;
        int64_t c2 = 0;
        if (s1 >= 0 && s1 < nxt) {  // and the call after it too
          sv2 = 1;
          load_record(s1, c2, t2, s2);
        }
        const int32_t e2 = alloc_e();  // the entry just freed guarantees room
        put_entry(e2, sc, t1, c1, s1, sv2, c2, t2, s2);
        ready_push(x, e2);
      }
      if (left == 0) {
        last_exit = k;
        last_exit_u = unew;
        leave_x(x, k, unew);
      } else {
        set_key(x, unew);
      }
    }
    if (code || overflow) break;
    if (literal) {
      if (min_fin <= s) {
        if (cm)
          finish_chunks();
        else
          finish_calls();
        stalled = false;
      }
      if (code) break;
    } else {
      debt = budget < 0 ? budget : 0;
    }
    if (nX > 0) {
      if (x_dirty) {
        minmax_x(x_mn, x_mx);
        x_dirty = false;
      }
      gap = x_mx - x_mn > gap ? x_mx - x_mn : gap;
      minX = x_mn;
    }
    ++s;
  }

  if (code) raise_err(a.err, code);
  flush_window();
  flush_decisions();
  if (cm && n_run > n_live) compact();  // the saved batch holds live calls only

  // ---- save: counters of queued users back to u; the queue itself is recovered next
  // time from the records that have arrived and are still undecided
  for (int32_t i = 0; i < nX; ++i) {
    const int32_t x = X.slot(i, nX);
    const int32_t k = X.get_user(x);
    const int64_t uval = slot_u(x);
    if (lane == 0) {
      S.u[k] = uval;
      if (S.xslot) S.xslot[k] = -1;
    }
  }
  wave_fence();
  __syncthreads();
  if (!S.users_global)
    for (int32_t k = lane; k < U; k += 64) u_all[k] = S.u[k];
  // lowest record index that may still be queued
  while (low < nxt) {
    const int64_t i = low + lane;
    const bool q = i < nxt && ld_fresh(fate + i) == -1;
    const uint64_t m = __ballot(q);
    if (m) {
      low += __ffsll((long long)m) - 1;
      break;
    }
    low += 64;
  }
  if (low > nxt) low = nxt;
  const bool drained = nxt == n && nX == 0 && n_live == 0;
  if (lane == 0) {
    rs->s = s;
    rs->nxt = nxt;
    rs->debt = debt;
    rs->backlog = backlog;
    rs->seq = seq;
    rs->gap = gap;
    rs->last_exit_u = last_exit_u;
    rs->low = low;
    rs->last_exit = last_exit;
    rs->done = drained ? 1 : 0;
    rs->overflow = overflow ? 1 : 0;
    rs->mid = 0;
    rs->s_end = s_end;
    rs->kv_used = kv_used;
    rs->n_run = n_run;
    if (!overflow) {
      a.steps[r] = s;
      a.decisions[r] = seq;
      a.max_gap[r] = gap;
    }
  }
  wave_fence();
  if (!overflow)
    for (int32_t k = lane; k < U; k += 64)
      a.counter[int64_t(r) * U + k] = S.users_global ? ld_fresh(u_all + k) : u_all[k];
}

// The global-memory form of the same pass (X and the counters in the state buffer).
__device__ __forceinline__ void global_replica_mem(const SchedArgs &a, int32_t r, Store &S,
                                                  const XBlocks &XB, RepState *rs) {
  const int64_t off = a.t.rep_off[r] + r;
  const int32_t cap = int32_t(a.t.rep_off[r + 1] - a.t.rep_off[r]) + 1;
  char *st = a.state;
  const StateLayout &L = a.L;
  XMem X;
  X.cap = cap;
  X.k = reinterpret_cast<uint64_t *>(st + L.xkey) + off;
  X.user = reinterpret_cast<int32_t *>(st + L.xuser) + off;
  X.q = reinterpret_cast<int32_t *>(st + L.xq) + off;
  X.fh = reinterpret_cast<int32_t *>(st + L.xfh) + off;
  X.ft = reinterpret_cast<int32_t *>(st + L.xft) + off;
  X.hh = reinterpret_cast<int32_t *>(st + L.xhh) + off;
  X.ht = reinterpret_cast<int32_t *>(st + L.xht) + off;
  X.sb = reinterpret_cast<int32_t *>(st + L.xsb) + off;
  X.rh = reinterpret_cast<int32_t *>(st + L.xrh) + off;
  X.rdy = reinterpret_cast<int32_t *>(st + L.xrdy) + off;
  S.u = reinterpret_cast<int64_t *>(st + L.u_all) + int64_t(r) * a.t.U;
  S.xslot = reinterpret_cast<int32_t *>(st + L.xslot_all) + int64_t(r) * a.t.U;
  S.users_global = true;
  run_replica<true>(a, S, X, XB, r, false);
  if (threadIdx.x == 0) rs->overflow = 0;
}


// A replica that overflowed on chip (or every replica, with global memory only), resumed
// from the state buffer.  gsm: the work-group's dynamic LDS; tab_lds: the user table and
// counters go there (U * kXLdsBytesPerUser bytes), hblk: block minima of X kept there
// after the table (0: none).  Called by the global-memory kernel, and by on-chip
// instances right after their own pass (the replica continues in the same launch).
// LDS_ONLY: only the LDS-table form is compiled (the caller has checked that it fits);
// EF: as for run_replica.
template <bool LDS_ONLY = false, int EF = -1>
__device__ __forceinline__ void global_replica(const SchedArgs &a, int32_t r, char *gsm, bool tab_lds,
                                               int32_t hblk) {
  RepState *rs = reinterpret_cast<RepState *>(a.state + a.L.reps) + r;
  const int64_t off = a.t.rep_off[r] + r;
  const int32_t cap = int32_t(a.t.rep_off[r + 1] - a.t.rep_off[r]) + 1;
  char *st = a.state;
  const StateLayout &L = a.L;
  Store S;
  S.pcap = cap;
  S.e = reinterpret_cast<Entry *>(st + L.e_all) + off;
  S.e_free = reinterpret_cast<int32_t *>(st + L.e_free) + off;
  XBlocks XB;
  {
    const size_t tab = tab_lds ? size_t(a.t.U) * kXLdsBytesPerUser : 0;
    char *b = gsm + (tab + 15) / 16 * 16;
    const int32_t nb = hblk > 0 ? hblk : 0;
    XB.cap = hblk;
    XB.k = reinterpret_cast<uint64_t *>(b);
    XB.u = reinterpret_cast<uint32_t *>(XB.k + nb);
  }
  if (tab_lds) {  // the table and the counters in LDS
    const int32_t U = a.t.U;
    XLds X;
    X.cap = U;
    S.u = reinterpret_cast<int64_t *>(gsm);
    X.k = reinterpret_cast<uint64_t *>(S.u + U);
    int32_t *p = reinterpret_cast<int32_t *>(X.k + U);
    X.user = p;
    X.q = p += U;
    X.fh = p += U;
    X.ft = p += U;
    X.hh = p += U;
    X.ht = p += U;
    X.sb = p += U;
    X.rh = p += U;
    X.rdy = p += U;
    X.xs = p += U;
    S.xslot = nullptr;
    S.users_global = false;
    run_replica<true, XLds, EF>(a, S, X, XB, r, false);
    if (threadIdx.x == 0) rs->overflow = 0;
    return;
  }
  if constexpr (!LDS_ONLY) global_replica_mem(a, r, S, XB, rs);
}

}  // namespace
}  // namespace fs

// WSC scheduler steps (Alg. 1, monitoring and execution streams) under the
// token-budget step engine: the on-chip kernel, one wavefront per trace replica.
//
// A replica is one dependent chain of arrivals and admissions, so its speed is the
// length of the wave's instruction stream per event.  Everything an event touches
// stays in registers or LDS, and nothing inside an event waits on HBM in the common
// case:
//   slots     one backlogged user per lane (the paper's Q keyed by user): user id,
//             key = tier << 62 | service counter (tier 0 while the user has a ready
//             later call of an incomplete interaction), the number of queued calls,
//             the ordinals of its FIFO of first calls (head, on-chip end, tail), the
//             head request's data, and its number of ready later calls.  The argmin
//             over (key, user id) is one 32-bit DPP minimum over tier << 31 | (u - B),
//             B being the least counter at the last step end, while every u - B fits
//             31 bits (two minimums over the full key otherwise).  A slot's state changes
//             in its own lane, under an exec mask, so an update costs no cross-lane
//             traffic.
//   ready     one ready later call (previous call admitted) per lane: owning slot,
//             record, data.  A user's earliest ready call is a masked DPP minimum,
//             needed only when it has more than one.
//   ring      per slot, the next first calls of the FIFO in LDS; a FIFO longer than
//             the ring continues in the user's segment of the state buffer (one entry
//             per request of the user) and comes back in coalesced refills.  First come,
//             first served keeps every queued call of a user in its FIFO (arrival
//             order is service order, so nothing needs the ready lanes).
//   cache     the data of the most recent arrivals in LDS, by record index, so a
//             later call that waited for its previous call becomes ready without
//             reading HBM.
//   window    the next 64 records, one per lane, with their step, packed request,
//             flags (first call, raw throttle reason, "head throttled", "previous
//             call admitted") and the user's counter; state changes patch it.
//   batch     (literal engine) the running calls in admission order: record, finish
//             step, packed request and user; a step's finishes are found by a wave scan
//             when the earliest finish step is due, charged in admission order, and the
//             batch is compacted in place.
// Outputs of arrivals and admissions are collected one per lane and written 64 at a
// time.  When an on-chip capacity would overflow, the wave stops before the event
// that needs it, saves the replica's state and the global-memory kernel resumes it.
#include <stddef.h>

#include <type_traits>

#include "fs_sched_global.h"

namespace fs {
namespace sched {
namespace {

constexpr int64_t kPackLimit = int64_t(1) << 40;  // costs that fit a packed request
constexpr uint64_t kTokMask = (uint64_t(1) << 24) - 1;
constexpr int kSlots = 64;
constexpr uint32_t kTier1 = 0x40000000u;  // the tier bit in a key's high word
constexpr uint32_t kValHi = 0x3fffffffu;  // the counter's bits in a key's high word
constexpr uint32_t kRelTier1 = 0x80000000u;  // the tier bit of a relative key
constexpr uint32_t kRelMax = 0x7fffffffu;    // largest relative counter (saturated)

// window flags
constexpr int32_t kFirst = 1;        // first call of its interaction
constexpr int32_t kReasonShift = 1;  // bits 1-2: raw throttle reason (0 within limits)
constexpr int32_t kHeadBlk = 8;      // later call whose interaction's first call was throttled
constexpr int32_t kPrevAdm = 16;     // later call whose previous call has been admitted
constexpr int32_t kBig = 32;         // cost too large for a packed request
constexpr int32_t kPrevDrop = 64;    // later call whose previous call was dropped

// A queued request on chip: record, its next call (-1: none), (cost << 24) | tokens.
struct __align__(16) Ent {
  int32_t rec, succ;
  uint32_t lo, hi;
};

// A batch of arrivals, lane-parallel: a user joining Q (its id, counter, segment and
// its batch lanes) and a ready later call (record, next call, packed request, slot).
struct __align__(16) JoinEnt {
  int32_t k;
  uint32_t seg, ulo, uhi, mlo, mhi, pad[2];
};
struct __align__(16) ReadyEnt {
  int32_t rec, succ;
  uint32_t lo, hi;
  int32_t x, pad[3];
};
constexpr size_t kArriveBytes = kSlots * (sizeof(JoinEnt) + sizeof(ReadyEnt) + 4);

__device__ inline Ent mk_ent(int32_t rec, int32_t sc, uint32_t lo, uint32_t hi) {
  Ent e;
  e.rec = rec;
  e.succ = sc;
  e.lo = lo;
  e.hi = hi;
  return e;
}

__device__ inline int32_t ff1(uint64_t m) { return __ffsll((long long)m) - 1; }

// A field of the kernel's argument block, loaded with a scalar load where it is used
// instead of being held in a scalar register for the whole kernel.  The block is the
// kernel's only argument, at the start of the kernarg segment.
template <class T>
__device__ __forceinline__ T arg_at(uint32_t off) {
  __asm__ volatile("" : "+s"(off));
  const __attribute__((address_space(4))) char *k =
      (const __attribute__((address_space(4))) char *)__builtin_amdgcn_kernarg_segment_ptr();
  return *(const __attribute__((address_space(4))) T *)(k + off);
}
#define KARG(f) arg_at<decltype(SchedArgs{}.f)>(uint32_t(offsetof(SchedArgs, f)))

#define STATE(T, field) reinterpret_cast<T *>(KARG(state) + KARG(L.field))

// FCFS: first come, first served; BLIND: interaction-blind limits; LITERAL: the literal
// engine (the engine flags).  LINKS: the trace has interactions of several calls (its
// call, head and prev arrays are set); without them every request is a first call, so
// nothing is ever a ready later call and the interaction bookkeeping compiles away.
template <bool FCFS, bool BLIND, bool LITERAL, bool LINKS>
__device__ __forceinline__ void onchip_replica(const SchedArgs &a, char *smem) {
  const int32_t r = blockIdx.x;
  if (*a.err) return;
  if (!state_header_ok(a)) return;
  if (finish_if_done(a, r)) return;

  const int lane = threadIdx.x;
  const int32_t D = a.oc.ring, M = a.oc.cache;
  const bool ulds = a.oc.users_lds != 0;
  const int32_t U = a.t.U;
  const int ubits = U > 1 ? 32 - __builtin_clz(uint32_t(U - 1)) : 0;  // bits of a user id
  const bool want_coa = a.counter_on_arrival != nullptr;
  const int32_t BQ = LITERAL ? a.oc.batch : 0;
  JoinEnt *const a_join = reinterpret_cast<JoinEnt *>(smem);              // [kSlots]
  ReadyEnt *const a_rdy = reinterpret_cast<ReadyEnt *>(a_join + kSlots);  // [kSlots]
  int32_t *const a_free = reinterpret_cast<int32_t *>(a_rdy + kSlots);    // [kSlots]
  Ent *const ring = reinterpret_cast<Ent *>(smem + kArriveBytes);  // [kSlots][D]
  Ent *const cache = ring + kSlots * D;             // [M]
  Ent *const bat = cache + M;                       // [BQ] rec, finish step, lo, hi
  int32_t *const bat_u = reinterpret_cast<int32_t *>(bat + BQ);  // [BQ] user
  int64_t *const u_lds = reinterpret_cast<int64_t *>(bat_u + BQ);
  // two bytes per user (by the user's low bits) for matching a batch of arrivals
  const int32_t u_tab = a.oc.user_tab;
  uint8_t *const u_rep = reinterpret_cast<uint8_t *>(u_lds + (ulds ? U : 0));
  uint8_t *const u_slot = u_rep + u_tab;
  const int64_t base = a.t.rep_off[r];
  const int32_t n = int32_t(a.t.rep_off[r + 1] - base);
  RepState *const rs = reinterpret_cast<RepState *>(a.state + a.L.reps) + r;
  int64_t *const u_all = reinterpret_cast<int64_t *>(a.state + a.L.u_all) + int64_t(r) * U;

  // ---- scalar state of the replica
  int32_t s = int32_t(uni64(rs->s)), nxt = int32_t(uni64(rs->nxt));
  int32_t low = int32_t(uni64(rs->low)), seq = int32_t(uni64(rs->seq));
  int64_t debt = uni64(rs->debt), backlog = uni64(rs->backlog), gap = uni64(rs->gap);
  int64_t last_exit_u = uni64(rs->last_exit_u);
  int32_t last_exit = uni(rs->last_exit);
  const int64_t s_end = a.n_steps < 0 ? INT64_MAX : int64_t(s) + a.n_steps;
  const int64_t C = a.cap, theta = a.theta;
  constexpr bool fcfs = FCFS, blind = BLIND;
  // literal engine: the running batch and the KV tokens it holds
  int64_t kv_used = LITERAL ? uni64(rs->kv_used) : 0;
  int32_t n_run = LITERAL ? int32_t(uni64(rs->n_run)) : 0;
  // stopped inside a step, or a batch larger than the LDS one: only the global-memory
  // kernel resumes that
  if (uni(rs->mid) || n_run > BQ) {
    if (lane == 0) {
      rs->overflow = 1;
      rs->s_end = s_end;
    }
    return;
  }

  if (ulds)
    for (int32_t k = lane; k < U; k += 64) u_lds[k] = u_all[k];
  // Literal engine: the batch is an array in admission order, [0, n_run), whose finished
  // entries are marked dead (finish step kDeadFin) and removed only when the array is
  // full or saved; n_live entries are alive.  Lane c holds the least finish step of the
  // live entries of chunk c (entries [64c, 64c + 64)), so a step visits only the chunks
  // with a finish due.
  constexpr uint32_t kDeadFin = 0x7fffffffu;
  uint32_t cmin = 0xffffffffu;
  int32_t n_live = n_run;
  int32_t nb0 = n_run;  // entries [nb0, n_run) still wait for their finish step
  bool stalled = false;  // the last admission found no room in the KV cache, nothing changed since
  if (LITERAL && n_run > 0) {
    const int32_t *const rr_ = STATE(const int32_t, run_rec) + base + r;
    const int32_t *const rf_ = STATE(const int32_t, run_fin) + base + r;
    const int32_t *const len_sys = KARG(t.len_sys);
    const int32_t *const len_in = KARG(t.len_in), *const len_out = KARG(t.len_out);
    const int32_t *const user = KARG(t.user);
    const int64_t *const costp = KARG(cost);
    for (int32_t b0 = 0; b0 < n_run; b0 += 64) {
      const int32_t i = b0 + lane;
      uint32_t mf = 0xffffffffu;
      if (i < n_run) {
        const int32_t rec = rr_[i], fin = rf_[i];
        const int64_t g = base + rec;
        const int32_t tok = len_in[g] + len_out[g] + (len_sys ? len_sys[g] : 0);
        const uint64_t pk = (uint64_t(costp[g]) << 24) | uint32_t(tok);
        bat[i] = mk_ent(rec, fin, uint32_t(pk), uint32_t(pk >> 32));
        bat_u[i] = user[g];
        mf = uint32_t(fin);
      }
      const uint32_t m = wave_min32(mf);
      if (lane == (b0 >> 6)) cmin = m;
    }
  }
  __syncthreads();
  // least live finish step of chunk c, into lane c
  auto chunk_min = [&](int32_t c) {
    const int32_t i = c * 64 + lane;
    const uint32_t f = i < n_run ? uint32_t(bat[i].succ) : 0xffffffffu;
    const uint32_t m = wave_min32(f == kDeadFin ? 0xffffffffu : f);
    if (lane == c) cmin = m;
  };
  // removes the dead entries, keeping the admission order
  auto compact = [&]() {
    const uint64_t lt = (uint64_t(1) << lane) - 1;
    int32_t kept = 0;
    for (int32_t b0 = 0; b0 < n_run; b0 += 64) {
      const int32_t i = b0 + lane;
      const bool valid = i < n_run;
      const Ent e = valid ? bat[i] : mk_ent(-1, int32_t(kDeadFin), 0, 0);
      const int32_t ku = valid ? bat_u[i] : -1;
      const bool live = valid && uint32_t(e.succ) != kDeadFin;
      const uint64_t km = __ballot(live);
      if (live) {
        const int32_t to = kept + __popcll(km & lt);
        bat[to] = e;
        bat_u[to] = ku;
      }
      kept += __popcll(km);
    }
    nb0 -= n_run - kept;  // the entries still waiting for their finish step are the last ones
    n_run = kept;
    cmin = 0xffffffffu;
    for (int32_t c = 0; c * 64 < n_run; ++c) chunk_min(c);
  };

  // a user's counter store, as an LDS store or a global one (typed pointers keep the
  // compiler from merging the two into one flat store, which would wait on both paths)
  auto set_u = [&](int32_t k, int64_t v) {
    if (ulds)
      ((__attribute__((address_space(3))) int64_t *)u_lds)[k] = v;
    else
      ((__attribute__((address_space(1))) int64_t *)u_all)[k] = v;
  };
  auto put_u = [&](int32_t k, int64_t v) {
    if (lane == 0) set_u(k, v);
  };

  // ---- slots: one backlogged user per lane
  uint32_t kh = 0xffffffffu, kl = 0xffffffffu;  // key (tier << 62 | counter); free = all ones
  uint32_t k32 = 0xffffffffu;                   // tier << 31 | (counter - B), saturated
  int32_t xu = -1;                              // user id, -1 = free
  int32_t xq = 0;                               // queued calls (first and later)
  int32_t xf = 0, xr = 0, xt = 0;               // FIFO ordinals: head, on-chip end, tail
  uint32_t xsb = 0;                             // the user's segment of first calls
  int32_t xn = 0;                               // ready later calls
  int32_t hrec = -1, hsucc = -1;                // FIFO head request
  uint32_t hlo = 0, hhi = 0;
  uint64_t occ = 0;
  int32_t nX = 0;
  // ---- ready later calls: one per lane
  int32_t p_x = -1, p_rec = INT32_MAX, p_succ = -1;
  uint32_t p_lo = 0, p_hi = 0;
  uint64_t pocc = 0;

  int64_t minX = 0;
  int64_t B = 0;      // base of the relative keys
  bool wide = false;  // some counter is 2^31 - 1 or more above B: compare full keys
  int32_t code = 0;
  bool overflow = false, mid = false;
  int64_t mid_budget = 0;

  auto rel_of = [&](int64_t u) -> uint32_t {
    const int64_t d = u - B;
    if (d < 0 || d >= int64_t(kRelMax)) {
      wide = true;
      return kRelMax;
    }
    return uint32_t(d);
  };
  // Relative keys recomputed from the full keys with base b.
  auto rebase_full = [&](int64_t b) {
    B = b;
    const bool oc = xu >= 0;
    const int64_t d = int64_t((uint64_t(kh & kValHi) << 32) | kl) - b;
    const bool sat = oc && (d < 0 || d >= int64_t(kRelMax));
    const uint32_t rv = sat ? kRelMax : uint32_t(d);
    k32 = oc ? (((kh & kTier1) << 1) | rv) : 0xffffffffu;
    wide = __ballot(sat) != 0;
  };

  // First call (rec, sc, lo, hi) joins the tail of slot x's FIFO: on chip while the
  // FIFO has no part in HBM and the ring has room, else in the user's segment.
  auto fifo_push = [&](int32_t x, int32_t rec, int32_t sc, uint32_t lo, uint32_t hi) {
    if (lane == x) {
      if (xt == xr && xr - xf < D) {
        ring[x * D + (xt & (D - 1))] = mk_ent(rec, sc, lo, hi);
        if (xt == xf) {
          hrec = rec;
          hsucc = sc;
          hlo = lo;
          hhi = hi;
        }
        ++xr;
      } else {
        STATE(Ent, seg_pk)[int64_t(xsb) + xt] = mk_ent(rec, sc, lo, hi);
      }
      ++xt;
    }
  };
  // Slot x's FIFO has nothing left on chip while its segment holds more: one
  // coalesced load moves up to a ring's worth back.
  auto fifo_refill = [&](int32_t x) {
    const int32_t f1 = rdl(xf, x), rr = rdl(xr, x), tt = rdl(xt, x);
    int32_t m = D - (rr - f1);
    if (m > tt - rr) m = tt - rr;
    wave_fence();
    if (lane < m) {
      const Ent v = STATE(Ent, seg_pk)[int64_t(rdlu(xsb, x)) + rr + lane];
      ring[x * D + ((rr + lane) & (D - 1))] = v;
    }
    if (lane == x) xr += m;
  };
  // Slot x gains ready later call (rec, sc, lo, hi); the caller has checked that a
  // ready lane is free.
  auto ready_add = [&](int32_t x, int32_t rec, int32_t sc, uint32_t lo, uint32_t hi) {
    const int32_t l = ff1(~pocc);
    pocc |= uint64_t(1) << l;
    if (lane == l) {
      p_x = x;
      p_rec = rec;
      p_succ = sc;
      p_lo = lo;
      p_hi = hi;
    }
    if (lane == x) {
      ++xn;
      kh &= kValHi;  // tier 0
      k32 &= kRelMax;
    }
  };
  // ---- window of upcoming records, one per lane
  int32_t wbase = nxt, cache_from = nxt, cache_lo = nxt;
  int32_t w_step = INT32_MAX, w_user = -1, w_flags = 0, w_head = -1, w_prev = -1, w_succ = -1;
  uint32_t w_seg = 0, w_lo = 0, w_hi = 0;
  int64_t c_u = 0;
  int32_t o_st = 0;
  int64_t o_coa = 0;
  bool w_wait = false;  // the window holds later calls whose previous call is not admitted
  // window lanes: the slot holding the lane's user (-1: none) and the window lanes of
  // the same user; slots: the window lanes of the slot's user
  int32_t w_slot = -1;
  uint64_t w_gm = 0, xwm = 0;
  // the next window's record fields, loaded one window ahead (while the current window's
  // arrivals and admissions run) and used raw when that window is taken
  struct RawRec {
    int64_t ts, cst;
    int32_t usr, call, hd, pv, li, lo, ls, why, sc;
  };
  RawRec pf{0, 0, -1, 0, -1, -1, 0, 0, 0, 0, -1};
  int32_t pf_at = -1;  // the window base pf was loaded for
  // Slot for user k with counter uk (tier 1, nothing queued yet).
  auto join = [&](int32_t k, int64_t uk, uint32_t sb) -> int32_t {
    const int32_t x = ff1(~occ);
    occ |= uint64_t(1) << x;
    if (nX++ == 0) {
      B = uk;
      wide = false;
    }
    const uint32_t rv = rel_of(uk);
    if (lane == x) {
      k32 = kRelTier1 | rv;
      kh = uint32_t(uint64_t(uk) >> 32) | kTier1;
      kl = uint32_t(uint64_t(uk));
      xu = k;
      xq = 0;
      xf = xr = xt = 0;
      xsb = sb;
      xn = 0;
    }
    const uint64_t km = __ballot(w_user == k);
    w_slot = (w_user == k) ? x : w_slot;
    xwm = lane == x ? km : xwm;
    return x;
  };
  // Data of an arrived record read from the inputs (when it is no longer cached).
  auto load_rec = [&](int32_t i, int32_t &sc, uint32_t &lo, uint32_t &hi) {
    const int64_t g = base + i;
    const int32_t *len_sys = KARG(t.len_sys);
    const int32_t tok =
        KARG(t.len_in)[g] + KARG(t.len_out)[g] + (len_sys ? len_sys[g] : 0);
    const uint64_t pk = (uint64_t(KARG(cost)[g]) << 24) | uint32_t(tok);
    sc = uni(STATE(const int32_t, succ)[base + i]);
    lo = uint32_t(uni(int32_t(uint32_t(pk))));
    hi = uint32_t(uni(int32_t(uint32_t(pk >> 32))));
  };

  // ---- admissions waiting to be written: lane i holds the i-th of nd
  int32_t d_rec = 0, d_step = 0, nd = 0;
  int64_t d_cnt = 0;
  auto flush_decisions = [&]() {
    if (nd == 0) return;
    int8_t *const fate = STATE(int8_t, fate);
    int8_t *const status = KARG(status);
    int32_t *const astep = KARG(admit_step);
    int32_t *const as = KARG(admit_seq);
    int64_t *const ca = KARG(counter_after);
    if (lane < nd) {
      const int64_t g = base + d_rec;
      fate[g] = 0;
      status[g] = 0;
      astep[g] = d_step;
      if (as) as[g] = seq - nd + lane;
      if (ca && !LITERAL) ca[g] = d_cnt;  // (the literal engine writes it at finish)
    }
    nd = 0;
  };

  auto flush_window = [&](int32_t wb) {
    const int32_t done = nxt - wb;
    int8_t *const fate = STATE(int8_t, fate);
    int8_t *const status = KARG(status);
    int32_t *const astep = KARG(admit_step);
    int32_t *const as = KARG(admit_seq);
    int64_t *const ca = KARG(counter_after);
    int64_t *const coa = KARG(counter_on_arrival);
    if (lane < done) {
      const int64_t g = base + wb + lane;
      if (o_st > 0) {
        fate[g] = int8_t(o_st);
        status[g] = int8_t(o_st);
        astep[g] = -1;
        if (as) as[g] = -1;
        if (ca) ca[g] = -1;
      }
      if (coa) coa[g] = o_coa;
    }
    o_st = 0;
  };
  // The window's users matched once per window: per-user tables in LDS, indexed by the
  // user's low bits, give a representative window lane (any lane of the user) and the
  // slot.  Entries taken by a colliding user are rejected by the checks below; a user
  // who lost its entry sends the window to the matching bit by bit.
  auto match_window = [&]() {
    const bool wv = w_user >= 0;
    const uint64_t wvm = __ballot(wv);
    const int32_t hw = w_user & (u_tab - 1), hx = xu & (u_tab - 1);
    if (wv) u_rep[hw] = uint8_t(lane);
    if (xu >= 0) u_slot[hx] = uint8_t(lane);
    wave_fence();
    const int32_t rr = wv ? int32_t(u_rep[hw]) : 64;
    const int32_t xs = wv ? int32_t(u_slot[hw]) : 64;
    const int32_t rx = xu >= 0 ? int32_t(u_rep[hx]) : 64;
    const bool lost = xu >= 0 && int32_t(u_slot[hx]) != lane;
    const int32_t rr_user = __builtin_amdgcn_ds_bpermute((rr & 63) << 2, w_user);
    const int32_t xs_user = __builtin_amdgcn_ds_bpermute((xs & 63) << 2, xu);
    const int32_t rx_user = __builtin_amdgcn_ds_bpermute((rx & 63) << 2, w_user);
    const int32_t rp = (wv && rr < 64 && rr_user == w_user) ? rr : 64;
    const int32_t rxv = (xu >= 0 && rx < 64 && rx_user == xu) ? rx : 64;
    uint64_t g = wvm, m = wvm;
    if (!__ballot(lost || (wv && rp == 64))) {
      w_slot = (wv && xs < 64 && ((occ >> xs) & 1) && xs_user == w_user) ? xs : -1;
      for (int b = 0; b < 6; ++b) {  // lanes match on their representative's bits
        const uint64_t W = __ballot(wv && ((rp >> b) & 1));
        g &= ((rp >> b) & 1) ? W : ~W;
        m &= ((rxv >> b) & 1) ? W : ~W;
      }
      xwm = (xu >= 0 && rxv < 64) ? m : 0;
    } else {
      uint64_t sm = occ;
      for (int b = 0; b < ubits; ++b) {
        const bool wb = (uint32_t(w_user) >> b) & 1u, xb = (uint32_t(xu) >> b) & 1u;
        const uint64_t W = __ballot(wv && wb), S = __ballot(xu >= 0 && xb);
        g &= wb ? W : ~W;
        sm &= wb ? S : ~S;
        m &= xb ? W : ~W;
      }
      w_slot = (wv && sm) ? ff1(sm) : -1;
      xwm = xu >= 0 ? m : 0;
    }
    w_gm = wv ? g : 0;
  };
  // old >= 0: the window that starts at old is done; its outputs are written here (after
  // the new window's dependent loads, or before them with interactions, whose loads read
  // the fates written), so that no wait for those loads also waits for these stores.
  auto load_window = [&](int32_t old) {
    wave_fence();
    const int32_t i = wbase + lane;
    w_step = INT32_MAX;
    w_user = -1;
    w_flags = 0;
    w_head = -1;
    w_prev = -1;
    w_succ = -1;
    w_seg = 0;
    w_lo = w_hi = 0;
    c_u = 0;
    // the argument fields first (scalar loads, one wait), then the records
    struct {
      const int64_t *ts;
      const int32_t *user, *call, *head, *prev, *len_in, *len_sys, *len_out;
    } T = {KARG(t.ts),   KARG(t.user),   KARG(t.call),    KARG(t.head),
           KARG(t.prev), KARG(t.len_in), KARG(t.len_sys), KARG(t.len_out)};
    const int64_t *const costp = KARG(cost);
    const uint8_t *const reason = KARG(reason);
    const int64_t tau = KARG(tau);
    char *const st = KARG(state);
    const size_t o_succ = KARG(L.succ), o_seg = KARG(L.seg_start), o_fate = KARG(L.fate);
    // record ii's fields, raw: no arithmetic on a loaded value here, so that nothing waits
    // for the loads.  Every load is issued (lanes past the last record read the last
    // record, the optional arrays are read at a stand-in address when absent), so the
    // loads form one straight sequence.
    auto fetch = [&](int32_t ii, RawRec &f) {
      const int64_t g = base + (ii < n ? ii : n - 1);
      f.call = LINKS ? T.call[g] : 0;
      f.usr = T.user[g];
      f.ts = T.ts[g];
      f.hd = LINKS ? T.head[g] : ii;
      f.pv = LINKS ? T.prev[g] : -1;
      f.li = T.len_in[g];
      f.lo = T.len_out[g];
      f.ls = (T.len_sys ? T.len_sys : T.len_in)[g];
      f.cst = costp[g];
      f.why = (reason ? reason : reinterpret_cast<const uint8_t *>(T.len_in))[g];
      f.sc = LINKS ? reinterpret_cast<const int32_t *>(st + o_succ)[g] : -1;
    };
    if (LINKS && old >= 0) {
      flush_window(old);
      flush_decisions();
    }
    if (pf_at != wbase) fetch(i, pf);  // (the first window of the call)
    const RawRec c = pf;
    // the loads that depend on a record's user (and, with interactions, on the state of
    // its previous and first calls) are issued before the next window's; the users of
    // every lane are valid ids (checked before the scheduler runs)
    const uint32_t sb = reinterpret_cast<const uint32_t *>(st + o_seg)[int64_t(r) * U + c.usr];
    const int64_t uu = ulds ? u_lds[c.usr] : ld_fresh(u_all + c.usr);
    int8_t pf_fate = -1, hf_fate = -1;
    if (LINKS && i < n && c.call > 0) {
      const int8_t *const fate = reinterpret_cast<const int8_t *>(st + o_fate) + base;
      pf_fate = ld_fresh(fate + c.pv);
      hf_fate = ld_fresh(fate + c.hd);
    }
    if (i < n) {
      const int32_t call = c.call;
      const int32_t usr = c.usr;
      const int64_t ts = c.ts;
      const int32_t hd = c.hd;
      const int32_t pv = c.pv;
      const int32_t tok = c.li + c.lo + (T.len_sys ? c.ls : 0);
      const int64_t cst = c.cst;
      const int32_t why = reason ? c.why : 0;
      const int32_t sc = c.sc;
      int32_t fl = call == 0 ? kFirst : 0;
      if (LINKS && call > 0)
        fl |= (pf_fate == 0 ? kPrevAdm : 0) | ((hf_fate == 1 || hf_fate == 2) ? kHeadBlk : 0) |
              (pf_fate > 0 ? kPrevDrop : 0);
      fl |= (why << kReasonShift) | (cst >= kPackLimit ? kBig : 0);
      const int64_t stp = ts / tau;
      w_step = stp < INT32_MAX ? int32_t(stp) : INT32_MAX;
      w_user = usr;
      w_flags = fl;
      w_head = hd;
      w_prev = pv;
      w_succ = sc;
      w_seg = sb;
      const uint64_t pk = (uint64_t(cst) << 24) | uint32_t(tok);
      w_lo = uint32_t(pk);
      w_hi = uint32_t(pk >> 32);
      c_u = uu;
      cache[i & (M - 1)] = mk_ent(i, sc, w_lo, w_hi);
    }
    // every loaded value is in its register from here on: no later wait on HBM
    __asm__ volatile("" ::"v"(w_step), "v"(w_user), "v"(w_flags), "v"(w_head), "v"(w_prev),
                     "v"(w_succ), "v"(w_seg), "v"(w_lo), "v"(w_hi), "v"(c_u));
    if (!LINKS && old >= 0) {
      flush_window(old);
      flush_decisions();
    }
    // the next window's records, into the registers this window's just left
    pf_at = wbase + 64;
    fetch(pf_at + lane, pf);
    const int32_t lo_ = wbase + 64 - M;
    cache_lo = lo_ > cache_from ? lo_ : cache_from;
    w_wait = LINKS && __ballot(w_user >= 0 && !(w_flags & (kFirst | kPrevAdm))) != 0;
    match_window();
  };
  auto advance_window = [&]() {
    const int32_t old = wbase;
    wbase = nxt;
    load_window(old);
  };

  // All arrivals of the current step in window lanes [j0, j1) at once (a user outside
  // X is lifted to minX, the least counter in X; with X empty the caller sets it to the
  // counter the first arrival joins with).  The overload test of
  // each arrival needs the tokens queued before it: as the queue only grows during
  // the arrivals, the first arrival that finds it above the threshold is found from
  // a prefix sum taken as if none were throttled, and every later arrival of the
  // step finds it above too.  Returns false, having changed nothing, when an
  // on-chip capacity might not suffice (the arrivals then go one at a time).
  auto arrive_batch = [&](int32_t j0, int32_t j1) -> bool {
    const bool inb = lane >= j0 && lane < j1;
    const bool first = !LINKS || (w_flags & kFirst) != 0;
    const int32_t why = (w_flags >> kReasonShift) & 3;
    const uint32_t tok = w_lo & uint32_t(kTokMask);
    bool bf = false;  // a first call throttled (over a limit while the system is overloaded)
    if (__ballot(inb && first && why != 0)) {
      const uint32_t c0 = (inb && (first || !(w_flags & kHeadBlk))) ? tok : 0u;
      const uint32_t excl = wave_incl_scan32(c0) - c0;
      const int64_t thr = theta - backlog;  // overloaded at a lane iff excl > thr
      const bool ovl =
          thr < 0 ? true : (thr >= int64_t(INT32_MAX) ? false : excl > uint32_t(thr));
      bf = inb && first && ovl && why != 0;
    }
    // a later call shares its first call's fate: throttled before the batch or in it
    bool hb_new = false;
    if (__ballot(bf)) {
      const int32_t hl = w_head - wbase;
      const bool hl_in = hl >= j0 && hl < j1;
      const int hb_src = __builtin_amdgcn_ds_bpermute((hl_in ? hl : lane) << 2, bf ? 1 : 0);
      hb_new = !first && w_head >= 0 && hl_in && hb_src != 0;
    }
    const bool bl = inb && !first && ((w_flags & kHeadBlk) || hb_new);
    const bool blk = bf || bl;
    const uint64_t ub = __ballot(inb && !blk);
    const uint64_t rdym =
        (fcfs || !LINKS) ? 0 : __ballot(inb && !blk && !first && (w_flags & kPrevAdm));
    if (__ballot(inb && !blk && (w_flags & kBig)) || __popcll(ub) > kSlots - nX ||
        __popcll(rdym) > kSlots - __popcll(pocc))
      return false;
    w_flags |= hb_new ? kHeadBlk : 0;
    o_st = inb ? (bf ? why : (bl ? 3 : 0)) : o_st;
    backlog += int64_t(wave_sum32(inb && !blk ? tok : 0u));
    // same: batch lanes with this lane's user; x0: the slot holding this lane's user;
    // mx: batch lanes with this slot's user
    const uint64_t lt = (uint64_t(1) << lane) - 1;
    const uint64_t inbm = __ballot(inb);
    const uint64_t same = w_gm & inbm;
    uint64_t mx = xwm & inbm;
    const int32_t x0 = w_slot;
    const int32_t lead = ff1(same);  // the user's first lane in the batch
    const uint64_t newm = __ballot(inb && x0 < 0);
    // users outside Q are lifted to the least counter in Q, on every arrival
    const int64_t lifted = c_u > minX ? c_u : minX;
    const bool is_lead = inb && lane == lead;
    if (is_lead && x0 < 0 && lifted != c_u) {
      set_u(w_user, lifted);
    }
    if (want_coa) {  // (an optional output)
      const int src = (x0 >= 0 ? x0 : lane) << 2;
      const uint32_t sh = uint32_t(__builtin_amdgcn_ds_bpermute(src, int(kh & kValHi)));
      const uint32_t sl = uint32_t(__builtin_amdgcn_ds_bpermute(src, int(kl)));
      const int64_t us = int64_t((uint64_t(sh) << 32) | sl);
      if (inb) o_coa = x0 >= 0 ? us : lifted;
    }
    if (w_user >= 0 && (same & newm)) c_u = lifted;
    // users joining Q, at their first batch lane.  Which slot a user holds changes no
    // result (ties go by user id), so each takes the slot of its own lane when all of
    // those are free, else the i-th takes the i-th free slot.
    const bool jl = is_lead && x0 < 0 && (same & ub) != 0;
    const uint64_t jm = __ballot(jl);
    int32_t xj = x0;
    if (jm && !(jm & occ)) {
      bool sat = false;
      if (jl) {
        const int64_t d = lifted - B;
        sat = d < 0 || d >= int64_t(kRelMax);
        k32 = kRelTier1 | (sat ? kRelMax : uint32_t(d));
        kh = uint32_t(uint64_t(lifted) >> 32) | kTier1;
        kl = uint32_t(uint64_t(lifted));
        xu = w_user;
        xq = 0;
        xf = xr = xt = 0;
        xsb = w_seg;
        xn = 0;
        mx = same;
        xwm = w_gm;
      }
      if (__ballot(sat)) wide = true;
      occ |= jm;
      nX += __popcll(jm);
      // every window lane of a joining user: the slot is its first batch lane
      if (lead >= 0 && ((jm >> lead) & 1)) {
        w_slot = lead;
        xj = lead;
      }
    } else if (jm) {
      const int32_t J = __popcll(jm);
      const bool fr = !((occ >> lane) & 1);
      const int32_t fi = __popcll(~occ & lt);
      if (fr) a_free[fi] = lane;
      const int32_t ji = __popcll(jm & lt);
      if (jl) {
        JoinEnt e;
        e.k = w_user;
        e.seg = w_seg;
        e.ulo = uint32_t(uint64_t(lifted));
        e.uhi = uint32_t(uint64_t(lifted) >> 32);
        e.mlo = uint32_t(w_gm);
        e.mhi = uint32_t(w_gm >> 32);
        a_join[ji] = e;
      }
      wave_fence();
      if (jl) xj = a_free[ji];
      const bool ns = fr && fi < J;  // a slot taken now
      bool sat = false;
      if (ns) {
        const JoinEnt e = a_join[fi];
        const int64_t uk = int64_t((uint64_t(e.uhi) << 32) | e.ulo);
        const int64_t d = uk - B;
        sat = d < 0 || d >= int64_t(kRelMax);
        k32 = kRelTier1 | (sat ? kRelMax : uint32_t(d));
        kh = e.uhi | kTier1;
        kl = e.ulo;
        xu = e.k;
        xq = 0;
        xf = xr = xt = 0;
        xsb = e.seg;
        xn = 0;
        xwm = (uint64_t(e.mhi) << 32) | e.mlo;
        mx = xwm & inbm;
      }
      if (__ballot(sat)) wide = true;
      occ |= __ballot(ns);
      nX += J;
      // every window lane of a joining user takes its slot from its first batch lane
      const int32_t xl = __builtin_amdgcn_ds_bpermute((lead >= 0 ? lead : lane) << 2, xj);
      if (lead >= 0 && ((jm >> lead) & 1)) {
        w_slot = xl;
        xj = xl;
      }
    }
    // per slot: queued calls, first calls for its FIFO (in lane order), ready calls
    const uint64_t F = ub & (fcfs ? ~uint64_t(0) : __ballot(first));
    const bool oc = xu >= 0;
    const uint64_t mF = oc ? (mx & F) : 0, mR = oc ? (mx & rdym) : 0, mU = oc ? (mx & ub) : 0;
    const int32_t cF = __popcll(mF), cR = __popcll(mR), cU = __popcll(mU);
    int32_t ring_n = 0;
    if (cF > 0 && xt == xr) {
      ring_n = xf + D - xr;
      if (ring_n > cF) ring_n = cF;
    }
    if (F) {
      const int src = (((F >> lane) & 1) ? xj : lane) << 2;
      const int32_t tt = __builtin_amdgcn_ds_bpermute(src, xt);
      const uint32_t sb = uint32_t(__builtin_amdgcn_ds_bpermute(src, int(xsb)));
      const int32_t rn = __builtin_amdgcn_ds_bpermute(src, ring_n);
      // the head of a FIFO that was empty: its first pushed call
      const int l0 = mF ? ff1(mF) : lane;
      const int32_t hs = __builtin_amdgcn_ds_bpermute(l0 << 2, w_succ);
      const uint32_t hl = uint32_t(__builtin_amdgcn_ds_bpermute(l0 << 2, int(w_lo)));
      const uint32_t hh = uint32_t(__builtin_amdgcn_ds_bpermute(l0 << 2, int(w_hi)));
      if ((F >> lane) & 1) {
        const int32_t rank = __popcll(same & F & lt);
        const int32_t ord = tt + rank;
        const Ent e = mk_ent(wbase + lane, w_succ, w_lo, w_hi);
        if (rank < rn)
          ring[xj * D + (ord & (D - 1))] = e;
        else
          STATE(Ent, seg_pk)[int64_t(sb) + ord] = e;
      }
      if (cF > 0 && xt == xf) {
        hrec = wbase + l0;
        hsucc = hs;
        hlo = hl;
        hhi = hh;
      }
      xr += ring_n;
      xt += cF;
    }
    xq += cU;
    if (rdym && !(rdym & pocc)) {  // ready later calls, each in the ready lane of its lane
      if ((rdym >> lane) & 1) {
        p_x = xj;
        p_rec = wbase + lane;
        p_succ = w_succ;
        p_lo = w_lo;
        p_hi = w_hi;
      }
      pocc |= rdym;
      if (cR > 0) {
        xn += cR;
        kh &= kValHi;  // tier 0
        k32 &= kRelMax;
      }
    } else if (rdym) {  // or the i-th takes the i-th free ready lane
      const int32_t NR = __popcll(rdym);
      const bool pf = !((pocc >> lane) & 1);
      const int32_t pi = __popcll(~pocc & lt);
      if ((rdym >> lane) & 1) {
        ReadyEnt e;
        e.rec = wbase + lane;
        e.succ = w_succ;
        e.lo = w_lo;
        e.hi = w_hi;
        e.x = xj;
        a_rdy[__popcll(rdym & lt)] = e;
      }
      wave_fence();
      const bool np = pf && pi < NR;
      if (np) {
        const ReadyEnt e = a_rdy[pi];
        p_x = e.x;
        p_rec = e.rec;
        p_succ = e.succ;
        p_lo = e.lo;
        p_hi = e.hi;
      }
      pocc |= __ballot(np);
      if (cR > 0) {
        xn += cR;
        kh &= kValHi;  // tier 0
        k32 &= kRelMax;
      }
    }
    return true;
  };

  // ---- rebuild the queue left by a previous call: arrived records still undecided
  for (int32_t b0 = low; b0 < nxt && !overflow; b0 += 64) {
    const int8_t *const fate = STATE(const int8_t, fate) + base;
    const int32_t i = b0 + lane;
    const bool q = i < nxt && ld_fresh(fate + i) == -1;
    uint64_t m = __ballot(q);
    while (m && !overflow) {
      const int l = ff1(m);
      m &= m - 1;
      const int32_t rec = b0 + l;
      const int64_t g = base + rec;
      const int32_t k = uni(KARG(t.user)[g]);
      const int32_t *const callp = KARG(t.call);
      const int32_t call = callp ? uni(callp[g]) : 0;
      int32_t sc;
      uint32_t lo, hi;
      load_rec(rec, sc, lo, hi);
      const bool padm = !fcfs && call > 0 && ld_fresh(fate + uni(KARG(t.prev)[g])) == 0;
      const uint64_t fm = __ballot(xu == k);
      const bool big = KARG(cost)[g] >= kPackLimit;
      if (big || (fm == 0 && nX == kSlots) || (padm && pocc == ~uint64_t(0))) {
        overflow = true;  // nothing in the state buffer has changed yet
        break;
      }
      int32_t x = ff1(fm);
      if (fm == 0) {
        const int64_t uk = uni64(ulds ? u_lds[k] : ld_fresh(u_all + k));
        const uint32_t sb = uint32_t(uni(int32_t(STATE(const uint32_t, seg_start)[int64_t(r) * U + k])));
        x = join(k, uk, sb);
      }
      if (lane == x) ++xq;
      if (call == 0 || fcfs)
        fifo_push(x, rec, sc, lo, hi);
      else if (padm)
        ready_add(x, rec, sc, lo, hi);
    }
  }
  if (overflow) {
    if (lane == 0) {
      rs->overflow = 1;
      rs->mid = 0;
      rs->s_end = s_end;
    }
    return;
  }
  if (nX > 0) {
    const bool oc = xu >= 0;
    const uint32_t uh = kh & kValHi;
    const uint32_t mh = wave_min32(oc ? uh : 0xffffffffu);
    const uint32_t ml = wave_min32(oc && uh == mh ? kl : 0xffffffffu);
    minX = int64_t((uint64_t(mh) << 32) | ml);
    rebase_full(minX);
  }
  if (nxt < n) load_window(-1);

  // Admissions of a step taken together (traces without interactions, counters the
  // decisions move, least-counter choice).  Every backlogged user's FIFO head is a
  // candidate; in the order of (key, user id) they are the step's admissions until the
  // budget runs out, as long as no user admitted earlier in that order comes back (with
  // its next request, at its charged counter) ahead of the next candidate.  Each user's
  // rank and the tokens ranked before it come from one pass over the occupied lanes; the
  // users that stay give the first rank their return would pre-empt; the ranks before
  // the least of those are admitted lane-parallel.  W: the keys compared are the full
  // ones (some relative key is saturated), else the relative ones.  Returns the number
  // admitted; the sequential loop takes the rest of the step.
  auto batch_admit = [&](int64_t &budget, auto w_tag) -> int32_t {
    constexpr bool W = decltype(w_tag)::value;
    const bool oc = xu >= 0;
    const uint64_t lt_l = (uint64_t(1) << lane) - 1;
    // relative keys: (key, user) in one word; full keys: the key word, then the user
    const uint64_t key = !oc ? ~uint64_t(0)
                         : W ? ((uint64_t(kh) << 32) | kl)
                             : ((uint64_t(k32) << 32) | uint32_t(xu));
    const uint32_t kuser = oc ? uint32_t(xu) : 0xffffffffu;
    auto before = [&](uint64_t ka, uint32_t ua, uint64_t kb, uint32_t ub) {
      return W ? (ka < kb || (ka == kb && ua < ub)) : ka < kb;
    };
    const uint32_t tok = hlo & uint32_t(kTokMask);
    uint32_t rank = 0, pre = 0;
    for (uint64_t om = occ; om; om &= om - 1) {
      const int32_t j = ff1(om);
      const uint64_t kj = (uint64_t(rdlu(uint32_t(key >> 32), j)) << 32) | rdlu(uint32_t(key), j);
      const uint32_t uj = W ? rdlu(kuser, j) : 0u;
      const uint32_t tj = rdlu(tok, j);  // (read by every lane: no branch around it)
      const bool lt = before(kj, uj, key, kuser);
      rank += lt ? 1u : 0u;
      pre += lt ? tj : 0u;
    }
    const bool adm = oc && int64_t(pre) < budget;  // the budget is positive before it
    const int64_t uk = W ? int64_t((uint64_t(kh & kValHi) << 32) | kl) : B + int64_t(k32 & kRelMax);
    const int64_t unew = uk + int64_t(((uint64_t(hhi) << 32) | hlo) >> 24);
    const bool stay = adm && xq > 1;
    const int64_t d = unew - B;
    const bool nsat = d < 0 || d >= int64_t(kRelMax);
    const uint32_t nk = kRelTier1 | (nsat ? kRelMax : uint32_t(d));
    // a stayer's return key, in the form compared
    const uint64_t nkey = W ? (uint64_t(unew) | (uint64_t(kTier1) << 32))
                            : ((uint64_t(nk) << 32) | uint32_t(xu));
    uint32_t cut = uint32_t(64 - nd);  // room left in the output staging
    for (uint64_t sm = __ballot(stay); sm; sm &= sm - 1) {
      const int32_t j = ff1(sm);
      uint32_t cj = rdlu(rank, j) + 1;  // (a saturated return: stop after it, full keys follow)
      if (W || !rdlu(uint32_t(nsat), j)) {
        const uint64_t nkj = (uint64_t(rdlu(uint32_t(nkey >> 32), j)) << 32) | rdlu(uint32_t(nkey), j);
        const uint32_t uj = W ? rdlu(kuser, j) : 0u;
        const uint32_t cnt = uint32_t(__popcll(__ballot(oc && before(key, kuser, nkj, uj))));
        cj = cnt > cj ? cnt : cj;
      }
      cut = cj < cut ? cj : cut;
    }
    const bool fin = adm && rank < cut;
    const uint64_t fm = __ballot(fin);
    if (!fm || __ballot(fin && unew >= kValueLimit)) return 0;
    const int32_t m = __popcll(fm);  // the admitted hold ranks 0 .. m - 1
    // outputs, in admission order, into staging lanes nd .. nd + m - 1: the admitted lane
    // of rank q sends to lane nd + q, the i-th other lane to the i-th lane outside the
    // staging range (a permutation: every lane receives from exactly one)
    const uint32_t oi = uint32_t(__popcll(~fm & lt_l));
    const uint32_t to = fin ? uint32_t(nd) + rank : (oi < uint32_t(nd) ? oi : oi + uint32_t(m));
    const int32_t o_rec = __builtin_amdgcn_ds_permute(int(to << 2), hrec);
    const uint32_t o_lo = uint32_t(__builtin_amdgcn_ds_permute(int(to << 2), int(uint32_t(unew))));
    const uint32_t o_hi =
        uint32_t(__builtin_amdgcn_ds_permute(int(to << 2), int(uint32_t(uint64_t(unew) >> 32))));
    if (lane >= nd && lane < nd + m) {
      d_rec = o_rec;
      d_step = s;
      d_cnt = int64_t((uint64_t(o_hi) << 32) | o_lo);
    }
    const int32_t lastl = ff1(__ballot(fin && rank == uint32_t(m - 1)));  // the last admitted
    const uint32_t used = rdlu(pre + tok, lastl);
    budget -= int64_t(used);
    backlog -= int64_t(used);
    seq += m;
    nd += m;
    // users that leave Q: the last one in admission order is e; counters back to u;
    // window lanes of those users (w_slot is the slot of a lane's user) take the counter
    const bool lv = fin && xq == 1;
    const uint64_t lm = __ballot(lv);
    if (lm) {
      uint32_t q = uint32_t(m - 1);
      int32_t ll = lastl;
      while (!((lm >> ll) & 1)) ll = ff1(__ballot(fin && rank == --q));
      last_exit = rdl(xu, ll);
      last_exit_u = rdl64(unew, ll);
      if (lv) set_u(xu, unew);
      const bool wh = w_slot >= 0 && ((lm >> (w_slot & 63)) & 1);
      const int wsrc = (w_slot >= 0 ? w_slot : lane) << 2;
      const uint32_t wl = uint32_t(__builtin_amdgcn_ds_bpermute(wsrc, int(uint32_t(unew))));
      const uint32_t wh32 = uint32_t(__builtin_amdgcn_ds_bpermute(wsrc, int(uint32_t(uint64_t(unew) >> 32))));
      if (wh) {
        c_u = int64_t((uint64_t(wh32) << 32) | wl);
        w_slot = -1;
      }
      occ &= ~lm;
      nX -= __popcll(lm);
    }
    // users that stay: the next head of the FIFO (refilled from the segment first when
    // its on-chip part is used up) and the key at the charged counter
    if (fin) {
      ++xf;
      --xq;
    }
    for (uint64_t rm = __ballot(stay && fin && xf == xr && xr < xt); rm; rm &= rm - 1)
      fifo_refill(ff1(rm));
    if (stay && fin) {
      if (xf < xt) {
        const Ent v = ring[lane * D + (xf & (D - 1))];
        hrec = v.rec;
        hsucc = v.succ;
        hlo = v.lo;
        hhi = v.hi;
      }
      kh = uint32_t(uint64_t(unew) >> 32) | kTier1;
      kl = uint32_t(uint64_t(unew));
      k32 = nk;
    }
    if (__ballot(stay && fin && nsat)) wide = true;
    if (lv) {
      kh = kl = k32 = 0xffffffffu;
      xu = -1;
      xq = 0;
    }
    if (FS_RARE(nd == 64)) flush_decisions();
    return m;
  };

  // Admissions of a step with one backlogged user (traces without interactions, counters
  // the decisions move, least-counter choice): the user's FIFO in order while the budget
  // lasts, its on-chip part at a time, the entries read once into lanes and taken in a
  // scalar loop (no choice to make).  Returns the number admitted (0: the sequential
  // loop takes over, e.g. to report a counter overflow).
  auto solo_admit = [&](int64_t &budget) -> int32_t {
    const int32_t x = ff1(occ);
    if (rdl(xf, x) == rdl(xr, x) && rdl(xr, x) < rdl(xt, x)) fifo_refill(x);
    const int32_t f0 = rdl(xf, x), q0 = rdl(xq, x);
    int32_t avail = rdl(xr, x) - f0;  // the FIFO's on-chip part
    if (avail > q0) avail = q0;
    if (avail > 64 - nd) avail = 64 - nd;  // room left in the output staging
    if (avail <= 0) return 0;
    const Ent e = lane < avail ? ring[x * D + ((f0 + lane) & (D - 1))] : mk_ent(-1, -1, 0, 0);
    int64_t u = int64_t((uint64_t(rdlu(kh, x) & kValHi) << 32) | rdlu(kl, x));
    int32_t k = 0;
    for (; k < avail && budget > 0; ++k) {
      const uint32_t lo = rdlu(e.lo, k), hi = rdlu(e.hi, k);
      const int64_t unew = u + int64_t(((uint64_t(hi) << 32) | lo) >> 24);
      if (FS_RARE(unew >= kValueLimit)) break;
      const int32_t tok = int32_t(lo & uint32_t(kTokMask));
      const int32_t st = nd + k;
      d_rec = lane == st ? rdl(e.rec, k) : d_rec;
      d_step = lane == st ? s : d_step;
      d_cnt = lane == st ? unew : d_cnt;
      budget -= tok;
      backlog -= tok;
      u = unew;
    }
    if (k == 0) return 0;
    seq += k;
    nd += k;
    if (lane == x) {
      xf += k;
      xq -= k;
    }
    if (q0 == k) {  // the user leaves Q
      const int32_t ku = rdl(xu, x);
      occ = 0;
      nX = 0;
      if (lane == x) {
        kh = kl = k32 = 0xffffffffu;
        xu = -1;
        xq = 0;
      }
      last_exit = ku;
      last_exit_u = u;
      put_u(ku, u);
      c_u = (w_user == ku) ? u : c_u;
      w_slot = (w_user == ku) ? -1 : w_slot;
    } else {
      // the next head (refilled from the segment first when the on-chip part is used
      // up) and the key at the charged counter
      if (FS_RARE((__ballot(xf == xr && xr < xt) >> x) & 1)) fifo_refill(x);
      const uint32_t rv = rel_of(u);
      if (lane == x) {
        const Ent v = ring[x * D + (xf & (D - 1))];
        hrec = v.rec;
        hsucc = v.succ;
        hlo = v.lo;
        hhi = v.hi;
        kh = uint32_t(uint64_t(u) >> 32) | kTier1;
        kl = uint32_t(uint64_t(u));
        k32 = kRelTier1 | rv;
      }
    }
    if (FS_RARE(nd == 64)) flush_decisions();
    return k;
  };

  // Step of the next arrival (nxt < n): its window lane, or, when the window is used up,
  // the first record of the next window, already loaded.  (The window itself advances in
  // one place, the arrivals below, so the next window's registers have one definition in
  // the loop: no copies of them that would wait for their loads.)
  auto next_arrival_step = [&]() -> int32_t {
    const int32_t j = nxt - wbase;
    if (j < 64) return rdl(w_step, j);
    const int64_t stp = rdl64(pf.ts, 0) / KARG(tau);
    return stp < INT32_MAX ? int32_t(stp) : INT32_MAX;
  };

  // ---- steps
  while (true) {
    if (s >= s_end) break;
    if (nxt == n && nX == 0 && n_live == 0) break;
    if (LITERAL) {
      if (nX == 0 || stalled) {
        // nothing queued, or the queue waits for KV: nothing happens before the next
        // arrival or the next finish
        int64_t target = nxt < n ? int64_t(next_arrival_step()) : INT64_MAX;
        const uint32_t mf = wave_min32(cmin);
        if (n_live > 0 && int64_t(mf) < target) target = int64_t(mf);
        if (target > s_end) target = s_end;
        if (target > s) {
          s = target >= int64_t(INT32_MAX) ? INT32_MAX : int32_t(target);
          if (s >= s_end) break;
        }
      }
    } else if (nX == 0 && nxt < n) {
      // nothing queued: the steps before the next arrival only pay back debt
      int64_t target = next_arrival_step();
      if (target > s_end) target = s_end;
      if (target > s) {
        const int64_t k = target - s;
        debt = (k >= (-debt + C - 1) / C) ? 0 : debt + k * C;
        s = int32_t(target);
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
      const int j = nxt - wbase;
      if (rdl(w_step, j) > s) break;
      if (LITERAL) stalled = false;
      // the step's arrivals in this window, together; with Q empty (traces without
      // interactions, a threshold of zero or more) the first arrival cannot be throttled
      // (nothing is queued), joins lifted to the last exit's counter, and is then the
      // least counter in Q, so the others are lifted to it
      if (!blind && (nX > 0 || (!LINKS && theta >= 0))) {
        const uint64_t after = __ballot(w_step > s) & (~uint64_t(0) << j);
        const int32_t j1 = after ? ff1(after) : 64;
        if (j1 - j > 1) {
          bool done;
          if (nX > 0) {
            done = arrive_batch(j, j1);
          } else {
            const int64_t m0 = minX, b0 = B;
            const bool w0 = wide;
            const int64_t u0 = rdl64(c_u, j), l0 = last_exit >= 0 ? last_exit_u : 0;
            minX = u0 > l0 ? u0 : l0;
            B = minX;
            wide = false;
            done = arrive_batch(j, j1);
            if (!done) {  // (nothing changed)
              minX = m0;
              B = b0;
              wide = w0;
            }
          }
          if (done) {
            nxt = wbase + j1;
            if (j1 < 64) break;  // lane j1 arrives in a later step
            continue;
          }
        }
      }
      const int32_t rec = nxt;
      const int32_t k = rdl(w_user, j);
      const int32_t fl = rdl(w_flags, j);
      const uint64_t fm = __ballot(xu == k);
      const int32_t xs = ff1(fm);
      int64_t uk, u_before = 0;
      if (fm) {
        uk = int64_t((uint64_t(rdlu(kh, xs) & kValHi) << 32) | rdlu(kl, xs));
      } else {  // counter lift for a user with nothing queued
        u_before = rdl64(c_u, j);
        const int64_t L = nX > 0 ? minX : (last_exit >= 0 ? last_exit_u : 0);
        uk = u_before > L ? u_before : L;
      }
      bool blocked;
      int32_t why;
      if (!LINKS || (fl & kFirst) || (blind && !(fl & kPrevDrop))) {
        why = (fl >> kReasonShift) & 3;
        blocked = backlog > theta && why != 0;
      } else if (blind) {  // interaction-blind limits: an earlier call of it was dropped
        why = 3;
        blocked = true;
      } else {
        why = 3;
        blocked = (fl & kHeadBlk) != 0;
      }
      if (blocked) {
        o_st = lane == j ? why : o_st;
        if (!fm && uk != u_before) {
          put_u(k, uk);
          c_u = (w_user == k) ? uk : c_u;
        }
        if (fl & kFirst) w_flags |= (w_head == rec && !(w_flags & kFirst)) ? kHeadBlk : 0;
        if (blind) {
          w_flags |= (w_prev == rec) ? kPrevDrop : 0;
          if (lane == 0) cache[rec & (M - 1)].rec = -1;  // dropped
        }
      } else {
        // capacity first: on overflow the state is as before this arrival
        const bool padm = LINKS && !(fl & kFirst) && (fl & kPrevAdm) && !fcfs;
        if (FS_RARE((fl & kBig) || (!fm && nX == kSlots) || (padm && pocc == ~uint64_t(0)))) {
          overflow = true;
          break;
        }
        const int32_t x = fm ? xs : join(k, uk, rdlu(w_seg, j));
        if (!fm && nX == 1) minX = uk;
        const uint32_t lo = rdlu(w_lo, j), hi = rdlu(w_hi, j);
        const int32_t sc = rdl(w_succ, j);
        if (lane == x) ++xq;
        if (!LINKS || (fl & kFirst) || fcfs)
          fifo_push(x, rec, sc, lo, hi);
        else if (padm)
          ready_add(x, rec, sc, lo, hi);
        backlog += int64_t(lo & uint32_t(kTokMask));
      }
      o_coa = lane == j ? uk : o_coa;
      ++nxt;
    }
    if (FS_RARE(overflow)) break;

    // execution stream: admit while the step has budget (literal engine: while the
    // chosen call fits in the free KV cache, or nothing runs)
    int64_t budget = C + debt;
    if (!FCFS && !BLIND && !LITERAL && !LINKS) {
      while (nX > 1 && budget > 0 &&
             (wide ? batch_admit(budget, std::true_type()) : batch_admit(budget, std::false_type())) > 1) {
      }
      while (nX == 1 && budget > 0 && solo_admit(budget) > 0) {
      }
    }
    while ((LITERAL || budget > 0) && nX > 0) {
      // least (key, user id): the ready tier first, then the least counter
      bool cand, tier0;
      int64_t uk;
      int32_t x, l = -1;
      if (fcfs) {
        // first come, first served: the earliest of the FIFO heads (each user's FIFO
        // holds all of its queued calls in arrival order)
        const uint32_t hv = (xu >= 0 && xf < xt) ? uint32_t(hrec) : 0xffffffffu;
        x = ff1(__ballot(hv == wave_min32v(hv)));
        tier0 = false;
        uk = int64_t((uint64_t(rdlu(kh, x) & kValHi) << 32) | rdlu(kl, x));
      } else {
        if (!wide) {
          const uint32_t mv = wave_min32v(k32);
          cand = k32 == mv;
          const uint32_t m = uint32_t(uni(int32_t(mv)));
          tier0 = LINKS && m < kRelTier1;
          uk = B + int64_t(m & kRelMax);
        } else {
          const uint32_t mh = wave_min32(kh);
          const uint32_t ml = wave_min32(kh == mh ? kl : 0xffffffffu);
          cand = kh == mh && kl == ml;
          tier0 = LINKS && mh < kTier1;
          uk = int64_t((uint64_t(mh & kValHi) << 32) | ml);
        }
        const uint64_t eq = __ballot(cand);
        if (FS_RARE(eq & (eq - 1))) {
          const uint32_t um = wave_min32v(cand ? uint32_t(xu) : 0xffffffffu);
          x = ff1(__ballot(cand && uint32_t(xu) == um));
        } else {
          x = ff1(eq);
        }
      }
      int32_t rec, sc;
      uint32_t lo, hi;
      if (tier0) {  // the user's earliest ready later call
        const uint64_t pm = __ballot(p_x == x);
        l = ff1(pm);
        if (FS_RARE(pm & (pm - 1))) {
          const uint32_t e = wave_min32v(p_x == x ? uint32_t(p_rec) : 0xffffffffu);
          l = ff1(__ballot(p_x == x && uint32_t(p_rec) == e));
        }
        rec = rdl(p_rec, l);
        sc = rdl(p_succ, l);
        lo = rdlu(p_lo, l);
        hi = rdlu(p_hi, l);
      } else {  // the head of the user's FIFO of first calls
        rec = rdl(hrec, x);
        sc = rdl(hsucc, x);
        lo = rdlu(hlo, x);
        hi = rdlu(hhi, x);
      }
      bool sc_now = LINKS && !fcfs && sc >= 0 && sc < nxt;  // its next call already arrived
      if (blind && sc_now) {  // interaction-blind limits may have dropped it
        if (sc >= cache_lo)
          sc_now = uni(cache[sc & (M - 1)].rec) >= 0;  // a dropped arrival's entry is marked
        else
          sc_now = ld_fresh(STATE(const int8_t, fate) + base + sc) <= 0;
      }
      if (LITERAL) {
        if (n_live > 0 && kv_used + int64_t(lo & uint32_t(kTokMask)) > C) {
          stalled = true;  // nothing of this admission has happened
          break;
        }
        if (FS_RARE(n_run == BQ)) {
          compact();
          if (n_run == BQ) {
            overflow = mid = true;  // the batch is full on chip: continue in global memory
            mid_budget = budget;
            break;
          }
        }
      }
      if (FS_RARE(sc_now && !tier0 && pocc == ~uint64_t(0))) {
        overflow = mid = true;  // nothing of this admission has happened yet
        mid_budget = budget;
        break;
      }
      const int32_t tok = int32_t(lo & uint32_t(kTokMask));
      // (literal engine: no charge now; the call runs until its last output token)
      const int64_t unew = LITERAL ? uk : uk + int64_t(((uint64_t(hi) << 32) | lo) >> 24);
      if (FS_RARE(unew >= kValueLimit)) {
        code = FS_E_OVERFLOW;
        break;
      }
      budget -= tok;
      backlog -= tok;
      d_rec = lane == nd ? rec : d_rec;
      d_step = lane == nd ? s : d_step;
      d_cnt = lane == nd ? unew : d_cnt;
      ++seq;
      if (LITERAL) {
        // join the batch; its finish step is resolved after the step's admissions
        const int32_t ku = rdl(xu, x);
        if (lane == 0) {
          bat[n_run] = mk_ent(rec, s, lo, hi);
          bat_u[n_run] = ku;
          int64_t *const ca = KARG(counter_after);
          if (ca) ca[base + rec] = -1;  // until it finishes
        }
        ++n_run;
        ++n_live;
        kv_used += tok;
      }
      if (FS_RARE(++nd == 64)) flush_decisions();
      if (LINKS && w_wait) w_flags |= (w_prev == rec) ? kPrevAdm : 0;
      const int32_t q = rdl(xq, x) - 1;
      if (tier0) {
        pocc &= ~(uint64_t(1) << l);
        if (lane == l) p_x = -1;
        if (lane == x) --xn;
      } else {
        if (lane == x) ++xf;
        // the on-chip part of the FIFO is used up and its segment holds more: refill
        if (FS_RARE((__ballot(xf == xr && xr < xt) >> x) & 1)) fifo_refill(x);
        if (lane == x && xf < xt) {
          const Ent v = ring[x * D + (xf & (D - 1))];
          hrec = v.rec;
          hsucc = v.succ;
          hlo = v.lo;
          hhi = v.hi;
        }
      }
      if (sc_now) {
        int32_t s2;
        uint32_t lo2, hi2;
        if (sc >= cache_lo) {
          const Ent e = cache[sc & (M - 1)];
          s2 = uni(e.succ);
          lo2 = uint32_t(uni(int32_t(e.lo)));
          hi2 = uint32_t(uni(int32_t(e.hi)));
        } else {
          load_rec(sc, s2, lo2, hi2);
        }
        ready_add(x, sc, s2, lo2, hi2);
      }
      if (q == 0) {  // the user leaves Q
        const int32_t k = rdl(xu, x);
        occ &= ~(uint64_t(1) << x);
        --nX;
        if (lane == x) {
          kh = kl = k32 = 0xffffffffu;
          xu = -1;
          xq = 0;
        }
        last_exit = k;
        last_exit_u = unew;
        put_u(k, unew);
        c_u = (w_user == k) ? unew : c_u;
        w_slot = (w_user == k) ? -1 : w_slot;
      } else {
        const uint32_t rv = rel_of(unew);
        if (lane == x) {
          --xq;
          kh = uint32_t(uint64_t(unew) >> 32) | ((LINKS && xn > 0) ? 0u : kTier1);
          kl = uint32_t(uint64_t(unew));
          k32 = ((LINKS && xn > 0) ? 0u : kRelTier1) | rv;
        }
      }
    }
    if (LITERAL && nb0 < n_run) {
      // finish steps of this step's admissions (also before a hand-over in the middle
      // of the admissions): one read of their output lengths
      const int32_t *const len_out = KARG(t.len_out);
      bool big = false;
      for (int32_t b0 = nb0; b0 < n_run; b0 += 64) {
        const int32_t i = b0 + lane;
        if (i < n_run) {
          const int32_t lout = len_out[base + bat[i].rec];
          const int64_t fin = int64_t(s) + (lout > 1 ? lout : 1) - 1;
          big = big || fin >= int64_t(kDeadFin);
          bat[i].succ = int32_t(fin);
        }
      }
      for (int32_t c = nb0 >> 6; c * 64 < n_run; ++c) chunk_min(c);
      nb0 = n_run;
      if (FS_RARE(__ballot(big) != 0)) code = FS_E_OVERFLOW;  // the step count would overflow
    }
    if (FS_RARE(overflow || code)) break;
    if (LITERAL) {
      // decode: calls whose last output token falls in step s finish in admission
      // order; each user is charged its call's cost and the call's KV is freed
      uint64_t due = __ballot(cmin <= uint32_t(s));
      if (due) stalled = false;
      int64_t *const ca = KARG(counter_after);
      while (due && !code) {
        const int32_t c = ff1(due);
        due &= due - 1;
        const int32_t i = c * 64 + lane;
        const bool valid = i < n_run;
        const Ent e = valid ? bat[i] : mk_ent(-1, int32_t(kDeadFin), 0, 0);
        const int32_t ku = valid ? bat_u[i] : -1;
        const bool done = valid && e.succ == s;
        if (done) bat[i].succ = int32_t(kDeadFin);
        uint64_t dm = __ballot(done);
        n_live -= __popcll(dm);
        while (dm) {
          const int l = ff1(dm);
          dm &= dm - 1;
          const int32_t rec = rdl(e.rec, l), k = rdl(ku, l);
          const uint32_t elo = rdlu(e.lo, l), ehi = rdlu(e.hi, l);
          const int64_t cst = int64_t(((uint64_t(ehi) << 32) | elo) >> 24);
          const uint64_t fm = __ballot(xu == k);
          int64_t uc;
          if (fm) {  // a queued user: its key moves, its tier stays
            const int32_t xx = ff1(fm);
            uc = int64_t((uint64_t(rdlu(kh, xx) & kValHi) << 32) | rdlu(kl, xx)) + cst;
            if (FS_RARE(uc >= kValueLimit)) {
              code = FS_E_OVERFLOW;
              break;
            }
            const uint32_t rv = rel_of(uc);
            if (lane == xx) {
              kh = uint32_t(uint64_t(uc) >> 32) | (xn > 0 ? 0u : kTier1);
              kl = uint32_t(uint64_t(uc));
              k32 = (xn > 0 ? 0u : kRelTier1) | rv;
            }
          } else {
            uc = uni64(ulds ? u_lds[k] : ld_fresh(u_all + k)) + cst;
            if (FS_RARE(uc >= kValueLimit)) {
              code = FS_E_OVERFLOW;
              break;
            }
            put_u(k, uc);
            c_u = (w_user == k) ? uc : c_u;
          }
          if (k == last_exit) last_exit_u = uc;
          if (lane == 0 && ca) ca[base + rec] = uc;
          kv_used -= int64_t(elo & uint32_t(kTokMask));
        }
        chunk_min(c);
      }
      if (code) break;
      if (n_live == 0) {  // nothing runs: start the array afresh
        n_run = nb0 = 0;
        cmin = 0xffffffffu;
      }
    } else {
      debt = budget < 0 ? budget : 0;
    }
    if (nX > 0) {  // the gap sample, and the least counter for the next arrivals
      const bool oc = xu >= 0;
      if (!wide) {
        const uint32_t rv = k32 & kRelMax;
        uint32_t mnv = oc ? rv : kRelMax, mxv = oc ? rv : 0u;
        wave_minmax32v(mnv, mxv);
        const uint32_t mnr = uint32_t(uni(int32_t(mnv))), mxr = uint32_t(uni(int32_t(mxv)));
        gap = int64_t(mxr - mnr) > gap ? int64_t(mxr - mnr) : gap;
        minX = B + mnr;
        B = minX;  // rebase: the relative keys only shrink
        if (oc) k32 -= mnr;
      } else {
        const uint32_t uh = kh & kValHi;
        uint32_t hv = oc ? uh : 0xffffffffu, hx = oc ? uh : 0u;
        wave_minmax32v(hv, hx);
        const uint32_t mnh = uint32_t(uni(int32_t(hv))), mxh = uint32_t(uni(int32_t(hx)));
        uint32_t lv = oc && uh == mnh ? kl : 0xffffffffu, lx = oc && uh == mxh ? kl : 0u;
        wave_minmax32v(lv, lx);
        const uint32_t mnl = uint32_t(uni(int32_t(lv))), mxl = uint32_t(uni(int32_t(lx)));
        const int64_t mn = int64_t((uint64_t(mnh) << 32) | mnl);
        const int64_t mx = int64_t((uint64_t(mxh) << 32) | mxl);
        gap = mx - mn > gap ? mx - mn : gap;
        minX = mn;
        rebase_full(mn);
      }
    }
    ++s;
  }

  if (code) raise_err(a.err, code);
  flush_window(wbase);
  flush_decisions();

  // ---- save: counters of queued users back to u; the queue itself is rebuilt from
  // the records that have arrived and are still undecided
  while (occ) {
    const int32_t x = ff1(occ);
    occ &= occ - 1;
    put_u(rdl(xu, x), int64_t((uint64_t(rdlu(kh, x) & kValHi) << 32) | rdlu(kl, x)));
  }
  wave_fence();
  __syncthreads();
  if (ulds)
    for (int32_t k = lane; k < U; k += 64) u_all[k] = u_lds[k];
  // lowest record index that may still be queued
  {
    const int8_t *const fate = STATE(const int8_t, fate) + base;
    while (low < nxt) {
      const int32_t i = low + lane;
      const bool q = i < nxt && ld_fresh(fate + i) == -1;
      const uint64_t m = __ballot(q);
      if (m) {
        low += ff1(m);
        break;
      }
      low += 64;
    }
    if (low > nxt) low = nxt;
  }
  if (LITERAL) {  // the running batch goes to the state buffer
    compact();
    int32_t *const rr_ = STATE(int32_t, run_rec) + base + r;
    int32_t *const rf_ = STATE(int32_t, run_fin) + base + r;
    for (int32_t i = lane; i < n_run; i += 64) {
      rr_[i] = bat[i].rec;
      rf_[i] = bat[i].succ;
    }
  }
  const bool drained = nxt == n && nX == 0 && n_live == 0;
  if (lane == 0) {
    rs->kv_used = kv_used;
    rs->n_run = n_run;
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
    rs->mid = mid ? 1 : 0;
    rs->mid_budget = mid_budget;
    rs->s_end = s_end;
    if (!overflow) {
      KARG(steps)[r] = s;
      KARG(decisions)[r] = seq;
      KARG(max_gap)[r] = gap;
    }
  }
  wave_fence();
  if (!overflow) {
    int64_t *const counter = KARG(counter) + int64_t(r) * U;
    for (int32_t k = lane; k < U; k += 64) counter[k] = ulds ? u_lds[k] : ld_fresh(u_all + k);
  }
}

// One replica per work-group (one wave).  With the engine's policy flags or the literal
// engine, whose queues outgrow the chip on the comparison workloads, a replica of a
// trace with interactions that is handed over continues in the global-memory pass in
// the same launch when that pass's user table fits in this work-group's LDS (its
// on-chip state is in the state buffer by then), so that a replica's two passes follow
// each other rather than every replica's on-chip pass finishing before any global pass
// starts.
template <bool FCFS, bool BLIND, bool LITERAL, bool LINKS>
__global__ void __launch_bounds__(64) k_schedule_onchip(SchedArgs a) {
  extern __shared__ __align__(16) char smem[];
  onchip_replica<FCFS, BLIND, LITERAL, LINKS>(a, smem);
  if constexpr ((FCFS || BLIND || LITERAL) && LINKS) {
    // the arguments read afresh through an opaque offset, so that no value of the on-chip
    // pass stays live into this one (scalar registers are the on-chip pass's bottleneck)
    uint32_t off0 = 0;
    __asm__ volatile("" : "+s"(off0));
    const __attribute__((address_space(4))) char *kp =
        (const __attribute__((address_space(4))) char *)__builtin_amdgcn_kernarg_segment_ptr();
    const SchedArgs &ka = *(const SchedArgs *)(const __attribute__((address_space(4))) SchedArgs *)(kp + off0);
    if (!ka.oc.inl_glds) return;  // (the global-memory kernel resumes it)
    const int32_t r = blockIdx.x;
    wave_fence();
    if (uni(ld_fresh(ka.err))) return;
    if (!state_header_ok(ka)) return;
    const RepState *rs = reinterpret_cast<const RepState *>(ka.state + ka.L.reps) + r;
    if (!uni(ld_fresh(&rs->overflow))) return;
    __syncthreads();
    global_replica<true, (FCFS ? 1 : 0) | (BLIND ? 2 : 0) | (LITERAL ? 4 : 0)>(ka, r, smem, true,
                                                                          ka.oc.inl_hblk);
  }
}

int max_lds_per_block() {
  static int cached = 0;
  if (cached == 0) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess ||
        v <= 0)
      v = 65536;
    cached = v;
  }
  return cached;
}

}  // namespace

OnchipCfg onchip_config(int32_t R, int32_t U, bool literal) {
  // enough LDS per work-group for all replicas to be resident at once (up to four
  // work-groups, i.e. one wave per SIMD, on each of the 256 CUs)
  const int per_cu = R <= 256 ? 1 : R <= 512 ? 2 : R <= 768 ? 3 : 4;
  size_t budget = size_t(160 * 1024) / per_cu - 1024;
  const size_t dev_max = size_t(max_lds_per_block());
  if (budget > dev_max) budget = dev_max;
  OnchipCfg c;
  // literal engine: a quarter for the running batch (20 bytes a call), at most 4096
  int batch = 0;
  if (literal) {
    batch = 4096;
    while (batch > 64 && size_t(batch) * (sizeof(Ent) + 4) > budget / 4) batch >>= 1;
  }
  c.batch = batch;
  c.glds = 0;
  c.hblk = 0;
  const size_t bat_bytes = size_t(batch) * (sizeof(Ent) + 4);
  c.users_lds = size_t(U) * 8 <= budget / 4 ? 1 : 0;
  const size_t users = c.users_lds ? size_t(U) * 8 : 0;
  int tab_n = 64;  // power of two, at least U up to 4096
  while (tab_n < U && tab_n < 4096) tab_n <<= 1;
  c.user_tab = tab_n;
  const size_t tab = size_t(tab_n) * 2;
  size_t left = budget - kArriveBytes - users - bat_bytes - tab;
  // about half for the rings, the rest for the arrival cache
  int ring = 64;
  while (ring > 8 && size_t(kSlots) * ring * sizeof(Ent) > left / 2) ring >>= 1;
  left -= size_t(kSlots) * ring * sizeof(Ent);
  int cache = 4096;
  while (cache > 64 && size_t(cache) * sizeof(Ent) > left) cache >>= 1;
  c.ring = ring;
  c.cache = cache;
  c.lds_bytes = kArriveBytes + size_t(kSlots) * ring * sizeof(Ent) + size_t(cache) * sizeof(Ent) +
                bat_bytes + users + tab;
  return c;
}

template <bool FCFS, bool BLIND, bool LITERAL, bool LINKS>
void launch_links(const SchedArgs &a, hipStream_t s) {
  const void *k = reinterpret_cast<const void *>(&k_schedule_onchip<FCFS, BLIND, LITERAL, LINKS>);
  if (a.oc.lds_bytes > 65536)
    (void)hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, int(a.oc.lds_bytes));
  hipLaunchKernelGGL((k_schedule_onchip<FCFS, BLIND, LITERAL, LINKS>), dim3(a.t.R), dim3(64),
                     a.oc.lds_bytes, s, a);
}

template <bool FCFS, bool BLIND, bool LITERAL>
void launch_mode(const SchedArgs &a, hipStream_t s) {
  a.t.call ? launch_links<FCFS, BLIND, LITERAL, true>(a, s)
           : launch_links<FCFS, BLIND, LITERAL, false>(a, s);
}

template <bool LITERAL>
void launch_engine(const SchedArgs &a, hipStream_t s) {
  if (a.fcfs)
    a.blind ? launch_mode<true, true, LITERAL>(a, s) : launch_mode<true, false, LITERAL>(a, s);
  else
    a.blind ? launch_mode<false, true, LITERAL>(a, s) : launch_mode<false, false, LITERAL>(a, s);
}

void launch_onchip(const SchedArgs &a, hipStream_t s) {
  a.literal ? launch_engine<true>(a, s) : launch_engine<false>(a, s);
}

}  // namespace sched
}  // namespace fs

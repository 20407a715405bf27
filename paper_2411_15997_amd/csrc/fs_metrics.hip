// Per-replica fairness and served-experience metrics (Sec. 5 definitions: service
// provided for requests and interactions, served users, delayed users, aborted
// interactions and wasted tokens) plus Jain's index of the charged service.
// Integer accumulation only (atomics on integers are order-independent, so the
// result is deterministic); Jain's sums are exact 128-bit before the fp64 division.
// Each replica's total charged service is also summed exactly (the low and high 32-bit
// halves of every admitted cost in two 64-bit counters): at 2^62 or more the call
// reports an overflow, and below that no per-user sum can wrap.
#include "fs_device.h"
#include "fs_launch.h"

namespace fs {
namespace {

enum : int {
  C_ADMITTED, C_THROTTLED, C_INTERACTIONS, C_FULL, C_ABORTED, C_WASTED,
  C_COST_LO,  // sum of the low 32 bits of the admitted costs
  C_COST_HI,  // sum of their high bits (costs are below 2^62)
  C_NUM = 8
};
enum : uint32_t { U_HAS = 1, U_FULL = 2, U_DELAYED = 4 };
enum : uint32_t { I_SERVED = 1, I_UNSERVED = 2 };

size_t up(size_t x) { return (x + 255) / 256 * 256; }

struct MLayout {
  size_t charged, uflags, iflags, counters, total;
};

MLayout mlayout(const fs_trace *t) {
  MLayout L;
  size_t ru = size_t(t->n_replicas) * size_t(t->n_users);
  size_t n = size_t(t->rep_off_h[t->n_replicas]);
  size_t o = 0;
  L.charged = o; o += up(ru * 8);
  L.uflags = o; o += up(ru * 4);
  L.iflags = o; o += up((n > 0 ? n : 1) * 4);
  L.counters = o; o += up(size_t(t->n_replicas) * C_NUM * 8);
  L.total = o;
  return L;
}

struct MArgs {
  DevTrace t;
  const int64_t *cost;
  const int8_t *status;
  const int32_t *admit_step;
  const int64_t *max_gap;
  int64_t tau;
  int32_t D;
  unsigned long long *charged;
  uint32_t *uflags, *iflags;
  unsigned long long *counters;
  fs_metrics m;
  int32_t *err;
};

__global__ void k_m_zero(MArgs a, int64_t RU, int64_t N) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < RU; i += stride) {
    a.charged[i] = 0;
    a.uflags[i] = 0;
  }
  if (a.t.call)  // (only later calls add interaction flags)
    for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < N; i += stride)
      a.iflags[i] = 0;
  for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < int64_t(a.t.R) * C_NUM;
       i += stride)
    a.counters[i] = 0;
}

__device__ inline bool first_call(const DevTrace &t, int64_t g) { return !t.call || t.call[g] == 0; }

// An interaction's flags: its later calls OR theirs into iflags[first call]; the first
// call's own flag comes from its status where it is read, which spares one atomic per
// interaction.
__device__ inline uint32_t own_iflag(int8_t st) { return st == 0 ? I_SERVED : I_UNSERVED; }

// The flags that the later calls of the interaction starting at g added (none, and
// the array is not cleared, when every record is a single-call interaction).
__device__ inline uint32_t later_iflags(const MArgs &a, int64_t g) {
  return a.t.call ? a.iflags[g] : 0u;
}

// admit_step - ts / tau > D.  For ts >= 0 the quotient is a floor, so this holds iff
// ts < (admit_step - D) * tau, which needs no division while the product fits.
__device__ inline bool is_delayed(int32_t astep, int64_t ts, int64_t tau, int32_t D) {
  if (ts >= 0 && tau <= (int64_t(1) << 30)) return ts < (int64_t(astep) - D) * tau;
  return int64_t(astep) - ts / tau > D;
}

__device__ inline unsigned long long wave_sum(unsigned long long v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    unsigned long long o = (unsigned long long)__shfl_xor((long long)v, m, 64);
    v += o;
  }
  return v;
}
__device__ inline uint32_t wave_or(uint32_t v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v |= uint32_t(__shfl_xor(int(v), m, 64));
  return v;
}

// Per-key aggregation within a wave before touching global memory: heavy users
// repeat many times in a wave, and all lanes usually share one replica.
// For each distinct key among the active lanes: one atomic add (and one atomic or).
__device__ inline void wave_add_by_key(bool active, int64_t key, unsigned long long v,
                                       unsigned long long *sum_base, uint32_t f,
                                       uint32_t *or_base) {
  const int lane = threadIdx.x & 63;
  uint64_t pending = __ballot(active);
  while (pending) {
    const int leader = __ffsll((long long)pending) - 1;
    const int64_t kl = __shfl(key, leader, 64);
    const bool mine = active && key == kl;
    const unsigned long long total = wave_sum(mine ? v : 0ull);
    const uint32_t flags = or_base ? wave_or(mine ? f : 0u) : 0u;
    if (lane == leader) {
      if (total) atomicAdd(sum_base + kl, total);
      if (or_base && flags) atomicOr(or_base + kl, flags);
    }
    pending &= ~__ballot(mine);
  }
}

// The same for keys that are mostly distinct within a wave (users): lanes of one key
// find a representative lane through a per-wave hash table in LDS (any lane of the key
// wins the slot), add into its LDS accumulator, and the representative issues one
// atomic.  A lane whose key lost its slot to another key updates its own key.
constexpr int kKeyTab = 1024;  // hash slots per wave
struct KeyScratch {
  uint8_t tab[kKeyTab];
  unsigned long long acc[64];
  uint32_t accf[64];
};
// (skip_set: read the flags first and skip the atomic when they are already set.)
__device__ inline void wave_add_by_key_hashed(bool active, int64_t key, unsigned long long v,
                                              unsigned long long *sum_base, uint32_t f,
                                              uint32_t *or_base, KeyScratch &ks,
                                              bool skip_set = false) {
  const int lane = threadIdx.x & 63;
  const uint32_t h = (uint32_t(uint64_t(key)) * 2654435761u) >> 22;  // 10 bits
  if (active) ks.tab[h] = uint8_t(lane);
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  const int rp = active ? int(ks.tab[h]) : lane;
  const int64_t rk = __shfl(key, rp, 64);
  const bool own = active && rk == key;
  const bool lead = own && rp == lane;
  if (lead) {
    ks.acc[lane] = 0;
    ks.accf[lane] = 0;
  }
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  if (own) {
    if (v) atomicAdd(&ks.acc[rp], v);
    if (or_base && f) atomicOr(&ks.accf[rp], f);
  }
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  if (lead) {
    const unsigned long long t = ks.acc[lane];
    const uint32_t fl = ks.accf[lane];
    if (t) atomicAdd(sum_base + key, t);
    if (or_base && fl && !(skip_set && (or_base[key] & fl) == fl)) atomicOr(or_base + key, fl);
  } else if (active && !own) {
    if (v) atomicAdd(sum_base + key, v);
    if (or_base && f && !(skip_set && (or_base[key] & f) == f)) atomicOr(or_base + key, f);
  }
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
}

// Up to three small per-replica counts (each below 2^16 in a wave) in one reduction:
// counters[r * C_NUM + c_i] += x_i for each distinct replica r of the active lanes.
__device__ inline void wave_count3(bool active, int32_t r, unsigned long long *counters,
                                   int c0, uint32_t x0, int c1, uint32_t x1, int c2, uint32_t x2) {
  const int lane = threadIdx.x & 63;
  uint64_t pending = __ballot(active);
  while (pending) {
    const int leader = __ffsll((long long)pending) - 1;
    const int32_t rl = __shfl(r, leader, 64);
    const bool mine = active && r == rl;
    const unsigned long long packed =
        mine ? (uint64_t(x0) | (uint64_t(x1) << 16) | (uint64_t(x2) << 32)) : 0ull;
    const unsigned long long total = wave_sum(packed);
    if (lane == leader) {
      unsigned long long *cr = counters + int64_t(rl) * C_NUM;
      const unsigned long long t0 = total & 0xffffu, t1 = (total >> 16) & 0xffffu,
                               t2 = (total >> 32) & 0xffffu;
      if (c0 >= 0 && t0) atomicAdd(cr + c0, t0);
      if (c1 >= 0 && t1) atomicAdd(cr + c1, t1);
      if (c2 >= 0 && t2) atomicAdd(cr + c2, t2);
    }
    pending &= ~__ballot(mine);
  }
}

// An admitted cost as charged service: in [0, 2^62), else a range error (not added).
__device__ inline bool cost_ok(int64_t c) { return c >= 0 && c < kValueLimit; }

// The exact per-replica total of the admitted costs: the low and high 32-bit halves of
// each cost summed separately (neither sum can wrap: fewer than 2^31 records).
__device__ inline void wave_cost2(bool active, int32_t r, unsigned long long *counters,
                                  int64_t c) {
  const int lane = threadIdx.x & 63;
  uint64_t pending = __ballot(active && c != 0);
  while (pending) {
    const int leader = __ffsll((long long)pending) - 1;
    const int32_t rl = __shfl(r, leader, 64);
    const bool mine = active && r == rl;
    const unsigned long long lo = wave_sum(mine ? (uint64_t(c) & 0xffffffffull) : 0ull);
    const unsigned long long hi = wave_sum(mine ? (uint64_t(c) >> 32) : 0ull);
    if (lane == leader) {
      unsigned long long *cr = counters + int64_t(rl) * C_NUM;
      if (lo) atomicAdd(cr + C_COST_LO, lo);
      if (hi) atomicAdd(cr + C_COST_HI, hi);
    }
    pending &= ~__ballot(mine);
  }
}

// The replica of record g, walking forward from the replica of the block's first
// record (records of a replica are contiguous, so a block spans few of them).
__device__ inline int32_t replica_from(const int64_t *rep_off, int32_t r0, int64_t g) {
  int32_t r = r0;
  while (__ldg(rep_off + r + 1) <= g) ++r;
  return r;
}

// Pass 1: per record -- validity, user flags, charged service, interaction flags.
__global__ void __launch_bounds__(256) k_m_records(MArgs a) {
  __shared__ KeyScratch ks[4];
  const DevTrace &t = a.t;
  int32_t code = 0;
  // grid-stride over whole waves so that every lane takes part in the wave reductions
  for (int64_t base0 = blockIdx.x * int64_t(blockDim.x); base0 < t.N;
       base0 += int64_t(gridDim.x) * blockDim.x) {
    const int64_t g = base0 + threadIdx.x;
    bool ok = g < t.N;
    int32_t r = 0, k = 0;
    int64_t base = 0, i = 0, h = 0;
    const int32_t r0 = replica_of(t.rep_off, t.R, base0);  // (a uniform search)
    if (ok) {
      r = replica_from(t.rep_off, r0, g);
      base = t.rep_off[r];
      i = g - base;
      k = t.user[g];
      if (k < 0 || k >= t.U || t.app[g] < 0 || t.app[g] >= t.A) {
        code = max(code, int32_t(FS_E_RANGE));
        ok = false;
      }
    }
    if (ok) {
      h = i;
      if (!first_call(t, g)) {
        h = t.head[g];
        if (h < 0 || h >= i) {
          code = max(code, int32_t(FS_E_RANGE));
          ok = false;
        }
      }
    }
    const int8_t st = ok ? a.status[g] : int8_t(-1);
    const bool served = ok && st == 0;
    int64_t cg = served ? a.cost[g] : 0;
    if (!cost_ok(cg)) {
      code = max(code, int32_t(FS_E_RANGE));
      cg = 0;
    }
    uint32_t uf = U_HAS;
    if (served && is_delayed(a.admit_step[g], t.ts[g], a.tau, a.D)) uf |= U_DELAYED;
    if (ok && h != i) atomicOr(a.iflags + base + h, own_iflag(st));
    const int64_t uk = int64_t(r) * t.U + k;
    wave_add_by_key_hashed(ok, uk, (unsigned long long)cg, a.charged, uf, a.uflags,
                           ks[threadIdx.x >> 6]);
    wave_count3(ok, r, a.counters, C_ADMITTED, served ? 1u : 0u, C_THROTTLED,
                (ok && st > 0) ? 1u : 0u, C_INTERACTIONS, (ok && first_call(t, g)) ? 1u : 0u);
    wave_cost2(ok, r, a.counters, cg);
  }
  if (code) raise_err(a.err, code);
}

// Pass 2: per interaction (first call) -- fully served, aborted midway.
__global__ void __launch_bounds__(256) k_m_interactions(MArgs a) {
  __shared__ KeyScratch ks[4];
  const DevTrace &t = a.t;
  for (int64_t base0 = blockIdx.x * int64_t(blockDim.x); base0 < t.N;
       base0 += int64_t(gridDim.x) * blockDim.x) {
    const int64_t g = base0 + threadIdx.x;
    bool ok = g < t.N && first_call(t, g);
    int32_t k = ok ? t.user[g] : 0;
    ok = ok && k >= 0 && k < t.U;
    const int32_t r0 = replica_of(t.rep_off, t.R, base0);
    const int32_t r = ok ? replica_from(t.rep_off, r0, g) : 0;
    const uint32_t f = ok ? (later_iflags(a, g) | own_iflag(a.status[g])) : 0u;
    const bool full = ok && !(f & I_UNSERVED);
    const bool aborted = ok && (f & I_SERVED) && (f & I_UNSERVED);
    // one flag per user and wave; a heavy user has many fully served interactions, so
    // the atomic is skipped once its flag is visible (a stale read only costs an atomic
    // that changes nothing)
    wave_add_by_key_hashed(full, int64_t(r) * t.U + k, 0ull, nullptr, U_FULL, a.uflags,
                           ks[threadIdx.x >> 6], true);
    wave_count3(ok, r, a.counters, C_FULL, full ? 1u : 0u, C_ABORTED, aborted ? 1u : 0u, -1, 0u);
  }
}

// Replicas whose users fit in LDS: a work-group takes kChunk consecutive records and,
// for each replica segment among them, sums the charged service and ORs the user
// flags in LDS tables indexed by user, then adds each touched user's values to global
// memory once.  Per-replica counts are reduced over the work-group.
constexpr int kChunk = 8192;
constexpr int kLdsUsers = 4096;

// Sums three per-thread counts over the work-group (256 threads) and adds them to the
// replica's counters c0, c1, c2 (c < 0: unused).
// (c0b >= 0: x0's total also goes to counter c0b)
__device__ inline void block_count3(uint32_t x0, uint32_t x1, uint32_t x2,
                                    unsigned long long *cr, int c0, int c1, int c2,
                                    unsigned long long (*s_red)[4], int c0b = -1) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const unsigned long long packed =
      uint64_t(x0) | (uint64_t(x1) << 21) | (uint64_t(x2) << 42);  // each at most kChunk
  const unsigned long long tw = wave_sum(packed);
  if (lane == 0) s_red[0][wave] = tw;
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned long long t = s_red[0][0] + s_red[0][1] + s_red[0][2] + s_red[0][3];
    const unsigned long long m = (uint64_t(1) << 21) - 1;
    if (c0 >= 0 && (t & m)) atomicAdd(cr + c0, t & m);
    if (c0b >= 0 && (t & m)) atomicAdd(cr + c0b, t & m);
    if (c1 >= 0 && ((t >> 21) & m)) atomicAdd(cr + c1, (t >> 21) & m);
    if (c2 >= 0 && ((t >> 42) & m)) atomicAdd(cr + c2, (t >> 42) & m);
  }
}

// Adds the work-group's sums of the admitted costs' low and high halves to the
// replica's counters (each block sum is below 2^45).
__device__ inline void block_cost2(unsigned long long lo, unsigned long long hi,
                                   unsigned long long *cr, unsigned long long (*s_red)[4]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const unsigned long long tl = wave_sum(lo), th = wave_sum(hi);
  if (lane == 0) {
    s_red[0][wave] = tl;
    s_red[1][wave] = th;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned long long l = s_red[0][0] + s_red[0][1] + s_red[0][2] + s_red[0][3];
    const unsigned long long h = s_red[1][0] + s_red[1][1] + s_red[1][2] + s_red[1][3];
    if (l) atomicAdd(cr + C_COST_LO, l);
    if (h) atomicAdd(cr + C_COST_HI, h);
  }
}

// Pass 1, LDS tables (U <= kLdsUsers): dynamic LDS of U * 12 bytes.
constexpr int kRecBatch = 4;  // records per thread whose loads are issued together
__global__ void __launch_bounds__(256) k_m_records_lds(MArgs a) {
  extern __shared__ unsigned long long s_dyn[];
  __shared__ unsigned long long s_red[2][4];
  const DevTrace &t = a.t;
  unsigned long long *const s_chg = s_dyn;
  uint32_t *const s_uf = reinterpret_cast<uint32_t *>(s_dyn + t.U);
  const int64_t c0 = blockIdx.x * int64_t(kChunk);
  const int64_t c1 = c0 + kChunk < t.N ? c0 + kChunk : t.N;
  int32_t r = replica_of(t.rep_off, t.R, c0);
  int32_t code = 0;
  for (int64_t s0 = c0; s0 < c1; s0 = t.rep_off[r + 1], ++r) {
    while (t.rep_off[r + 1] <= s0) ++r;  // (empty replicas)
    const int64_t base = t.rep_off[r];
    const int64_t s1 = t.rep_off[r + 1] < c1 ? t.rep_off[r + 1] : c1;
    for (int32_t k = threadIdx.x; k < t.U; k += 256) {
      s_chg[k] = 0;
      s_uf[k] = 0;
    }
    __syncthreads();
    uint32_t n_adm = 0, n_thr = 0, n_int = 0;
    unsigned long long c_lo = 0, c_hi = 0;
    for (int64_t g0 = s0 + threadIdx.x; g0 < s1; g0 += kRecBatch * 256) {
      int32_t uk[kRecBatch], ap[kRecBatch], cl[kRecBatch], hd[kRecBatch], as[kRecBatch];
      int8_t st[kRecBatch];
      int64_t ts[kRecBatch], cs[kRecBatch];
#pragma unroll
      for (int j = 0; j < kRecBatch; ++j) {
        const int64_t g = g0 + j * 256;
        const bool v = g < s1;
        uk[j] = v ? t.user[g] : 0;
        ap[j] = v ? t.app[g] : 0;
        cl[j] = (v && t.call) ? t.call[g] : 0;
        hd[j] = (v && t.call) ? t.head[g] : 0;
        st[j] = v ? a.status[g] : int8_t(-1);
        as[j] = v ? a.admit_step[g] : 0;
        ts[j] = v ? t.ts[g] : 0;
        cs[j] = v ? a.cost[g] : 0;
      }
#pragma unroll
      for (int j = 0; j < kRecBatch; ++j) {
        const int64_t g = g0 + j * 256;
        if (g >= s1) continue;
        const int64_t i = g - base;
        const int32_t k = uk[j];
        bool ok = k >= 0 && k < t.U && ap[j] >= 0 && ap[j] < t.A;
        const bool fc = cl[j] == 0;
        int64_t h = i;
        if (ok && !fc) {
          h = hd[j];
          ok = h >= 0 && h < i;
        }
        if (!ok) {
          code = int32_t(FS_E_RANGE);
          continue;
        }
        const bool served = st[j] == 0;
        uint32_t uf = U_HAS;
        if (served && is_delayed(as[j], ts[j], a.tau, a.D)) uf |= U_DELAYED;
        // without interaction links a served request is a fully served interaction (the
        // interaction pass is not run)
        if (served && !t.call) uf |= U_FULL;
        if (!fc) atomicOr(a.iflags + base + h, own_iflag(st[j]));
        if (served && !cost_ok(cs[j])) {
          code = int32_t(FS_E_RANGE);
        } else if (served && cs[j]) {
          atomicAdd(&s_chg[k], (unsigned long long)cs[j]);
          c_lo += uint64_t(cs[j]) & 0xffffffffull;
          c_hi += uint64_t(cs[j]) >> 32;
        }
        atomicOr(&s_uf[k], uf);
        n_adm += served ? 1u : 0u;
        n_thr += st[j] > 0 ? 1u : 0u;
        n_int += fc ? 1u : 0u;
      }
    }
    __syncthreads();
    unsigned long long *const chg = a.charged + int64_t(r) * t.U;
    uint32_t *const ufg = a.uflags + int64_t(r) * t.U;
    for (int32_t k = threadIdx.x; k < t.U; k += 256) {
      const uint32_t f = s_uf[k];
      if (!f) continue;
      const unsigned long long c = s_chg[k];
      if (c) atomicAdd(chg + k, c);
      if ((ufg[k] & f) != f) atomicOr(ufg + k, f);
    }
    block_count3(n_adm, n_thr, n_int, a.counters + int64_t(r) * C_NUM, C_ADMITTED, C_THROTTLED,
                 C_INTERACTIONS, s_red, t.call ? -1 : int(C_FULL));
    __syncthreads();
    block_cost2(c_lo, c_hi, a.counters + int64_t(r) * C_NUM, s_red);
    __syncthreads();
  }
  if (code) raise_err(a.err, code);
}

// Pass 2, LDS tables (U <= kLdsUsers).
__global__ void __launch_bounds__(256) k_m_interactions_lds(MArgs a) {
  extern __shared__ unsigned long long s_dyn[];
  __shared__ unsigned long long s_red[2][4];
  const DevTrace &t = a.t;
  uint8_t *const s_full = reinterpret_cast<uint8_t *>(s_dyn);
  const int64_t c0 = blockIdx.x * int64_t(kChunk);
  const int64_t c1 = c0 + kChunk < t.N ? c0 + kChunk : t.N;
  int32_t r = replica_of(t.rep_off, t.R, c0);
  for (int64_t s0 = c0; s0 < c1; s0 = t.rep_off[r + 1], ++r) {
    while (t.rep_off[r + 1] <= s0) ++r;
    const int64_t s1 = t.rep_off[r + 1] < c1 ? t.rep_off[r + 1] : c1;
    for (int32_t k = threadIdx.x; k < t.U; k += 256) s_full[k] = 0;
    __syncthreads();
    uint32_t n_full = 0, n_ab = 0;
    for (int64_t g = s0 + threadIdx.x; g < s1; g += 256) {
      if (!first_call(t, g)) continue;
      const int32_t k = t.user[g];
      if (k < 0 || k >= t.U) continue;
      const uint32_t f = later_iflags(a, g) | own_iflag(a.status[g]);
      const bool full = !(f & I_UNSERVED);
      if (full) s_full[k] = 1;  // (the same value from every writer)
      n_full += full ? 1u : 0u;
      n_ab += ((f & I_SERVED) && (f & I_UNSERVED)) ? 1u : 0u;
    }
    __syncthreads();
    uint32_t *const ufg = a.uflags + int64_t(r) * t.U;
    for (int32_t k = threadIdx.x; k < t.U; k += 256)
      if (s_full[k] && !(ufg[k] & U_FULL)) atomicOr(ufg + k, uint32_t(U_FULL));
    block_count3(n_full, n_ab, 0, a.counters + int64_t(r) * C_NUM, C_FULL, C_ABORTED, -1, s_red);
    __syncthreads();
  }
}

// Pass 3: per admitted record of an aborted interaction -- wasted tokens.  Chunked like
// the LDS passes; a replica segment without aborted interactions (every replica under
// the paper's policy) is skipped without reading its records.
__global__ void __launch_bounds__(256) k_m_wasted(MArgs a) {
  __shared__ unsigned long long s_red[1][4];
  const DevTrace &t = a.t;
  const int64_t c0 = blockIdx.x * int64_t(kChunk);
  const int64_t c1 = c0 + kChunk < t.N ? c0 + kChunk : t.N;
  int32_t r = replica_of(t.rep_off, t.R, c0);
  for (int64_t s0 = c0; s0 < c1; s0 = t.rep_off[r + 1], ++r) {
    while (t.rep_off[r + 1] <= s0) ++r;
    const int64_t base = t.rep_off[r];
    const int64_t s1 = t.rep_off[r + 1] < c1 ? t.rep_off[r + 1] : c1;
    unsigned long long *const cr = a.counters + int64_t(r) * C_NUM;
    if (cr[C_ABORTED] == 0) continue;  // (uniform over the work-group)
    unsigned long long w = 0;
    for (int64_t g = s0 + threadIdx.x; g < s1; g += 256) {
      if (a.status[g] != 0) continue;
      const int64_t i = g - base;
      const int64_t h = first_call(t, g) ? i : t.head[g];
      if (h < 0 || h > i) continue;
      const uint32_t f =
          later_iflags(a, base + h) | (h == i ? I_SERVED : own_iflag(a.status[base + h]));
      if ((f & I_SERVED) && (f & I_UNSERVED)) w += (unsigned long long)tokens_of(t, g);
    }
    const unsigned long long tw = wave_sum(w);
    if ((threadIdx.x & 63) == 0) s_red[0][threadIdx.x >> 6] = tw;
    __syncthreads();
    if (threadIdx.x == 0) {
      const unsigned long long tot = s_red[0][0] + s_red[0][1] + s_red[0][2] + s_red[0][3];
      if (tot) atomicAdd(cr + C_WASTED, tot);
    }
    __syncthreads();
  }
}

struct U128 {
  unsigned long long lo, hi;
};
__device__ inline U128 add128(U128 a, U128 b) {
  U128 c;
  c.lo = a.lo + b.lo;
  c.hi = a.hi + b.hi + (c.lo < a.lo ? 1ull : 0ull);
  return c;
}
__device__ inline double to_double(U128 v) {
  return double(v.hi) * 18446744073709551616.0 + double(v.lo);
}

// Pass 4: one block per replica -- Jain's index and the percentages.
__global__ void __launch_bounds__(256) k_m_finish(MArgs a) {
  const int32_t r = blockIdx.x;
  const int32_t U = a.t.U;
  __shared__ U128 s1s[256], s2s[256];
  __shared__ unsigned long long cnt[256][3];
  U128 s1 = {0, 0}, s2 = {0, 0};
  unsigned long long users = 0, full = 0, delayed = 0;
  for (int32_t k = threadIdx.x; k < U; k += blockDim.x) {
    int64_t uk = int64_t(r) * U + k;
    uint32_t f = a.uflags[uk];
    if (!(f & U_HAS)) continue;
    unsigned long long x = a.charged[uk];
    users += 1;
    full += (f & U_FULL) ? 1 : 0;
    delayed += (f & U_DELAYED) ? 1 : 0;
    s1 = add128(s1, U128{x, 0});
    U128 sq{x * x, __umul64hi(x, x)};
    s2 = add128(s2, sq);
  }
  s1s[threadIdx.x] = s1;
  s2s[threadIdx.x] = s2;
  cnt[threadIdx.x][0] = users;
  cnt[threadIdx.x][1] = full;
  cnt[threadIdx.x][2] = delayed;
  __syncthreads();
  for (int w = blockDim.x / 2; w > 0; w >>= 1) {
    if (threadIdx.x < w) {
      s1s[threadIdx.x] = add128(s1s[threadIdx.x], s1s[threadIdx.x + w]);
      s2s[threadIdx.x] = add128(s2s[threadIdx.x], s2s[threadIdx.x + w]);
      for (int c = 0; c < 3; ++c) cnt[threadIdx.x][c] += cnt[threadIdx.x + w][c];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const unsigned long long *C = a.counters + r * C_NUM;
    const int64_t n = a.t.rep_off[r + 1] - a.t.rep_off[r];
    U128 S1 = s1s[0], S2 = s2s[0];
    const unsigned long long nu = cnt[0][0];
    // the exact total charged service: hi * 2^32 + lo
    const unsigned long long lo = C[C_COST_LO], hi = C[C_COST_HI];
    if ((hi >> 30) != 0 || ((hi << 32) + lo) < (hi << 32) ||
        (hi << 32) + lo >= (unsigned long long)kValueLimit)
      raise_err(a.err, FS_E_OVERFLOW);
    double jain = 1.0;
    if (S2.lo != 0 || S2.hi != 0) {
      double d1 = to_double(S1);
      jain = (d1 * d1) / (double(nu) * to_double(S2));
    }
    auto pct = [](unsigned long long x, unsigned long long y) {
      return y == 0 ? 0.0 : 100.0 * double(x) / double(y);
    };
    a.m.jain[r] = jain;
    a.m.max_gap_tokens[r] = double(a.max_gap[r]) / 65536.0;
    a.m.svc_req_pct[r] = pct(C[C_ADMITTED], (unsigned long long)n);
    a.m.svc_int_pct[r] = pct(C[C_FULL], C[C_INTERACTIONS]);
    a.m.served_users_pct[r] = pct(cnt[0][1], nu);
    a.m.delayed_users_pct[r] = pct(cnt[0][2], nu);
    a.m.throttled[r] = int64_t(C[C_THROTTLED]);
    a.m.aborted_midway[r] = int64_t(C[C_ABORTED]);
    a.m.wasted_tokens[r] = int64_t(C[C_WASTED]);
  }
}

int grid_for(int64_t n, int threads) {
  int64_t b = (n + threads - 1) / threads;
  if (b < 1) b = 1;
  if (b > 65536) b = 65536;
  return int(b);
}

}  // namespace

size_t metrics_workspace_bytes(const fs_trace *t) { return mlayout(t).total; }

hipError_t launch_metrics(const fs_trace *t, const int64_t *cost, const fs_outputs *out,
                          const fs_engine *eng, int32_t delay_steps, fs_metrics *m, void *ws,
                          hipStream_t s) {
  MLayout L = mlayout(t);
  char *w = static_cast<char *>(ws);
  MArgs a;
  a.t = dev_trace(t);
  a.cost = cost;
  a.status = out->status;
  a.admit_step = out->admit_step;
  a.max_gap = out->max_gap;
  a.tau = eng->step_us;
  a.D = delay_steps;
  a.charged = reinterpret_cast<unsigned long long *>(w + L.charged);
  a.uflags = reinterpret_cast<uint32_t *>(w + L.uflags);
  a.iflags = reinterpret_cast<uint32_t *>(w + L.iflags);
  a.counters = reinterpret_cast<unsigned long long *>(w + L.counters);
  a.m = *m;
  a.err = out->err;
  const int64_t RU = int64_t(t->n_replicas) * t->n_users;
  const int64_t N = a.t.N;
  hipLaunchKernelGGL(k_m_zero, dim3(grid_for(RU > N ? RU : N, 256)), dim3(256), 0, s, a, RU, N);
  if (N > 0) {
    const int64_t chunks = (N + kChunk - 1) / kChunk;
    if (t->n_users <= kLdsUsers) {
      hipLaunchKernelGGL(k_m_records_lds, dim3(chunks), dim3(256), size_t(t->n_users) * 12, s, a);
      if (t->call)  // (without links the records pass counts the fully served interactions)
        hipLaunchKernelGGL(k_m_interactions_lds, dim3(chunks), dim3(256), size_t(t->n_users), s, a);
    } else {
      hipLaunchKernelGGL(k_m_records, dim3(grid_for(N, 256)), dim3(256), 0, s, a);
      hipLaunchKernelGGL(k_m_interactions, dim3(grid_for(N, 256)), dim3(256), 0, s, a);
    }
    hipLaunchKernelGGL(k_m_wasted, dim3(chunks), dim3(256), 0, s, a);
  }
  hipLaunchKernelGGL(k_m_finish, dim3(t->n_replicas), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace fs

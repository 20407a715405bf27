// Workload analysis of Sec. 3 on the device: each user's requests and tokens per
// minute, overall and per application, as histograms of users over exact log2 bins
// (Fig. 2), the token lengths and interaction sizes per application (Figs. 3-5), and
// the graph-size table (Table 2).  HBM-bound streaming passes; every accumulation is
// an integer atomic (order-independent, so results are deterministic), aggregated per
// wave over the lanes that share a key before it reaches memory.
//   1. k_ws_records   per request: validity, the replica's latest arrival, requests and
//                     tokens per (replica, user, app), the length histograms and sums per
//                     (replica, app) (in LDS per work-group and replica segment), and one
//                     count at the interaction's first call
//   2. k_ws_graph     per request: its interaction's size (the count at its first call)
//                     gives its Table 2 row; first calls add to the size histogram (both
//                     in LDS per work-group and replica segment)
//   3. k_ws_users     per (replica, user) and per (replica, user, app): the rate bins
#include "fs_device.h"
#include "fs_launch.h"

namespace fs {
namespace {

constexpr int kThreads = 256;
constexpr int kRateBins = 128, kLenBins = 32, kSizeBins = 64, kGraphBins = 7;

struct WsArgs {
  DevTrace t;
  int64_t minute_us;
  fs_wstats o;
  unsigned long long *ua_req, *ua_tok;  // [R][U][A] (the outputs when given)
  unsigned int *size;                   // [N] records per first call
  unsigned long long *max_ts;           // [R]
  int32_t *err;
};

__device__ inline unsigned long long wsum64(unsigned long long v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += (unsigned long long)__shfl_xor((long long)v, m, 64);
  return v;
}

// For every distinct key among the active lanes, one atomic per array and wave:
// COUNT: cnt[key] += the number of lanes with the key (c is ignored), else += the sum of
// their c; val (may be null) += the sum of their v.
template <bool COUNT>
__device__ inline void wave_add2(bool active, int64_t key, unsigned long long c,
                                 unsigned long long v, unsigned long long *cnt,
                                 unsigned long long *val) {
  const int lane = threadIdx.x & 63;
  uint64_t pending = __ballot(active);
  while (pending) {
    const int leader = __ffsll((long long)pending) - 1;
    const int64_t kl = __shfl(key, leader, 64);
    const bool mine = active && key == kl;
    const uint64_t mm = __ballot(mine);
    const unsigned long long tc = COUNT ? (unsigned long long)__popcll(mm) : wsum64(mine ? c : 0);
    const unsigned long long tv = val ? wsum64(mine ? v : 0ull) : 0ull;
    if (lane == leader) {
      if (tc) atomicAdd(cnt + kl, tc);
      if (val && tv) atomicAdd(val + kl, tv);
    }
    pending &= ~mm;
  }
}

__device__ inline int len_bin(int64_t L) { return L == 0 ? 0 : 64 - __clzll((long long)L); }

// 64 + floor(log2(x / M)) for x >= 1, M >= 1 (0 for x == 0): the exponents of the
// leading bits, then one comparison at that exponent difference (no shifted value
// reaches 2^64: both are below 2^63).
__device__ inline int rate_bin(uint64_t x, uint64_t M) {
  if (x == 0) return 0;
  const int a = 63 - __clzll((long long)x), b = 63 - __clzll((long long)M);
  const int d = a - b;
  int k;
  if (d >= 0)
    k = (M << d) <= x ? d : d - 1;
  else
    k = (x << (-d)) >= M ? d : d - 1;
  return 64 + k;
}

__device__ inline int graph_bin(uint32_t s) {
  return s <= 1 ? 0 : s <= 10 ? 1 : s <= 20 ? 2 : s <= 30 ? 3 : s <= 40 ? 4 : s <= 50 ? 5 : 6;
}

__device__ inline bool first_of(const DevTrace &t, int64_t g) { return !t.call || t.call[g] == 0; }

__global__ void __launch_bounds__(kThreads) k_ws_zero(WsArgs a, int64_t RUA, int64_t RU) {
  const DevTrace &t = a.t;
  const int64_t stride = int64_t(gridDim.x) * kThreads;
  const int64_t i0 = blockIdx.x * int64_t(kThreads) + threadIdx.x;
  for (int64_t i = i0; i < RUA; i += stride) {
    a.ua_req[i] = 0;
    a.ua_tok[i] = 0;
  }
  // an interaction's size starts at one for its first call; its later calls add to it
  for (int64_t i = i0; i < t.N; i += stride) a.size[i] = (t.call && t.call[i] != 0) ? 0u : 1u;
  const int64_t R = t.R, A = t.A;
  for (int64_t i = i0; i < R; i += stride) a.max_ts[i] = 0;
  for (int64_t i = i0; i < R * (A + 1) * 2 * kRateBins; i += stride) a.o.rate_hist[i] = 0;
  for (int64_t i = i0; i < R * A * 3 * kLenBins; i += stride) a.o.len_hist[i] = 0;
  for (int64_t i = i0; i < R * A * 3; i += stride) a.o.len_sum[i] = 0;
  for (int64_t i = i0; i < R * A * kSizeBins; i += stride) a.o.size_hist[i] = 0;
  for (int64_t i = i0; i < R * kGraphBins * 5; i += stride) a.o.graph[i] = 0;
  (void)RU;
}

// Records are taken in chunks of kChunk consecutive requests per work-group; within a
// chunk, each replica segment accumulates its per-application histograms and sums in
// LDS (when the apps fit, kLdsApps) and adds each nonzero entry to global memory once.
constexpr int kChunk = 8192;
constexpr int kLdsApps = 64;

struct RecLds {
  uint32_t lh[kLdsApps * 3 * kLenBins];     // length histograms [A][3][bins]
  unsigned long long ls[kLdsApps * 3];      // length sums [A][3]
  unsigned long long red[kThreads / 64];    // per-wave maxima
};

template <bool LDS>
__global__ void __launch_bounds__(kThreads) k_ws_records(WsArgs a) {
  __shared__ RecLds sm;
  const DevTrace &t = a.t;
  int32_t code = 0;
  unsigned long long *const lh = reinterpret_cast<unsigned long long *>(a.o.len_hist);
  unsigned long long *const lsum = reinterpret_cast<unsigned long long *>(a.o.len_sum);
  const int64_t c0 = blockIdx.x * int64_t(kChunk);
  const int64_t c1 = c0 + kChunk < t.N ? c0 + kChunk : t.N;
  const int32_t A = t.A;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (LDS) {
    for (int k = threadIdx.x; k < A * 3 * kLenBins; k += kThreads) sm.lh[k] = 0;
    for (int k = threadIdx.x; k < A * 3; k += kThreads) sm.ls[k] = 0;
  }
  int32_t r = c0 < c1 ? replica_of(t.rep_off, t.R, c0) : 0;
  for (int64_t s0 = c0; s0 < c1; s0 = t.rep_off[r + 1], ++r) {
    while (t.rep_off[r + 1] <= s0) ++r;  // (empty replicas)
    const int64_t base = t.rep_off[r];
    const int64_t s1 = t.rep_off[r + 1] < c1 ? t.rep_off[r + 1] : c1;
    __syncthreads();
    unsigned long long mts = 0;
    bool any = false;
    // whole waves step through the segment so that every lane joins the reductions
    for (int64_t w0 = s0; w0 < s1; w0 += kThreads) {
      const int64_t g = w0 + threadIdx.x;
      bool ok = g < s1;
      int32_t u = 0, ap = 0;
      int64_t L[3] = {0, 0, 0}, ts = 0, h = 0;
      if (ok) {
        const int64_t i = g - base;
        u = t.user[g];
        ap = t.app[g];
        ts = t.ts[g];
        L[0] = t.len_in[g];
        L[1] = t.len_sys ? t.len_sys[g] : 0;
        L[2] = t.len_out[g];
        ok = u >= 0 && u < t.U && ap >= 0 && ap < A && ts >= 0 && len_ok(int32_t(L[0])) &&
             len_ok(int32_t(L[1])) && len_ok(int32_t(L[2]));
        h = i;
        if (ok && !first_of(t, g)) {
          h = t.head[g];
          ok = h >= 0 && h < i;
        }
        if (!ok) code = FS_E_RANGE;
      }
      if (ok) {
        mts = (unsigned long long)ts > mts ? (unsigned long long)ts : mts;
        any = true;
      }
      const int64_t tok = L[0] + L[1] + L[2];
      wave_add2<true>(ok, (int64_t(r) * t.U + u) * A + ap, 1ull, (unsigned long long)tok,
                      a.ua_req, a.ua_tok);
#pragma unroll
      for (int x = 0; x < 3; ++x) {
        if (LDS) {
          if (ok) {
            atomicAdd(&sm.lh[(ap * 3 + x) * kLenBins + len_bin(L[x])], 1u);
            if (L[x]) atomicAdd(&sm.ls[ap * 3 + x], (unsigned long long)L[x]);
          }
        } else {
          const int64_t ra = (int64_t(r) * A + ap) * 3 + x;
          wave_add2<true>(ok, ra * kLenBins + len_bin(L[x]), 1ull, 0ull, lh, nullptr);
          wave_add2<false>(ok && L[x] != 0, ra, (unsigned long long)L[x], 0ull, lsum, nullptr);
        }
      }
      if (ok && h != g - base) atomicAdd(a.size + base + h, 1u);
    }
    // the segment's latest arrival, once per work-group
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      const unsigned long long o = (unsigned long long)__shfl_xor((long long)mts, m, 64);
      mts = o > mts ? o : mts;
    }
    const bool any_w = __ballot(any) != 0;
    if (lane == 0) sm.red[wave] = any_w ? mts + 1 : 0;  // 0: no valid request
    __syncthreads();
    if (threadIdx.x == 0) {
      unsigned long long m = 0;
      for (int w = 0; w < kThreads / 64; ++w) m = sm.red[w] > m ? sm.red[w] : m;
      if (m) atomicMax(a.max_ts + r, m - 1);
    }
    if (LDS) {
      for (int k = threadIdx.x; k < A * 3 * kLenBins; k += kThreads) {
        const uint32_t c = sm.lh[k];
        if (c) {
          atomicAdd(lh + int64_t(r) * A * 3 * kLenBins + k, (unsigned long long)c);
          sm.lh[k] = 0;
        }
      }
      for (int k = threadIdx.x; k < A * 3; k += kThreads) {
        const unsigned long long c = sm.ls[k];
        if (c) {
          atomicAdd(lsum + int64_t(r) * A * 3 + k, c);
          sm.ls[k] = 0;
        }
      }
    }
  }
  if (code) raise_err(a.err, code);
}

struct GraphLds {
  uint32_t sh[kLdsApps * kSizeBins];        // size histogram [A][bins]
  unsigned long long gr[kGraphBins * 5];    // Table 2 rows
};

template <bool LDS>
__global__ void __launch_bounds__(kThreads) k_ws_graph(WsArgs a) {
  __shared__ GraphLds sm;
  const DevTrace &t = a.t;
  unsigned long long *const gr = reinterpret_cast<unsigned long long *>(a.o.graph);
  unsigned long long *const sh = reinterpret_cast<unsigned long long *>(a.o.size_hist);
  const int64_t c0 = blockIdx.x * int64_t(kChunk);
  const int64_t c1 = c0 + kChunk < t.N ? c0 + kChunk : t.N;
  const int32_t A = t.A;
  for (int k = threadIdx.x; k < kGraphBins * 5; k += kThreads) sm.gr[k] = 0;
  if (LDS)
    for (int k = threadIdx.x; k < A * kSizeBins; k += kThreads) sm.sh[k] = 0;
  int32_t r = c0 < c1 ? replica_of(t.rep_off, t.R, c0) : 0;
  for (int64_t s0 = c0; s0 < c1; s0 = t.rep_off[r + 1], ++r) {
    while (t.rep_off[r + 1] <= s0) ++r;
    const int64_t base = t.rep_off[r];
    const int64_t s1 = t.rep_off[r + 1] < c1 ? t.rep_off[r + 1] : c1;
    __syncthreads();
    for (int64_t g = s0 + threadIdx.x; g < s1; g += kThreads) {
      const int64_t i = g - base;
      const int32_t u = t.user[g], ap = t.app[g];
      const bool first = first_of(t, g);
      const int64_t h = first ? i : int64_t(t.head[g]);
      const bool ok =
          u >= 0 && u < t.U && ap >= 0 && ap < A && h >= 0 && (first ? h == i : h < i);
      if (!ok) continue;
      const uint32_t sz = a.size[base + h];
      const int b = graph_bin(sz);
      unsigned long long *row = sm.gr + b * 5;
      if (first) atomicAdd(row, 1ull);
      atomicAdd(row + 1, 1ull);
      const int64_t li = t.len_in[g], lo = t.len_out[g], ls = t.len_sys ? t.len_sys[g] : 0;
      if (li) atomicAdd(row + 2, (unsigned long long)li);
      if (lo) atomicAdd(row + 3, (unsigned long long)lo);
      if (ls) atomicAdd(row + 4, (unsigned long long)ls);
      if (first && sz > 0) {
        const int sb = (sz < kSizeBins ? int(sz) : kSizeBins) - 1;
        if (LDS)
          atomicAdd(&sm.sh[ap * kSizeBins + sb], 1u);
        else
          atomicAdd(sh + (int64_t(r) * A + ap) * kSizeBins + sb, 1ull);
      }
    }
    __syncthreads();
    for (int k = threadIdx.x; k < kGraphBins * 5; k += kThreads) {
      const unsigned long long c = sm.gr[k];
      if (c) {
        atomicAdd(gr + int64_t(r) * kGraphBins * 5 + k, c);
        sm.gr[k] = 0;
      }
    }
    if (LDS)
      for (int k = threadIdx.x; k < A * kSizeBins; k += kThreads) {
        const uint32_t c = sm.sh[k];
        if (c) {
          atomicAdd(sh + int64_t(r) * A * kSizeBins + k, (unsigned long long)c);
          sm.sh[k] = 0;
        }
      }
  }
}

// Thread per (replica, user): the totals over apps and the overall rate bins; then per
// (replica, user, app): the per-app rate bins.
__global__ void __launch_bounds__(kThreads) k_ws_users(WsArgs a, int64_t RU) {
  const DevTrace &t = a.t;
  unsigned long long *const rh = reinterpret_cast<unsigned long long *>(a.o.rate_hist);
  const int64_t A = t.A;
  for (int64_t base0 = blockIdx.x * int64_t(kThreads); base0 < RU;
       base0 += int64_t(gridDim.x) * kThreads) {
    const int64_t ru = base0 + threadIdx.x;
    const bool v = ru < RU;
    const int32_t r = v ? int32_t(ru / t.U) : 0;
    const bool has = v && t.rep_off[r + 1] > t.rep_off[r];
    const uint64_t M = has ? a.max_ts[r] / uint64_t(a.minute_us) + 1 : 0;
    unsigned long long nreq = 0, ntok = 0;
    if (v) {
      for (int64_t ap = 0; ap < A; ++ap) {
        nreq += a.ua_req[ru * A + ap];
        ntok += a.ua_tok[ru * A + ap];
      }
      a.o.user_req[ru] = int64_t(nreq);
      a.o.user_tok[ru] = int64_t(ntok);
      if (ru % t.U == 0) a.o.minutes[r] = int64_t(M);
    }
    const bool act = v && nreq > 0;
    const int64_t row = (int64_t(r) * (A + 1) + A) * 2;
    wave_add2<true>(act, row * kRateBins + rate_bin(nreq, M ? M : 1), 1ull, 0ull, rh, nullptr);
    wave_add2<true>(act, (row + 1) * kRateBins + rate_bin(ntok, M ? M : 1), 1ull, 0ull, rh, nullptr);
  }
  const int64_t RUA = RU * A;
  for (int64_t base0 = blockIdx.x * int64_t(kThreads); base0 < RUA;
       base0 += int64_t(gridDim.x) * kThreads) {
    const int64_t k = base0 + threadIdx.x;
    const bool v = k < RUA;
    const int32_t r = v ? int32_t(k / (int64_t(t.U) * A)) : 0;
    const int32_t ap = v ? int32_t(k % A) : 0;
    const unsigned long long n = v ? a.ua_req[k] : 0ull, tk = v ? a.ua_tok[k] : 0ull;
    const uint64_t M = (v && n > 0) ? a.max_ts[r] / uint64_t(a.minute_us) + 1 : 1;
    const int64_t row = (int64_t(r) * (A + 1) + ap) * 2;
    wave_add2<true>(n > 0, row * kRateBins + rate_bin(n, M), 1ull, 0ull, rh, nullptr);
    wave_add2<true>(n > 0, (row + 1) * kRateBins + rate_bin(tk, M), 1ull, 0ull, rh, nullptr);
  }
}

// One work-group per replica when the replica's (user, app) table fits in LDS (and
// there are replicas enough to fill the chip): records, interaction sizes, graph rows
// and rate bins of the replica in one kernel, every accumulation an LDS atomic (the
// graph rows aggregated per wave first: almost every request adds to the same row),
// and every output of the replica written once with plain stores.  Three passes over
// the replica's records: the tables and the later calls' counts at their first calls;
// the interaction sizes into the size histogram and graph rows; the users' totals
// and rate bins from the table.
constexpr int kRepThreads = 1024;
constexpr int32_t kRepMin = 256;                 // replicas for the per-replica kernel (a CU each)
constexpr size_t kRepLdsMax = 150 * 1024;        // its LDS, at most

struct RepLds {  // byte offsets into the dynamic LDS of k_ws_replica
  size_t tok, ls, gr, red, req, lh, sh, rate, total;
  int copies;                 // of the length sums and histograms, chosen by lane
  int ls_stride, lh_stride;   // entries per copy (one of padding, for the banks)
};

// The per-app length sums and histograms take an LDS atomic per request and field, and
// a wave's lanes hit few of their entries (a handful of apps, lengths in a few bins):
// when LDS allows, kWsCopies copies of them, lane l adding to copy l % kWsCopies, cut
// the lanes of one instruction that meet on one entry by that factor.
constexpr int kWsCopies = 8;
__host__ __device__ inline RepLds rep_lds_n(int32_t U, int32_t A, int copies) {
  RepLds L;
  const size_t ua = size_t(U) * size_t(A);
  L.copies = copies;
  L.ls_stride = A * 3 + (copies > 1 ? 1 : 0);
  L.lh_stride = A * 3 * kLenBins + (copies > 1 ? 1 : 0);
  size_t o = 0;
  L.tok = o;  o += ua * 8;                                 // tokens per (user, app)
  L.ls = o;   o += size_t(copies) * L.ls_stride * 8;       // length sums [A][3]
  L.gr = o;   o += size_t(kGraphBins) * 5 * 8;             // Table 2 rows
  L.red = o;  o += size_t(kRepThreads / 64) * 8;           // per-wave maxima
  L.req = o;  o += ua * 4;                                 // requests per (user, app)
  L.lh = o;   o += size_t(copies) * L.lh_stride * 4;       // length histograms
  L.sh = o;   o += size_t(A) * kSizeBins * 4;              // size histogram
  L.rate = o; o += size_t(A + 1) * 2 * kRateBins * 4;      // rate histograms
  L.total = (o + 15) / 16 * 16;
  return L;
}
__host__ __device__ inline RepLds rep_lds(int32_t U, int32_t A) {
  const RepLds c = rep_lds_n(U, A, kWsCopies);
  return c.total <= kRepLdsMax ? c : rep_lds_n(U, A, 1);
}

__device__ inline unsigned long long wmax64(unsigned long long v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const unsigned long long o = (unsigned long long)__shfl_xor((long long)v, m, 64);
    v = o > v ? o : v;
  }
  return v;
}

__global__ void __launch_bounds__(kRepThreads) k_ws_replica(WsArgs a) {
  extern __shared__ __align__(16) unsigned char dsm[];
  const DevTrace &t = a.t;
  const int32_t r = blockIdx.x, U = t.U, A = t.A;
  const RepLds L = rep_lds(U, A);
  unsigned long long *const tok = reinterpret_cast<unsigned long long *>(dsm + L.tok);
  unsigned long long *const ls = reinterpret_cast<unsigned long long *>(dsm + L.ls);
  unsigned long long *const gr = reinterpret_cast<unsigned long long *>(dsm + L.gr);
  unsigned long long *const red = reinterpret_cast<unsigned long long *>(dsm + L.red);
  uint32_t *const req = reinterpret_cast<uint32_t *>(dsm + L.req);
  uint32_t *const lh = reinterpret_cast<uint32_t *>(dsm + L.lh);
  uint32_t *const sh = reinterpret_cast<uint32_t *>(dsm + L.sh);
  uint32_t *const rate = reinterpret_cast<uint32_t *>(dsm + L.rate);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t UA = int64_t(U) * A;
  for (int64_t k = tid; k < UA; k += kRepThreads) {
    tok[k] = 0;
    req[k] = 0;
  }
  for (int k = tid; k < L.copies * L.ls_stride; k += kRepThreads) ls[k] = 0;
  for (int k = tid; k < kGraphBins * 5; k += kRepThreads) gr[k] = 0;
  for (int k = tid; k < L.copies * L.lh_stride; k += kRepThreads) lh[k] = 0;
  const int cp = lane & (L.copies - 1);  // this lane's copy of the length tables
  uint32_t *const lh_c = lh + cp * L.lh_stride;
  unsigned long long *const ls_c = ls + cp * L.ls_stride;
  for (int k = tid; k < A * kSizeBins; k += kRepThreads) sh[k] = 0;
  for (int k = tid; k < (A + 1) * 2 * kRateBins; k += kRepThreads) rate[k] = 0;
  const int64_t base = t.rep_off[r], n = t.rep_off[r + 1] - base;
  if (t.call)  // an interaction's size starts at one for its first call
    for (int64_t i = tid; i < n; i += kRepThreads) a.size[base + i] = t.call[base + i] != 0 ? 0u : 1u;
  __syncthreads();

  // pass 1: the (user, app) table, length histograms and sums, latest arrival, and one
  // count at the first call of each later call (the checks of k_ws_records)
  int32_t code = 0;
  unsigned long long mts = 0;
  bool any = false;
  for (int64_t i0 = tid; i0 < n; i0 += 2 * kRepThreads) {  // two records a thread, loads together
    int32_t u[2], ap[2];
    int64_t ts[2], Lx[2][3], h[2];
    bool ok[2], first[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int64_t i = i0 + j * kRepThreads, g = base + i;
      ok[j] = i < n;
      u[j] = ok[j] ? t.user[g] : 0;
      ap[j] = ok[j] ? t.app[g] : 0;
      ts[j] = ok[j] ? t.ts[g] : 0;
      Lx[j][0] = ok[j] ? t.len_in[g] : 0;
      Lx[j][1] = (ok[j] && t.len_sys) ? t.len_sys[g] : 0;
      Lx[j][2] = ok[j] ? t.len_out[g] : 0;
      first[j] = !(ok[j] && t.call && t.call[g] != 0);
      h[j] = first[j] ? i : int64_t(t.head[g]);
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int64_t i = i0 + j * kRepThreads;
      if (i >= n) continue;
      bool v = u[j] >= 0 && u[j] < U && ap[j] >= 0 && ap[j] < A && ts[j] >= 0 &&
               len_ok(int32_t(Lx[j][0])) && len_ok(int32_t(Lx[j][1])) && len_ok(int32_t(Lx[j][2]));
      if (v && !first[j]) v = h[j] >= 0 && h[j] < i;
      if (!v) {
        code = FS_E_RANGE;
        continue;
      }
      mts = (unsigned long long)ts[j] > mts ? (unsigned long long)ts[j] : mts;
      any = true;
      const int64_t k = int64_t(u[j]) * A + ap[j];
      atomicAdd(&req[k], 1u);
      atomicAdd(&tok[k], (unsigned long long)(Lx[j][0] + Lx[j][1] + Lx[j][2]));
#pragma unroll
      for (int x = 0; x < 3; ++x) {
        atomicAdd(&lh_c[(ap[j] * 3 + x) * kLenBins + len_bin(Lx[j][x])], 1u);
        if (Lx[j][x]) atomicAdd(&ls_c[ap[j] * 3 + x], (unsigned long long)Lx[j][x]);
      }
      if (!first[j]) atomicAdd(a.size + base + h[j], 1u);
    }
  }
  mts = wmax64(mts);
  if (lane == 0) red[wave] = (__ballot(any) != 0) ? mts + 1 : 0;  // 0: no valid request
  __syncthreads();
  unsigned long long mx = 0;
  for (int w = 0; w < kRepThreads / 64; ++w) mx = red[w] > mx ? red[w] : mx;
  const uint64_t M = n > 0 ? (mx ? mx - 1 : 0) / uint64_t(a.minute_us) + 1 : 0;

  // pass 2: sizes into the size histogram (first calls) and the graph rows (every
  // request, by its interaction's size; the checks of k_ws_graph)
  for (int64_t i0 = 0; i0 < n; i0 += kRepThreads) {
    const int64_t i = i0 + tid, g = base + i;
    bool ok = i < n;
    bool first = true;
    int32_t ap = 0;
    uint32_t sz = 0;
    unsigned long long l0 = 0, l1 = 0, l2 = 0;
    if (ok) {
      const int32_t uu = t.user[g];
      ap = t.app[g];
      first = first_of(t, g);
      const int64_t hh = first ? i : int64_t(t.head[g]);
      ok = uu >= 0 && uu < U && ap >= 0 && ap < A && hh >= 0 && (first ? hh == i : hh < i);
      if (ok) {
        // (written by this work-group's atomics: read past the L1 cache)
        sz = t.call ? __hip_atomic_load(a.size + base + hh, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                    : 1u;
        l0 = (unsigned long long)t.len_in[g];
        l1 = (unsigned long long)t.len_out[g];
        l2 = t.len_sys ? (unsigned long long)t.len_sys[g] : 0ull;
        if (first && sz > 0) atomicAdd(&sh[ap * kSizeBins + (sz < kSizeBins ? int(sz) : kSizeBins) - 1], 1u);
      }
    }
    // graph rows: per distinct bin among the wave's lanes, one add per field
    const int b = graph_bin(sz);
    uint64_t pending = __ballot(ok);
    while (pending) {
      const int bl = __shfl(b, __ffsll((long long)pending) - 1, 64);
      const bool mine = ok && b == bl;
      const uint64_t mm = __ballot(mine);
      const unsigned long long nf = __popcll(__ballot(mine && first));
      const unsigned long long nr = __popcll(mm);
      const unsigned long long s0 = wsum64(mine ? l0 : 0ull), s1 = wsum64(mine ? l1 : 0ull),
                               s2 = wsum64(mine ? l2 : 0ull);
      if (lane == 0) {
        unsigned long long *row = gr + bl * 5;
        if (nf) atomicAdd(row, nf);
        atomicAdd(row + 1, nr);
        if (s0) atomicAdd(row + 2, s0);
        if (s1) atomicAdd(row + 3, s1);
        if (s2) atomicAdd(row + 4, s2);
      }
      pending &= ~mm;
    }
  }
  __syncthreads();

  // pass 3: the table's entries (per-app rate bins) and each user's totals
  const int64_t ro = int64_t(r) * UA;
  for (int64_t k = tid; k < UA; k += kRepThreads) {
    const uint32_t nq = req[k];
    const unsigned long long tk = tok[k];
    if (a.o.user_app_req) a.o.user_app_req[ro + k] = int64_t(nq);
    if (a.o.user_app_tok) a.o.user_app_tok[ro + k] = int64_t(tk);
    if (nq > 0) {
      const int ap = int(k % A);
      atomicAdd(&rate[(ap * 2) * kRateBins + rate_bin(nq, M)], 1u);
      atomicAdd(&rate[(ap * 2 + 1) * kRateBins + rate_bin(tk, M)], 1u);
    }
  }
  for (int32_t u = tid; u < U; u += kRepThreads) {
    unsigned long long nq = 0, nt = 0;
    for (int32_t ap = 0; ap < A; ++ap) {
      nq += req[int64_t(u) * A + ap];
      nt += tok[int64_t(u) * A + ap];
    }
    a.o.user_req[int64_t(r) * U + u] = int64_t(nq);
    a.o.user_tok[int64_t(r) * U + u] = int64_t(nt);
    if (nq > 0) {
      atomicAdd(&rate[(A * 2) * kRateBins + rate_bin(nq, M)], 1u);
      atomicAdd(&rate[(A * 2 + 1) * kRateBins + rate_bin(nt, M)], 1u);
    }
  }
  __syncthreads();
  // the replica's histograms and sums, written once
  if (tid == 0) a.o.minutes[r] = int64_t(M);
  for (int k = tid; k < (A + 1) * 2 * kRateBins; k += kRepThreads)
    a.o.rate_hist[int64_t(r) * (A + 1) * 2 * kRateBins + k] = int64_t(rate[k]);
  for (int k = tid; k < A * 3 * kLenBins; k += kRepThreads) {
    uint64_t v = 0;
    for (int c = 0; c < L.copies; ++c) v += lh[c * L.lh_stride + k];
    a.o.len_hist[int64_t(r) * A * 3 * kLenBins + k] = int64_t(v);
  }
  for (int k = tid; k < A * 3; k += kRepThreads) {
    unsigned long long v = 0;
    for (int c = 0; c < L.copies; ++c) v += ls[c * L.ls_stride + k];
    a.o.len_sum[int64_t(r) * A * 3 + k] = int64_t(v);
  }
  for (int k = tid; k < A * kSizeBins; k += kRepThreads)
    a.o.size_hist[int64_t(r) * A * kSizeBins + k] = int64_t(sh[k]);
  for (int k = tid; k < kGraphBins * 5; k += kRepThreads)
    a.o.graph[int64_t(r) * kGraphBins * 5 + k] = int64_t(gr[k]);
  if (code) raise_err(a.err, code);
}

int grid_for(int64_t n) {
  int64_t b = (n + kThreads - 1) / kThreads;
  if (b < 1) b = 1;
  if (b > 16384) b = 16384;
  return int(b);
}

size_t up256(size_t x) { return (x + 255) / 256 * 256; }

struct WsLayout {
  size_t ua_req, ua_tok, size, max_ts, total;
};

WsLayout ws_layout(const fs_trace *t, bool own_req, bool own_tok) {
  const size_t rua = size_t(t->n_replicas) * size_t(t->n_users) * size_t(t->n_apps);
  const size_t n = size_t(t->rep_off_h[t->n_replicas]);
  WsLayout L;
  size_t o = 0;
  L.ua_req = o; o += own_req ? 0 : up256(rua * 8);
  L.ua_tok = o; o += own_tok ? 0 : up256(rua * 8);
  L.size = o; o += up256((n > 0 ? n : 1) * 4);
  L.max_ts = o; o += up256(size_t(t->n_replicas) * 8);
  L.total = o;
  return L;
}

}  // namespace

size_t workload_workspace_bytes(const fs_trace *t) { return ws_layout(t, false, false).total; }

hipError_t launch_workload(const fs_trace *t, int64_t minute_us, const fs_wstats *out, void *ws,
                           int32_t *err, hipStream_t s) {
  const WsLayout L = ws_layout(t, false, false);
  char *w = static_cast<char *>(ws);
  WsArgs a;
  a.t = dev_trace(t);
  a.minute_us = minute_us;
  a.o = *out;
  a.ua_req = out->user_app_req ? reinterpret_cast<unsigned long long *>(out->user_app_req)
                               : reinterpret_cast<unsigned long long *>(w + L.ua_req);
  a.ua_tok = out->user_app_tok ? reinterpret_cast<unsigned long long *>(out->user_app_tok)
                               : reinterpret_cast<unsigned long long *>(w + L.ua_tok);
  a.size = reinterpret_cast<unsigned int *>(w + L.size);
  a.max_ts = reinterpret_cast<unsigned long long *>(w + L.max_ts);
  a.err = err;
  const int64_t RU = int64_t(t->n_replicas) * t->n_users, RUA = RU * t->n_apps;
  const int64_t N = a.t.N;
  // one work-group per replica when its table fits in LDS and replicas fill the chip
  const RepLds RL = rep_lds(t->n_users, t->n_apps);
  int64_t most_n = 0;
  for (int32_t r = 0; r < t->n_replicas; ++r)
    most_n = std::max<int64_t>(most_n, t->rep_off_h[r + 1] - t->rep_off_h[r]);
  if (t->n_replicas >= kRepMin && RL.total <= kRepLdsMax && most_n < (int64_t(1) << 31)) {
    if (RL.total > 65536) {
      const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(k_ws_replica),
                                               hipFuncAttributeMaxDynamicSharedMemorySize,
                                               int(RL.total));
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(k_ws_replica, dim3(t->n_replicas), dim3(kRepThreads), RL.total, s, a);
    return hipGetLastError();
  }
  const int64_t most = std::max<int64_t>(std::max<int64_t>(RUA, N),
                                         int64_t(t->n_replicas) * (t->n_apps + 1) * 2 * kRateBins);
  hipLaunchKernelGGL(k_ws_zero, dim3(grid_for(most)), dim3(kThreads), 0, s, a, RUA, RU);
  if (N > 0) {
    const dim3 chunks(uint32_t((N + kChunk - 1) / kChunk));
    if (t->n_apps <= kLdsApps) {
      hipLaunchKernelGGL(k_ws_records<true>, chunks, dim3(kThreads), 0, s, a);
      hipLaunchKernelGGL(k_ws_graph<true>, chunks, dim3(kThreads), 0, s, a);
    } else {
      hipLaunchKernelGGL(k_ws_records<false>, chunks, dim3(kThreads), 0, s, a);
      hipLaunchKernelGGL(k_ws_graph<false>, chunks, dim3(kThreads), 0, s, a);
    }
  }
  hipLaunchKernelGGL(k_ws_users, dim3(grid_for(RUA > RU ? RUA : RU)), dim3(kThreads), 0, s, a, RU);
  return hipGetLastError();
}

}  // namespace fs

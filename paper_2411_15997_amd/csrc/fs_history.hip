// Offline derivation of the WSC weights and the OIT app limits from a historical trace
// (Eq. 1 with the expected token counts taken as the history's sample means; Sec. 4,
// OIT, the app limit scaled by the app's mean number of LLM calls per interaction).
//
// Pass 1 (k_hist_accum) is a segmented sum by (app, stage) over the record stream:
// each work-group keeps the group table in LDS (one packed records | first-calls
// word and three token sums per group), replicated up to 16 times so that lanes adding
// to the same group mostly hit different words, reads four records per thread with
// 16-byte loads (two such vectors in flight), and stores its table as one row of the
// workspace; k_hist_reduce sums the rows in chunks of 64.  Tables too large for LDS
// accumulate straight into the global table with atomics.
// Pass 2 (k_hist_final, one work-group) pools empty groups and divides exactly in
// integers, one thread per coefficient.
#include <algorithm>

#include "fs_device.h"
#include "fs_launch.h"

namespace fs {

namespace {

constexpr int kHistThreads = 256;
constexpr int kHistSlots = 4;                 // per group in LDS: records|first, in, sys, out
constexpr int64_t kHistLdsBytes = 65536;      // LDS for the replicated group tables
constexpr int kHistMaxCopies = 16;
constexpr int kFinalThreads = 1024;           // one thread per app (n_apps <= 1024)
constexpr int64_t kMaxRecords = int64_t(1) << 36;

struct HistArgs {
  const int32_t *app, *call, *len_in, *len_sys, *len_out;
  int64_t N;
  int32_t A, J;
  int64_t *stats;           // [A][J][5]
  unsigned long long *part;  // [work-groups][A*J*5] partial tables (LDS path)
  int32_t *err;
};

// stats fields
enum { kN = 0, kFirst = 1, kIn = 2, kSys = 3, kOut = 4 };

// Clears the global table and the status word.
__global__ void __launch_bounds__(kHistThreads) k_hist_zero(int64_t *p, int64_t n, int32_t *err) {
  if (blockIdx.x == 0 && threadIdx.x == 0) *err = 0;
  for (int64_t i = blockIdx.x * int64_t(kHistThreads) + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * kHistThreads)
    p[i] = 0;
}

// One record: its group and the amounts it adds, or false when it is out of range.
__device__ inline bool hist_record(const HistArgs &a, int32_t app, int32_t call, int32_t li,
                                   int32_t ls, int32_t lo, int32_t &grp) {
  if (app < 0 || app >= a.A || call < 0 || !len_ok(li) || !len_ok(ls) || !len_ok(lo))
    return false;
  const int32_t j = call < a.J - 1 ? call : a.J - 1;
  grp = app * a.J + j;
  return true;
}

template <bool LDS>
__device__ inline void hist_add(const HistArgs &a, unsigned long long *tab, int32_t grp,
                                int32_t call, int32_t li, int32_t ls, int32_t lo) {
  if (LDS) {
    unsigned long long *t = tab + int64_t(grp) * kHistSlots;
    // records in the low 32 bits, first calls in the high 32 (a work-group reads
    // fewer than 2^32 records)
    atomicAdd(t, 1ull | (call == 0 ? (1ull << 32) : 0ull));
    atomicAdd(t + 1, (unsigned long long)li);
    if (a.len_sys) atomicAdd(t + 2, (unsigned long long)ls);
    atomicAdd(t + 3, (unsigned long long)lo);
  } else {
    unsigned long long *t = reinterpret_cast<unsigned long long *>(a.stats) + int64_t(grp) * 5;
    atomicAdd(t + kN, 1ull);
    if (call == 0) atomicAdd(t + kFirst, 1ull);
    atomicAdd(t + kIn, (unsigned long long)li);
    if (a.len_sys) atomicAdd(t + kSys, (unsigned long long)ls);
    atomicAdd(t + kOut, (unsigned long long)lo);
  }
}

struct Vec4Rec {
  int4 app, li, lo, ls, call;
};

__device__ inline Vec4Rec load_vec4(const HistArgs &a, int64_t v) {
  Vec4Rec r;
  r.app = __ldg(reinterpret_cast<const int4 *>(a.app) + v);
  r.li = __ldg(reinterpret_cast<const int4 *>(a.len_in) + v);
  r.lo = __ldg(reinterpret_cast<const int4 *>(a.len_out) + v);
  r.ls = a.len_sys ? __ldg(reinterpret_cast<const int4 *>(a.len_sys) + v) : make_int4(0, 0, 0, 0);
  r.call = a.call ? __ldg(reinterpret_cast<const int4 *>(a.call) + v) : make_int4(0, 0, 0, 0);
  return r;
}

template <bool LDS>
__device__ inline void add_vec4(const HistArgs &a, unsigned long long *tab, const Vec4Rec &r,
                                int32_t &code) {
  const int32_t ap[4] = {r.app.x, r.app.y, r.app.z, r.app.w};
  const int32_t ca[4] = {r.call.x, r.call.y, r.call.z, r.call.w};
  const int32_t i4[4] = {r.li.x, r.li.y, r.li.z, r.li.w}, s4[4] = {r.ls.x, r.ls.y, r.ls.z, r.ls.w};
  const int32_t o4[4] = {r.lo.x, r.lo.y, r.lo.z, r.lo.w};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    int32_t grp;
    if (hist_record(a, ap[k], ca[k], i4[k], s4[k], o4[k], grp))
      hist_add<LDS>(a, tab, grp, ca[k], i4[k], s4[k], o4[k]);
    else
      code = FS_E_RANGE;
  }
}

// LDS: `copies` replicas of the [A*J][kHistSlots] table; lane l adds into replica
// l % copies, so lanes of one wave that hit the same group mostly touch different words.
template <bool LDS>
__global__ void __launch_bounds__(kHistThreads) k_hist_accum(HistArgs a, int64_t n_vec,
                                                             int32_t copies) {
  extern __shared__ unsigned long long lds_tab[];
  const int64_t G = int64_t(a.A) * a.J;
  if (LDS) {
    for (int64_t i = threadIdx.x; i < G * kHistSlots * copies; i += kHistThreads) lds_tab[i] = 0;
    __syncthreads();
  }
  unsigned long long *tab = lds_tab + (LDS ? int64_t(threadIdx.x & (copies - 1)) * G * kHistSlots : 0);
  int32_t code = 0;
  const int64_t stride = int64_t(gridDim.x) * kHistThreads;
  int64_t v = blockIdx.x * int64_t(kHistThreads) + threadIdx.x;
  // two vectors in flight per thread
  for (; v + stride < n_vec; v += 2 * stride) {
    const Vec4Rec r0 = load_vec4(a, v), r1 = load_vec4(a, v + stride);
    add_vec4<LDS>(a, tab, r0, code);
    add_vec4<LDS>(a, tab, r1, code);
  }
  if (v < n_vec) add_vec4<LDS>(a, tab, load_vec4(a, v), code);
  // the ragged tail (the last N % 4 records, or every record of unaligned arrays)
  for (int64_t g = n_vec * 4 + blockIdx.x * int64_t(kHistThreads) + threadIdx.x; g < a.N;
       g += stride) {
    const int32_t call = a.call ? a.call[g] : 0, ls = a.len_sys ? a.len_sys[g] : 0;
    int32_t grp;
    if (hist_record(a, a.app[g], call, a.len_in[g], ls, a.len_out[g], grp))
      hist_add<LDS>(a, tab, grp, call, a.len_in[g], ls, a.len_out[g]);
    else
      code = FS_E_RANGE;
  }
  if (code) raise_err(a.err, code);
  if (LDS) {
    // this work-group's table, summed over its replicas, to its own partial row
    __syncthreads();
    unsigned long long *row = a.part + int64_t(blockIdx.x) * G * 5;
    for (int64_t gi = threadIdx.x; gi < G; gi += kHistThreads) {
      unsigned long long nf = 0, si = 0, ss = 0, so = 0;
      for (int c = 0; c < copies; ++c) {
        const unsigned long long *t = lds_tab + (int64_t(c) * G + gi) * kHistSlots;
        nf += t[0];  // per replica fewer than 2^32 records and first calls: no carry
        si += t[1];
        ss += t[2];
        so += t[3];
      }
      row[gi * 5 + kN] = nf & 0xffffffffull;
      row[gi * 5 + kFirst] = nf >> 32;
      row[gi * 5 + kIn] = si;
      row[gi * 5 + kSys] = ss;
      row[gi * 5 + kOut] = so;
    }
  }
}

// stats[c] += sum of part[b][c] over a chunk of kReduceRows work-group rows (all of
// a thread's loads are issued before the first add).
constexpr int kReduceRows = 16;
__global__ void __launch_bounds__(kHistThreads) k_hist_reduce(const unsigned long long *part,
                                                              int64_t rows, int64_t cols,
                                                              int64_t *stats) {
  const int64_t idx = blockIdx.x * int64_t(kHistThreads) + threadIdx.x;
  const int64_t col = idx % cols, chunk = idx / cols;
  const int64_t b0 = chunk * kReduceRows;
  if (b0 >= rows) return;
  const int64_t b1 = b0 + kReduceRows < rows ? b0 + kReduceRows : rows;
  unsigned long long v[kReduceRows];
#pragma unroll
  for (int k = 0; k < kReduceRows; ++k) v[k] = b0 + k < b1 ? part[(b0 + k) * cols + col] : 0ull;
  unsigned long long sum = 0;
#pragma unroll
  for (int k = 0; k < kReduceRows; ++k) sum += v[k];
  if (sum) atomicAdd(reinterpret_cast<unsigned long long *>(stats) + col, sum);
}

// floor((hi * 2^64 + lo) / d) and the remainder, for hi < d (the quotient fits in 64
// bits); shift-subtract long division, exact.
__device__ inline uint64_t udiv128(uint64_t hi, uint64_t lo, uint64_t d, uint64_t &rem) {
  uint64_t q = 0;
  for (int b = 63; b >= 0; --b) {
    const uint64_t top = hi >> 63;  // the bit shifted out of the 128-bit remainder
    hi = (hi << 1) | (lo >> 63);
    lo <<= 1;
    q <<= 1;
    if (top || hi >= d) {
      hi -= d;
      q |= 1;
    }
  }
  rem = hi;
  return q;
}

// round_half_even(m * f / d) for the product of two 64-bit values; false when the
// result does not fit below `limit`.
__device__ inline bool muldiv_rhe(uint64_t m, uint64_t f, uint64_t d, uint64_t limit,
                                  uint64_t &out) {
  const uint64_t lo = m * f, hi = __umul64hi(m, f);
  if (hi >= d) return false;
  uint64_t r, q;
  if (hi == 0) {
    q = lo / d;
    r = lo - q * d;
  } else {
    q = udiv128(hi, lo, d, r);
  }
  // compare 2r with d without overflow (r < d)
  const bool above = r > d - r, tie = r == d - r;
  if (above || (tie && (q & 1))) ++q;
  if (q >= limit) return false;
  out = q;
  return true;
}

struct FinalArgs {
  const int64_t *stats;
  int32_t A, J;
  int64_t K;
  int32_t base;
  int64_t *coef;   // [A][J][3] or null
  int32_t *t_app;  // [A] or null
  int32_t *err;
};

// One work-group: the per-app pools (one thread per app), the history's pool, then one
// thread per (app, stage, token class) coefficient.
__global__ void __launch_bounds__(kFinalThreads) k_hist_final(FinalArgs a) {
  __shared__ uint64_t s_n[kFinalThreads], s_D[kFinalThreads], s_first[kFinalThreads];
  __shared__ uint64_t r_n[kFinalThreads], r_D[kFinalThreads];
  const int t = threadIdx.x;
  const int64_t cls[3] = {1, 2, 1};  // alpha, beta, gamma: input, system, output tokens
  uint64_t n_a = 0, D_a = 0, first_a = 0;
  if (t < a.A)
#pragma unroll 4
    for (int32_t j = 0; j < a.J; ++j) {
      const int64_t *s = a.stats + (int64_t(t) * a.J + j) * 5;
      n_a += uint64_t(s[kN]);
      first_a += uint64_t(s[kFirst]);
      D_a += uint64_t(cls[0] * s[kIn] + cls[1] * s[kSys] + cls[2] * s[kOut]);
    }
  s_n[t] = r_n[t] = n_a;
  s_D[t] = r_D[t] = D_a;
  s_first[t] = first_a;
  __syncthreads();
  for (int h = kFinalThreads / 2; h > 0; h >>= 1) {
    if (t < h) {
      r_n[t] += r_n[t + h];
      r_D[t] += r_D[t + h];
    }
    __syncthreads();
  }
  const uint64_t all_n = r_n[0], all_D = r_D[0];
  int32_t code = 0;
  const int64_t n_coef = a.coef ? int64_t(a.A) * a.J * 3 : 0;
  for (int64_t i = t; i < n_coef; i += kFinalThreads) {
    const int64_t gi = i / 3;
    const int x = int(i - gi * 3);
    const int32_t app = int32_t(gi / a.J);
    const int64_t *s = a.stats + gi * 5;
    uint64_t n = uint64_t(s[kN]);
    uint64_t D = uint64_t(cls[0] * s[kIn] + cls[1] * s[kSys] + cls[2] * s[kOut]);
    // a group with no records or no tokens takes its app's stages, then the history's
    if (n == 0 || D == 0) {
      n = s_n[app];
      D = s_D[app];
    }
    if (n == 0 || D == 0) {
      n = all_n;
      D = all_D;
    }
    if (n == 0 || D == 0) {
      n = 1;
      D = uint64_t(a.K);
    }
    // 2^16 K x / w_aj with w_aj = D / n
    uint64_t q;
    if (!muldiv_rhe(uint64_t(65536 * a.K * cls[x]), n, D, uint64_t(kCoefLimit), q)) {
      code = FS_E_RANGE;
      q = 0;
    }
    a.coef[i] = int64_t(q);
  }
  if (a.t_app && t < a.A) {
    int64_t lim = a.base;
    if (first_a > 0) {
      // ceil(base * records / first calls) = floor((base * records + first - 1) / first)
      const uint64_t lo = uint64_t(a.base) * n_a, hi = __umul64hi(uint64_t(a.base), n_a);
      const uint64_t lo2 = lo + (first_a - 1), hi2 = hi + (lo2 < lo ? 1 : 0);
      uint64_t r, q = 0;
      if (hi2 >= first_a || (q = udiv128(hi2, lo2, first_a, r)) > uint64_t(INT32_MAX)) {
        code = FS_E_RANGE;
        q = 0;
      }
      lim = int64_t(q);
    }
    a.t_app[t] = int32_t(lim);
  }
  if (code) raise_err(a.err, code);
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// Work-groups of the LDS path for N records (0: the table does not fit in LDS and the
// records accumulate straight into the global table).
int64_t history_blocks(int64_t N, int64_t G) {
  const int64_t table = G * kHistSlots * int64_t(sizeof(unsigned long long));
  if (table > kHistLdsBytes) return 0;
  const int64_t units = (N + 3) / 4;
  // about eight 4-record vectors per thread, at most 1024 work-groups and 32 MB of
  // partial tables
  int64_t blocks = (units + kHistThreads * 8 - 1) / (kHistThreads * 8);
  const int64_t cap = std::max<int64_t>(1, (int64_t(32) << 20) / (G * 5 * 8));
  return std::max<int64_t>(1, std::min<int64_t>(blocks, std::min<int64_t>(1024, cap)));
}

}  // namespace

size_t history_workspace_bytes(const fs_trace *t, int32_t n_stages) {
  const int64_t N = t->rep_off_h[t->n_replicas];
  const int64_t G = int64_t(t->n_apps) * n_stages;
  return size_t(history_blocks(N, G) * G * 5) * sizeof(unsigned long long);
}

hipError_t launch_history(const fs_trace *t, int32_t n_stages, int64_t K, int32_t base_limit,
                          int64_t *stats, int64_t *coef, int32_t *t_app, void *ws,
                          int32_t *err, hipStream_t s) {
  const int64_t N = t->rep_off_h[t->n_replicas];
  const int64_t G = int64_t(t->n_apps) * n_stages;
  hipLaunchKernelGGL(k_hist_zero, dim3(std::min<int64_t>((G * 5 + kHistThreads - 1) / kHistThreads,
                                                         1024)),
                     dim3(kHistThreads), 0, s, stats, G * 5, err);
  if (N > 0) {
    unsigned long long *part = static_cast<unsigned long long *>(ws);
    HistArgs ha{t->app, t->call, t->len_in, t->len_sys, t->len_out, N, t->n_apps, n_stages,
                stats, part, err};
    const bool vec = aligned16(t->app) && aligned16(t->len_in) && aligned16(t->len_out) &&
                     (!t->len_sys || aligned16(t->len_sys)) && (!t->call || aligned16(t->call));
    const int64_t n_vec = vec ? N / 4 : 0;
    const int64_t blocks = history_blocks(N, G);
    if (blocks > 0) {
      const int64_t table = G * kHistSlots * int64_t(sizeof(unsigned long long));
      int32_t copies = 1;
      while (copies < kHistMaxCopies && table * copies * 2 <= kHistLdsBytes) copies *= 2;
      hipLaunchKernelGGL(k_hist_accum<true>, dim3(blocks), dim3(kHistThreads),
                         size_t(table * copies), s, ha, n_vec, copies);
      const int64_t cols = G * 5, chunks = (blocks + kReduceRows - 1) / kReduceRows;
      hipLaunchKernelGGL(k_hist_reduce, dim3((cols * chunks + kHistThreads - 1) / kHistThreads),
                         dim3(kHistThreads), 0, s, part, blocks, cols, stats);
    } else {
      const int64_t units = std::max(n_vec, (N - n_vec * 4 + 3) / 4);
      const int64_t gb = std::max<int64_t>(
          1, std::min<int64_t>((units + kHistThreads * 8 - 1) / (kHistThreads * 8), 1024));
      hipLaunchKernelGGL(k_hist_accum<false>, dim3(gb), dim3(kHistThreads), 0, s, ha, n_vec, 1);
    }
  }
  FinalArgs fa{stats, t->n_apps, n_stages, K, base_limit, coef, t_app, err};
  hipLaunchKernelGGL(k_hist_final, dim3(1), dim3(kFinalThreads), 0, s, fa);
  return hipGetLastError();
}

int64_t history_max_records() { return kMaxRecords; }

}  // namespace fs

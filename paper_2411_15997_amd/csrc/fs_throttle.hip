// OIT sliding-window limit test (Alg. 1 monitoring stream: every arrival is counted
// per user and per (user, app); Sec. 4, OIT: the user limit is checked first, then
// the app limit; a later call of an interaction is never checked and shares its
// first call's fate).
//
// Method.  For a key k (a user, or a (user, app) pair) let the key's records be
// taken in stream order.  The window count of record i exceeds T iff the record T
// positions earlier in the same key sequence exists and arrived after ts_i - W
// (the T+1 most recent arrivals of the key, i included, all lie in the window).
// So the test is O(1) once each key's records are contiguous in stream order:
//   1. key = replica*U + user (low B_u bits) with the app above it (B_a bits);
//   2. stable LSD radix sort of (key, index) over the user bits -> user order;
//      test the user limit at distance T_user;
//   3. one more stable radix pass over the app bits -> (app, user) order, where
//      every (user, app) pair is contiguous and still in stream order;
//      test the app limit at distance T_app[app];
//   4. back in stream order: combine the two flags, apply overload gating and the
//      interaction rule, pack the bitmap with wave ballots.
// Radix passes: per-tile digit histograms, a device-wide exclusive scan, then a
// stable scatter (wave-match ranking, tile reordered in LDS so the global writes
// of each digit run are contiguous).
#include "fs_device.h"
#include "fs_launch.h"

namespace fs {
namespace {

constexpr int kThreads = 256;
constexpr int kItems = 16;
constexpr int kTile = kThreads * kItems;  // 4096 records per radix tile
constexpr int kRadixBits = 8;
constexpr int kRadix = 1 << kRadixBits;
constexpr int kScanThreads = 1024;
constexpr int kScanItems = 4;
constexpr int kScanChunk = kScanThreads * kScanItems;

int bits_for(int64_t n_values) {  // bits to represent 0 .. n_values-1 (at least 1)
  int b = 1;
  while ((int64_t(1) << b) < n_values) ++b;
  return b;
}

size_t up(size_t x) { return (x + 255) / 256 * 256; }

struct Layout {
  int64_t N;
  int64_t tiles;
  int Bu, Ba;
  size_t off_keyA, off_idxA, off_keyB, off_idxB, off_eu, off_ea, off_hist, off_part, off_tapp;
  size_t total;
};

Layout layout(const fs_trace *t) {
  Layout L;
  L.N = t->rep_off_h[t->n_replicas];
  L.tiles = (L.N + kTile - 1) / kTile;
  L.Bu = bits_for(int64_t(t->n_replicas) * t->n_users);
  L.Ba = bits_for(t->n_apps);
  size_t n = size_t(L.N > 0 ? L.N : 1);
  size_t hist_len = size_t(kRadix) * size_t(L.tiles > 0 ? L.tiles : 1);
  size_t o = 0;
  L.off_keyA = o; o += up(n * 4);
  L.off_idxA = o; o += up(n * 4);
  L.off_keyB = o; o += up(n * 4);
  L.off_idxB = o; o += up(n * 4);
  L.off_eu = o; o += up(n);
  L.off_ea = o; o += up(n);
  L.off_hist = o; o += up(hist_len * 4);
  L.off_part = o; o += up(((hist_len + kScanChunk - 1) / kScanChunk + 1) * 4);
  L.off_tapp = o; o += up(kMaxApps * 4);
  L.total = o;
  return L;
}

// ---------------------------------------------------------------- block helpers

// Inclusive prefix sum over the block (blockDim.x threads, multiple of 64).
__device__ uint32_t block_inclusive_scan(uint32_t v, uint32_t *s_waves, uint32_t &total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    uint32_t y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  if (lane == 63) s_waves[wave] = x;
  __syncthreads();
  if (wave == 0) {
    uint32_t w = lane < nw ? s_waves[lane] : 0;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      uint32_t y = __shfl_up(w, d, 64);
      if (lane >= d) w += y;
    }
    if (lane < nw) s_waves[lane] = w;
  }
  __syncthreads();
  uint32_t before = wave > 0 ? s_waves[wave - 1] : 0;
  total = s_waves[nw - 1];
  __syncthreads();
  return x + before;
}

// ---------------------------------------------------------------- init + checks

struct InitArgs {
  DevTrace t;
  int Bu;
  bool check_chain;
  uint32_t *key;
  uint32_t *idx;
  int32_t *err;
};

__global__ void __launch_bounds__(kThreads) k_thr_init(InitArgs a) {
  int32_t code = 0;
  const DevTrace &t = a.t;
  for (int64_t g = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; g < t.N;
       g += int64_t(gridDim.x) * blockDim.x) {
    int32_t r = replica_of(t.rep_off, t.R, g);
    int64_t base = t.rep_off[r];
    int32_t u = t.user[g], ap = t.app[g];
    int64_t ts = t.ts[g];
    bool ok_ids = u >= 0 && u < t.U && ap >= 0 && ap < t.A;
    if (!ok_ids) code = max(code, int32_t(FS_E_RANGE));
    if (ts < 0) code = max(code, int32_t(FS_E_RANGE));
    if (g > base && t.ts[g - 1] > ts) code = max(code, int32_t(FS_E_ORDER));
    if (t.call) {
      int32_t c = t.call[g];
      if (c < 0) code = max(code, int32_t(FS_E_RANGE));
      if (a.check_chain) {
        int64_t i = g - base;
        int32_t h = t.head[g], p = t.prev[g];
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
    }
    uint32_t ku = ok_ids ? uint32_t(int64_t(r) * t.U + u) : 0u;
    uint32_t ka = ok_ids ? uint32_t(ap) : 0u;
    a.key[g] = (ka << a.Bu) | ku;
    a.idx[g] = uint32_t(g);
  }
  if (code) raise_err(a.err, code);
}

// ---------------------------------------------------------------- radix sort pass

__global__ void __launch_bounds__(kThreads) k_radix_hist(const uint32_t *key, int64_t N, int shift,
                                                          uint32_t mask, uint32_t *hist,
                                                          int64_t tiles) {
  __shared__ uint32_t h[kRadix];
  const int t = threadIdx.x;
  h[t] = 0;
  __syncthreads();
  const int64_t base = blockIdx.x * int64_t(kTile);
  const int lane = t & 63;
#pragma unroll 4
  for (int i = 0; i < kItems; ++i) {
    int64_t e = base + i * kThreads + t;
    bool valid = e < N;
    uint32_t d = valid ? (key[e] >> shift) & mask : 0u;
    // aggregate equal digits within the wave before touching LDS
    uint64_t peers = __ballot(valid);
    for (int b = 0; b < kRadixBits; ++b) {
      uint64_t m = __ballot((d >> b) & 1u);
      peers &= ((d >> b) & 1u) ? m : ~m;
    }
    if (valid && (peers & ((uint64_t(1) << lane) - 1)) == 0)
      atomicAdd(&h[d], uint32_t(__popcll(peers)));
  }
  __syncthreads();
  hist[int64_t(t) * tiles + blockIdx.x] = h[t];
}

__global__ void __launch_bounds__(kThreads) k_radix_scatter(const uint32_t *kin,
                                                             const uint32_t *iin, uint32_t *kout,
                                                             uint32_t *iout, int64_t N, int shift,
                                                             uint32_t mask, const uint32_t *offs,
                                                             int64_t tiles) {
  __shared__ uint32_t s_key[kTile];
  __shared__ uint32_t s_idx[kTile];
  __shared__ uint32_t run[kRadix];
  __shared__ uint32_t wcnt[kThreads / 64][kRadix];
  __shared__ uint32_t loc[kRadix];
  __shared__ uint32_t goff[kRadix];
  __shared__ uint32_t s_waves[kThreads / 64];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int64_t base = blockIdx.x * int64_t(kTile);
  goff[t] = offs[int64_t(t) * tiles + blockIdx.x];
  run[t] = 0;
#pragma unroll
  for (int w = 0; w < kThreads / 64; ++w) wcnt[w][t] = 0;
  __syncthreads();

  uint32_t k_r[kItems], i_r[kItems], rank[kItems];
  const uint64_t lt = (uint64_t(1) << lane) - 1;
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    int64_t e = base + i * kThreads + t;
    bool valid = e < N;
    k_r[i] = valid ? kin[e] : 0u;
    i_r[i] = valid ? iin[e] : 0u;
    uint32_t d = (k_r[i] >> shift) & mask;
    uint64_t peers = __ballot(valid);
    for (int b = 0; b < kRadixBits; ++b) {
      uint64_t m = __ballot((d >> b) & 1u);
      peers &= ((d >> b) & 1u) ? m : ~m;
    }
    uint32_t rw = uint32_t(__popcll(peers & lt));
    if (valid && (peers & lt) == 0) wcnt[wave][d] = uint32_t(__popcll(peers));
    __syncthreads();
    if (valid) {
      uint32_t r = run[d] + rw;
      for (int w = 0; w < wave; ++w) r += wcnt[w][d];
      rank[i] = r;
    } else {
      rank[i] = 0xffffffffu;
    }
    __syncthreads();
    uint32_t add = 0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) {
      add += wcnt[w][t];
      wcnt[w][t] = 0;
    }
    run[t] += add;
    __syncthreads();
  }
  // tile-local exclusive offsets of each digit
  uint32_t total;
  uint32_t incl = block_inclusive_scan(run[t], s_waves, total);
  loc[t] = incl - run[t];
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    if (rank[i] != 0xffffffffu) {
      uint32_t d = (k_r[i] >> shift) & mask;
      uint32_t pos = loc[d] + rank[i];
      s_key[pos] = k_r[i];
      s_idx[pos] = i_r[i];
    }
  }
  __syncthreads();
  const int64_t n_here = N - base < kTile ? N - base : kTile;
  for (int j = t; j < n_here; j += kThreads) {
    uint32_t k = s_key[j];
    uint32_t d = (k >> shift) & mask;
    uint32_t dst = goff[d] + (uint32_t(j) - loc[d]);
    if (dst < N) {
      kout[dst] = k;
      iout[dst] = s_idx[j];
    }
  }
}

// ---------------------------------------------------------------- exclusive scan (u32)

__global__ void __launch_bounds__(kScanThreads) k_scan_partials(const uint32_t *in, int64_t n,
                                                                 uint32_t *part) {
  __shared__ uint32_t s_waves[kScanThreads / 64];
  const int64_t base = blockIdx.x * int64_t(kScanChunk);
  uint32_t v = 0;
  for (int i = 0; i < kScanItems; ++i) {
    int64_t e = base + int64_t(i) * kScanThreads + threadIdx.x;
    if (e < n) v += in[e];
  }
  uint32_t total;
  block_inclusive_scan(v, s_waves, total);
  if (threadIdx.x == 0) part[blockIdx.x] = total;
}

__global__ void __launch_bounds__(kScanThreads) k_scan_spine(uint32_t *part, int64_t n_part) {
  __shared__ uint32_t s_waves[kScanThreads / 64];
  uint32_t carry = 0;
  for (int64_t base = 0; base < n_part; base += kScanThreads) {
    int64_t e = base + threadIdx.x;
    uint32_t v = e < n_part ? part[e] : 0;
    uint32_t total;
    uint32_t incl = block_inclusive_scan(v, s_waves, total);
    if (e < n_part) part[e] = carry + incl - v;
    carry += total;
  }
}

__global__ void __launch_bounds__(kScanThreads) k_scan_apply(const uint32_t *in, int64_t n,
                                                              const uint32_t *part, uint32_t *out) {
  __shared__ uint32_t s_waves[kScanThreads / 64];
  const int64_t base = blockIdx.x * int64_t(kScanChunk);
  // blocked arrangement: thread owns kScanItems consecutive elements
  uint32_t v[kScanItems];
  uint32_t sum = 0;
  for (int i = 0; i < kScanItems; ++i) {
    int64_t e = base + int64_t(threadIdx.x) * kScanItems + i;
    v[i] = e < n ? in[e] : 0;
    sum += v[i];
  }
  uint32_t total;
  uint32_t incl = block_inclusive_scan(sum, s_waves, total);
  uint32_t run = part[blockIdx.x] + incl - sum;
  for (int i = 0; i < kScanItems; ++i) {
    int64_t e = base + int64_t(threadIdx.x) * kScanItems + i;
    if (e < n) out[e] = run;
    run += v[i];
  }
}


// ---------------------------------------------------------------- window tests

struct TestArgs {
  const uint32_t *key;
  const uint32_t *idx;
  int64_t N;
  uint32_t cmp_mask;  // key bits that identify the key (user, or user and app)
  int Bu;
  bool per_app;       // limit from t_app[key >> Bu], else t_user
  int32_t t_user;
  const int32_t *t_app;
  int32_t A;
  const int64_t *ts;
  int64_t window;
  uint8_t *flag;      // [N] stream order
  int32_t *cnt;       // [N] stream order, optional
};

__global__ void __launch_bounds__(kThreads) k_thr_test(TestArgs a) {
  for (int64_t p = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; p < a.N;
       p += int64_t(gridDim.x) * blockDim.x) {
    uint32_t kp = a.key[p];
    uint32_t k = kp & a.cmp_mask;
    uint32_t g = a.idx[p];
    if (g >= a.N) continue;
    int64_t T;
    if (a.per_app) {
      uint32_t ap = kp >> a.Bu;
      T = ap < uint32_t(a.A) ? a.t_app[ap] : 0;
    } else {
      T = a.t_user;
    }
    int64_t lo = a.ts[g] - a.window;  // window is (ts - W, ts]
    uint8_t f = 0;
    if (T <= p) {
      int64_t q = p - T;
      uint32_t gq = a.idx[q];
      if ((a.key[q] & a.cmp_mask) == k && gq < a.N && a.ts[gq] > lo) f = 1;
    }
    a.flag[g] = f;
    if (a.cnt) {
      // first position of this key: keys are sorted by the compared bits
      int64_t l = 0, h = p;
      while (l < h) {
        int64_t m = (l + h) >> 1;
        if ((a.key[m] & a.cmp_mask) < k) l = m + 1; else h = m;
      }
      // first position in [l, p] whose arrival lies in the window
      int64_t h2 = p;
      while (l < h2) {
        int64_t m = (l + h2) >> 1;
        uint32_t gm = a.idx[m];
        if (gm < a.N && a.ts[gm] > lo) h2 = m; else l = m + 1;
      }
      a.cnt[g] = int32_t(p - l + 1);
    }
  }
}

// ---------------------------------------------------------------- combine

struct CombineArgs {
  DevTrace t;
  const uint8_t *eu, *ea;
  const uint8_t *overloaded;
  bool raw;
  uint32_t *bitmap;
  uint8_t *reason;
  int64_t n_words;
};

__device__ inline uint8_t raw_reason(const CombineArgs &a, int64_t g) {
  return a.eu[g] ? 1 : (a.ea[g] ? 2 : 0);
}

__global__ void __launch_bounds__(kThreads) k_thr_combine(CombineArgs a) {
  const int64_t N = a.t.N;
  const int lane = threadIdx.x & 63;
  for (int64_t base = blockIdx.x * int64_t(blockDim.x); base < N;
       base += int64_t(gridDim.x) * blockDim.x) {
    int64_t g = base + threadIdx.x;
    uint8_t code = 0;
    if (g < N) {
      uint8_t rr = raw_reason(a, g);
      if (a.raw) {
        code = rr;
      } else if (!a.t.call || a.t.call[g] == 0) {
        bool over = a.overloaded ? a.overloaded[g] != 0 : true;
        code = over ? rr : 0;
      } else {
        int32_t r = replica_of(a.t.rep_off, a.t.R, g);
        int64_t lo = a.t.rep_off[r], hi = a.t.rep_off[r + 1];
        int64_t h = lo + a.t.head[g];
        if (h >= lo && h < hi) {
          bool hover = a.overloaded ? a.overloaded[h] != 0 : true;
          code = (hover && raw_reason(a, h) != 0) ? 3 : 0;
        }
      }
      if (a.reason) a.reason[g] = code;
    }
    uint64_t bits = __ballot(g < N && code != 0);
    if (lane == 0) {
      int64_t w = (base + (threadIdx.x & ~63)) >> 5;
      if (w < a.n_words) a.bitmap[w] = uint32_t(bits);
      if (w + 1 < a.n_words) a.bitmap[w + 1] = uint32_t(bits >> 32);
    }
  }
}

int grid_for(int64_t n, int threads) {
  int64_t b = (n + threads - 1) / threads;
  if (b < 1) b = 1;
  if (b > 131072) b = 131072;
  return int(b);
}

}  // namespace

size_t scan_partials_bytes(int64_t n) { return size_t((n + kScanChunk - 1) / kScanChunk + 1) * 4; }

hipError_t exclusive_scan(uint32_t *data, int64_t n, uint32_t *part, hipStream_t s) {
  int64_t blocks = (n + kScanChunk - 1) / kScanChunk;
  if (blocks < 1) return hipSuccess;
  hipLaunchKernelGGL(k_scan_partials, dim3(blocks), dim3(kScanThreads), 0, s, data, n, part);
  hipLaunchKernelGGL(k_scan_spine, dim3(1), dim3(kScanThreads), 0, s, part, blocks);
  hipLaunchKernelGGL(k_scan_apply, dim3(blocks), dim3(kScanThreads), 0, s, data, n, part, data);
  return hipGetLastError();
}

size_t throttle_workspace_bytes(const fs_trace *t) { return layout(t).total; }

hipError_t launch_throttle(const fs_trace *t, const fs_limits *lim, const uint8_t *overloaded,
                           uint32_t flags, uint32_t *bitmap, uint8_t *reason, int32_t *cnt_user,
                           int32_t *cnt_app, void *ws, int32_t *err, hipStream_t s) {
  Layout L = layout(t);
  if (L.Bu + L.Ba > 32) return hipErrorInvalidValue;
  if (L.N == 0) return hipSuccess;
  char *w = static_cast<char *>(ws);
  uint32_t *keyA = reinterpret_cast<uint32_t *>(w + L.off_keyA);
  uint32_t *idxA = reinterpret_cast<uint32_t *>(w + L.off_idxA);
  uint32_t *keyB = reinterpret_cast<uint32_t *>(w + L.off_keyB);
  uint32_t *idxB = reinterpret_cast<uint32_t *>(w + L.off_idxB);
  uint8_t *eu = reinterpret_cast<uint8_t *>(w + L.off_eu);
  uint8_t *ea = reinterpret_cast<uint8_t *>(w + L.off_ea);
  uint32_t *hist = reinterpret_cast<uint32_t *>(w + L.off_hist);
  uint32_t *part = reinterpret_cast<uint32_t *>(w + L.off_part);
  int32_t *tapp = reinterpret_cast<int32_t *>(w + L.off_tapp);
  const bool raw = (flags & FS_THROTTLE_RAW) != 0;
  hipError_t e = hipMemcpyAsync(tapp, lim->t_app_h, sizeof(int32_t) * t->n_apps,
                                hipMemcpyHostToDevice, s);
  if (e != hipSuccess) return e;

  InitArgs ia{dev_trace(t), L.Bu, !raw, keyA, idxA, err};
  hipLaunchKernelGGL(k_thr_init, dim3(grid_for(L.N, kThreads)), dim3(kThreads), 0, s, ia);

  uint32_t *kin = keyA, *iin = idxA, *kout = keyB, *iout = idxB;
  auto pass = [&](int shift, int width) {
    uint32_t mask = (1u << width) - 1u;
    hipLaunchKernelGGL(k_radix_hist, dim3(L.tiles), dim3(kThreads), 0, s, kin, L.N, shift, mask,
                       hist, L.tiles);
    (void)exclusive_scan(hist, int64_t(kRadix) * L.tiles, part, s);
    hipLaunchKernelGGL(k_radix_scatter, dim3(L.tiles), dim3(kThreads), 0, s, kin, iin, kout,
                       iout, L.N, shift, mask, hist, L.tiles);
    uint32_t *tk = kin, *ti = iin;
    kin = kout; iin = iout; kout = tk; iout = ti;
  };
  for (int sh = 0; sh < L.Bu; sh += kRadixBits) pass(sh, L.Bu - sh < kRadixBits ? L.Bu - sh : kRadixBits);

  const uint32_t umask = L.Bu >= 32 ? 0xffffffffu : ((1u << L.Bu) - 1u);
  TestArgs ta{kin, iin, L.N, umask, L.Bu, false, lim->t_user, tapp, t->n_apps, t->ts_us,
              lim->window_us, eu, cnt_user};
  hipLaunchKernelGGL(k_thr_test, dim3(grid_for(L.N, kThreads)), dim3(kThreads), 0, s, ta);

  for (int sh = L.Bu; sh < L.Bu + L.Ba; sh += kRadixBits) {
    int end = L.Bu + L.Ba;
    pass(sh, end - sh < kRadixBits ? end - sh : kRadixBits);
  }
  TestArgs tb{kin, iin, L.N, 0xffffffffu, L.Bu, true, lim->t_user, tapp, t->n_apps, t->ts_us,
              lim->window_us, ea, cnt_app};
  hipLaunchKernelGGL(k_thr_test, dim3(grid_for(L.N, kThreads)), dim3(kThreads), 0, s, tb);

  CombineArgs ca{dev_trace(t), eu, ea, overloaded, raw, bitmap, reason, (L.N + 31) / 32};
  hipLaunchKernelGGL(k_thr_combine, dim3(grid_for(L.N, kThreads)), dim3(kThreads), 0, s, ca);
  return hipGetLastError();
}

}  // namespace fs

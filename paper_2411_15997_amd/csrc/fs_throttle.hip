// OIT sliding-window limit test (Alg. 1 monitoring stream: every arrival is counted
// per user and per (user, app); Sec. 4, OIT: the user limit is checked first, then
// the app limit; a later call of an interaction is never checked and shares its
// first call's fate).
//
// Method.  For a key k (a user, or a (user, app) pair) let the key's records be
// taken in stream order.  The window count of record i exceeds T iff the record T
// positions earlier in the same key sequence exists and arrived after ts_i - W
// (the T+1 most recent arrivals of the key, i included, all lie in the window).
// So the test is O(1) once each key's records are contiguous in stream order.
//
// Every record becomes one 64-bit element, most significant field first:
//   key   B_k bits   (app << B_u) | (replica * U + user)
//   index B_i bits   global record index
//   time  B_q bits   (ts - ts of the replica's first record) >> sh, sh the smallest
//                    shift that fits every replica's span
//   flag  1 bit      user limit exceeded (set by the pass that tests it)
// A stable LSD radix sort over the user bits of the key gives each user's records
// in stream order; the first radix pass over the app bits tests the user limit as it
// reads that order and sets the flag; after the app passes every (user, app) pair
// is contiguous and the app limit is tested.  The result goes back to stream order
// with one scatter through the index field.  The window test on the quantised
// time is exact whenever it is decisive (the interval of possible gaps lies wholly
// below or above W) and falls back to the two exact arrival times otherwise.
// Radix pass: per-tile digit histograms (the first one fused into element
// construction), a device-wide exclusive scan, then a stable scatter (wave-match
// ranking, the tile reordered in LDS so the global writes of each digit run are
// contiguous).
//
// Fused path (user limit T_u <= kHaloMax, per-(user, app) key, no window counts
// asked for): only the user bits are sorted, and one kernel tests both limits in user
// order.  When the user limit holds, the user has at most T_u requests in the window,
// all among its last T_u positions; so the app limit is exceeded iff the T_a-th
// previous request of the same app within those positions is in the window.  A tile
// keeps T_u positions of halo in LDS and finds that request through a stable counting
// sort of its positions by app (the T_a-th previous entry of the app's list, checked
// to be the same user's and recent enough).  Only the requests whose reason
// is used are stored (every request raw; first calls gated), as bytes over a fill with
// the likelier reason (estimated from a sample of the user test).
#include <algorithm>

#include "fs_device.h"
#include "fs_launch.h"

namespace fs {
namespace {

constexpr int kThreads = 256;
constexpr int kItems = 16;
constexpr int kTile = kThreads * kItems;  // 4096 records per radix tile
constexpr int kRadixBits = 8;              // widest digit
constexpr int kRadix = 1 << kRadixBits;
constexpr int kScanThreads = 1024;
constexpr int kScanItems = 4;
constexpr int kScanChunk = kScanThreads * kScanItems;
// Records over the user limit are counted in kFlagSlots counters, one per 64-byte line
// (a work-group adds to counter blockIdx % kFlagSlots), after the time shift's line.
constexpr int kFlagSlots = 64;
constexpr int kFlagStride = 16;

int bits_for(int64_t n_values) {  // bits to represent 0 .. n_values-1 (at least 1)
  int b = 1;
  while ((int64_t(1) << b) < n_values) ++b;
  return b;
}

size_t up(size_t x) { return (x + 255) / 256 * 256; }

// Field positions of the packed element.
struct Pack {
  int Bu, Ba, Bk, Bi, Bq;
  int SK;  // key shift (64 - Bk)
  int SI;  // index shift (1 + Bq)
  uint64_t imask, qmask;
};

Pack make_pack(const fs_trace *t, int64_t N) {
  Pack p;
  p.Bu = bits_for(int64_t(t->n_replicas) * t->n_users);
  p.Ba = bits_for(t->n_apps);
  p.Bk = p.Bu + p.Ba;
  p.Bi = bits_for(N > 0 ? N : 1);
  p.Bq = 64 - p.Bk - p.Bi - 1;
  if (p.Bq < 0) p.Bq = 0;
  p.SK = 64 - p.Bk;
  p.SI = 1 + p.Bq;
  p.imask = (uint64_t(1) << p.Bi) - 1;
  p.qmask = p.Bq > 0 ? (uint64_t(1) << p.Bq) - 1 : 0;
  return p;
}

struct Layout {
  int64_t N;
  int64_t tiles;
  Pack pk;
  size_t off_a, off_b, off_dig, off_hist, off_part, off_tapp, off_sh;
  size_t total;
};

Layout layout(const fs_trace *t) {
  Layout L;
  L.N = t->rep_off_h[t->n_replicas];
  L.tiles = (L.N + kTile - 1) / kTile;
  L.pk = make_pack(t, L.N);
  size_t n = size_t(L.N > 0 ? L.N : 1);
  size_t hist_len = size_t(kRadix) * size_t(L.tiles > 0 ? L.tiles : 1);
  size_t o = 0;
  L.off_a = o; o += up(n * 8);
  L.off_b = o; o += up(n * 8);
  L.off_dig = o; o += up(n);  // the next pass's digit of each element, one byte
  L.off_hist = o; o += up(hist_len * 4);
  L.off_part = o; o += up(((hist_len + kScanChunk - 1) / kScanChunk + 1) * 4);
  L.off_tapp = o; o += up(kMaxApps * 4);
  L.off_sh = o; o += up(4 * kFlagStride * (kFlagSlots + 1));  // time shift, flag counters
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

// Lanes of the wave holding the same digit as this lane (one ballot per digit bit;
// `width` is the digit's bit count, at most kRadixBits).
__device__ inline uint64_t digit_peers(uint32_t d, bool valid, int width) {
  const uint64_t v = __ballot(valid);
  uint32_t lo = uint32_t(v), hi = uint32_t(v >> 32);
  for (int b = 0; b < width; ++b) {
    // s: all ones where the lane's bit b is set; m: the lanes whose bit b is set.  A
    // lane keeps the lanes where m agrees with its own bit: those of ~(m ^ s).
    const uint32_t s = uint32_t(__builtin_amdgcn_sbfe(int32_t(d), uint32_t(b), 1u));
    const uint64_t m = __builtin_amdgcn_uicmp(s, 0u, 33);  // the ballot of s != 0
    lo &= ~(uint32_t(m) ^ s);
    hi &= ~(uint32_t(m >> 32) ^ s);
  }
  return (uint64_t(hi) << 32) | lo;
}

__host__ __device__ inline int mask_width(uint32_t mask) {
  int w = 0;
  while (w < 32 && (mask >> w) != 0) ++w;
  return w;
}

// Adds one item row to the tile histogram in LDS.  Narrow digits (few bins, so many
// lanes of a wave share one) are aggregated per wave first.  Wide digits go straight to
// LDS atomics on one of kHistCopies copies of the histogram chosen by the lane's low
// bits: lanes of a heavy key's digit then add to different words in different banks
// (each copy is padded by one word) instead of stalling on one address.
constexpr int kPlainHistWidth = 6;
constexpr int kHistCopies = 8;
constexpr int kHistStride = kRadix + 1;
constexpr int kHistWords = kHistCopies * kHistStride;
__device__ inline void hist_add(uint32_t *h, uint32_t d, bool valid, int width) {
  if (width >= kPlainHistWidth) {
    if (valid) atomicAdd(&h[(threadIdx.x & (kHistCopies - 1)) * kHistStride + d], 1u);
    return;
  }
  const int lane = threadIdx.x & 63;
  const uint64_t peers = digit_peers(d, valid, width);
  if (valid && (peers & ((uint64_t(1) << lane) - 1)) == 0) atomicAdd(&h[d], uint32_t(__popcll(peers)));
}

// Bin b of the tile histogram: the sum of its copies (narrow digits use copy 0 only).
__device__ inline uint32_t hist_total(const uint32_t *h, int b) {
  uint32_t v = 0;
#pragma unroll
  for (int c = 0; c < kHistCopies; ++c) v += h[c * kHistStride + b];
  return v;
}

// Work-groups are dealt to the 8 XCDs round robin (block b runs on XCD b % 8).  This
// maps blocks to tiles so that each XCD sweeps one contiguous range of tiles in
// order; a record's interaction links then point mostly into data that XCD's own
// L2 has just cached.
__device__ inline int64_t xcd_tile(int64_t b, int64_t n) {
  const int64_t x = b & 7, i = b >> 3, per = n >> 3, extra = n & 7;
  return x * per + (x < extra ? x : extra) + i;
}

// ---------------------------------------------------------------- window test

struct Win {
  int64_t W;
  const int32_t *sh_dev;  // written on the device by k_thr_span
  int sh;                 // loaded from sh_dev at the start of each kernel
  bool has_q;
  Pack pk;
  const int64_t *ts;
};

__device__ inline Win load_win(const Win &w) {
  Win v = w;
  v.sh = *w.sh_dev;
  return v;
}

// Is ts(p) - ts(q) < W for two records of the same key, q earlier in the stream?
__device__ inline bool in_window(uint64_t ep, uint64_t eq, const Win &w) {
  if (w.has_q) {
    const uint64_t tp = (ep >> 1) & w.pk.qmask, tq = (eq >> 1) & w.pk.qmask;
    const uint64_t d = tp - tq;
    const uint64_t span = (uint64_t(1) << w.sh) - 1;  // the quantisation error bound
    const uint64_t mid = d << w.sh;
    // the true gap lies in [mid - span, mid + span]
    if (mid + span < uint64_t(w.W)) return true;
    if (mid >= span && mid - span >= uint64_t(w.W)) return false;
  }
  const int64_t gp = int64_t((ep >> w.pk.SI) & w.pk.imask);
  const int64_t gq = int64_t((eq >> w.pk.SI) & w.pk.imask);
  return w.ts[gp] - w.ts[gq] < w.W;
}

// ---------------------------------------------------------------- shift of the time field

__global__ void __launch_bounds__(kThreads) k_thr_span(const int64_t *rep_off, const int64_t *ts,
                                                        int32_t R, int Bq, int32_t *sh_out) {
  __shared__ int64_t s_max[kThreads];
  int64_t m = 0;
  for (int32_t r = threadIdx.x; r < R; r += kThreads) {
    const int64_t a = rep_off[r], b = rep_off[r + 1];
    if (b > a) {
      const int64_t span = ts[b - 1] - ts[a];
      m = span > m ? span : m;
    }
  }
  s_max[threadIdx.x] = m;
  __syncthreads();
  for (int s = kThreads / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s && s_max[threadIdx.x + s] > s_max[threadIdx.x])
      s_max[threadIdx.x] = s_max[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    int sh = 0;
    if (Bq > 0)
      while (sh < 63 && (uint64_t(s_max[0]) >> sh) >= (uint64_t(1) << Bq)) ++sh;
    sh_out[0] = sh;
  }
  if (threadIdx.x < kFlagSlots) sh_out[kFlagStride * (threadIdx.x + 1)] = 0;  // user-test counts
}

// ---------------------------------------------------------------- element construction

struct InitArgs {
  DevTrace t;
  Pack pk;
  bool gated;      // gated mode: checks the links to the first calls
  int mark;        // flag bit: 0 none, 1 every request, 2 first calls only
  const int32_t *sh;
  uint64_t *el;
  int shift;      // first radix digit
  uint32_t mask;
  uint32_t *hist;
  int64_t tiles;
  int32_t *err;
  const uint8_t *uflag;  // when set: the flag bit is this byte per request (stream order)
};

// Builds the elements of one tile in stream order, checks the fields the throttle
// reads, and counts the tile's first radix digit.
__global__ void __launch_bounds__(kThreads) k_thr_init(InitArgs a) {
  __shared__ uint32_t h[kHistWords];
  __shared__ int32_t s_r0;
  const int t = threadIdx.x;
  const DevTrace &tr = a.t;
  const int64_t tile = xcd_tile(blockIdx.x, gridDim.x);
  const int64_t base = tile * kTile;
  for (int j = t; j < kHistWords; j += kThreads) h[j] = 0;
  if (t == 0) s_r0 = replica_of(tr.rep_off, tr.R, base);
  __syncthreads();
  const int sh = *a.sh;
  const int width = mask_width(a.mask);
  int32_t r = s_r0;
  int64_t r_end = tr.rep_off[r + 1], r_base = tr.rep_off[r];
  int64_t ts_base = tr.ts[r_base];
  int32_t code = 0;
  for (int i = 0; i < kItems; ++i) {
    const int64_t g = base + int64_t(i) * kThreads + t;
    const bool valid = g < tr.N;
    uint32_t d = 0;
    if (valid) {
      if (g >= r_end) {
        while (g >= tr.rep_off[r + 1]) ++r;
        r_base = tr.rep_off[r];
        r_end = tr.rep_off[r + 1];
        ts_base = tr.ts[r_base];
      }
      const int32_t u = tr.user[g], ap = tr.app[g];
      const int64_t ts = tr.ts[g];
      const bool ok_ids = u >= 0 && u < tr.U && ap >= 0 && ap < tr.A;
      if (!ok_ids) code = max(code, int32_t(FS_E_RANGE));
      if (ts < 0) code = max(code, int32_t(FS_E_RANGE));
      if (g > r_base && tr.ts[g - 1] > ts) code = max(code, int32_t(FS_E_ORDER));
      bool first = true;
      if (tr.head && a.gated) {  // the only link the gated mode follows: to the first call
        const int64_t li = g - r_base;
        const int32_t hd = tr.head[g];
        if (hd < 0 || hd > li) code = max(code, int32_t(FS_E_RANGE));
        first = hd == li;
      }
      const uint64_t key = ok_ids ? ((uint64_t(ap) << a.pk.Bu) | uint64_t(int64_t(r) * tr.U + u)) : 0;
      uint64_t q = 0;
      if (a.pk.Bq > 0) {
        const int64_t rel = ts - ts_base;
        q = rel > 0 ? uint64_t(rel) >> sh : 0;
        if (q > a.pk.qmask) q = a.pk.qmask;  // only for unsorted input, which is an error
      }
      const uint64_t fl = a.uflag ? (a.uflag[g] != 0 ? 1u : 0u)
                                  : ((a.mark == 1 || (a.mark == 2 && first)) ? 1u : 0u);
      const uint64_t e = (key << a.pk.SK) | (uint64_t(g) << a.pk.SI) | (q << 1) | fl;
      a.el[g] = e;
      d = uint32_t(e >> (a.pk.SK + a.shift)) & a.mask;
    }
    hist_add(h, d, valid, width);
  }
  if (code) raise_err(a.err, code);
  __syncthreads();
  if (t <= int(a.mask)) a.hist[int64_t(t) * a.tiles + tile] = hist_total(h, t);
}

// ---------------------------------------------------------------- radix sort pass

__global__ void __launch_bounds__(kThreads) k_radix_hist(const uint64_t *el, int64_t N, int shift,
                                                          uint32_t mask, uint32_t *hist,
                                                          int64_t tiles) {
  __shared__ uint32_t h[kHistWords];
  const int t = threadIdx.x;
  for (int j = t; j < kHistWords; j += kThreads) h[j] = 0;
  __syncthreads();
  const int64_t base = blockIdx.x * int64_t(kTile);
  const int width = mask_width(mask);
#pragma unroll 4
  for (int i = 0; i < kItems; ++i) {
    const int64_t e = base + i * kThreads + t;
    const bool valid = e < N;
    const uint32_t d = valid ? uint32_t(el[e] >> shift) & mask : 0u;
    hist_add(h, d, valid, width);
  }
  __syncthreads();
  if (t <= int(mask)) hist[int64_t(t) * tiles + blockIdx.x] = hist_total(h, t);
}

// The same tile histogram from the digits the previous pass's scatter wrote out, one byte
// per element at its new position: 1 byte read per element instead of 8.  Thread t
// counts the tile's 16 consecutive elements from 16 t.
__global__ void __launch_bounds__(kThreads) k_radix_hist8(const uint8_t *dig, int64_t N,
                                                           uint32_t mask, uint32_t *hist,
                                                           int64_t tiles) {
  static_assert(kTile == kThreads * 16, "one 16-byte load per thread");
  __shared__ uint32_t h[kHistWords];
  const int t = threadIdx.x;
  for (int j = t; j < kHistWords; j += kThreads) h[j] = 0;
  const int64_t e0 = blockIdx.x * int64_t(kTile) + int64_t(t) * 16;
  uint32_t w[4] = {0u, 0u, 0u, 0u};
  if (e0 + 16 <= N) {
    const uint4 q = *reinterpret_cast<const uint4 *>(dig + e0);
    w[0] = q.x;
    w[1] = q.y;
    w[2] = q.z;
    w[3] = q.w;
  } else {
    for (int i = 0; i < 16; ++i)
      if (e0 + i < N) w[i >> 2] |= uint32_t(dig[e0 + i]) << (8 * (i & 3));
  }
  __syncthreads();
  const int width = mask_width(mask);
#pragma unroll
  for (int i = 0; i < 16; ++i)
    hist_add(h, (w[i >> 2] >> (8 * (i & 3))) & mask, e0 + i < N, width);
  __syncthreads();
  if (t <= int(mask)) hist[int64_t(t) * tiles + blockIdx.x] = hist_total(h, t);
}

struct ScatterArgs {
  const uint64_t *in;
  uint64_t *out;
  int64_t N;
  int shift;  // absolute bit position of the digit in the element
  uint32_t mask;
  const uint32_t *offs;
  int64_t tiles;
  // user-limit test on the way through (the input is in user order)
  int32_t t_user;
  uint64_t user_mask;  // element bits of the user part of the key
  Win win;
  int32_t *n_flag;     // counters of records over the user limit (TEST_USER)
  uint8_t *next_dig;   // when set: each element's next digit, at its new position
  int next_shift;
  uint32_t next_mask;
};

// Stable scatter of one tile.  Wave w owns the contiguous sub-tile
// [w * kWaveSpan, (w + 1) * kWaveSpan) and ranks its rows in order against a
// wave-private digit counter, so the tile needs only a handful of barriers; the
// waves' counts then give each digit's offset per wave and per tile.
constexpr int kWaves = kThreads / 64;
constexpr int kWaveSpan = kTile / kWaves;  // 1024 records, kItems rows of 64

template <bool TEST_USER>
__global__ void __launch_bounds__(kThreads) k_radix_scatter(ScatterArgs a) {
  __shared__ uint64_t s_el[kTile];
  __shared__ uint32_t cnt[kWaves][kRadix];
  __shared__ uint32_t loc[kRadix];
  __shared__ uint32_t goff[kRadix];
  __shared__ uint32_t s_waves[kWaves];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int64_t base = blockIdx.x * int64_t(kTile);
  const int64_t wbase = base + int64_t(wave) * kWaveSpan;
  const Win win = TEST_USER ? load_win(a.win) : a.win;
  goff[t] = t <= int(a.mask) ? a.offs[int64_t(t) * a.tiles + blockIdx.x] : 0u;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) cnt[w][t] = 0;
  __syncthreads();

  uint64_t k_r[kItems];
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const int64_t e = wbase + i * 64 + lane;
    k_r[i] = e < a.N ? a.in[e] : 0u;
  }
  if (TEST_USER) {
    int32_t nf = 0;
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
      const int64_t e = wbase + i * 64 + lane;
      if (e < a.N && int64_t(a.t_user) <= e) {
        const uint64_t eq = a.in[e - a.t_user];
        if (((k_r[i] ^ eq) & a.user_mask) == 0 && in_window(k_r[i], eq, win)) k_r[i] |= 1u;
      }
      nf += __popcll(__ballot(k_r[i] & 1u));
    }
    if (lane == 0 && nf) atomicAdd(a.n_flag + kFlagStride * (blockIdx.x % kFlagSlots), nf);
  }
  uint32_t rank[kItems];
  const uint64_t lt = (uint64_t(1) << lane) - 1;
  uint32_t *my = cnt[wave];
  const int width = mask_width(a.mask);
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const int64_t e = wbase + i * 64 + lane;
    const bool valid = e < a.N;
    const uint32_t d = uint32_t(k_r[i] >> a.shift) & a.mask;
    const uint64_t peers = digit_peers(d, valid, width);
    const uint32_t before = valid ? my[d] : 0u;  // this wave's earlier rows with digit d
    rank[i] = valid ? before + uint32_t(__popcll(peers & lt)) : 0xffffffffu;
    if (valid && (peers & lt) == 0) my[d] = before + uint32_t(__popcll(peers));
  }
  __syncthreads();
  // per digit: offsets of the waves within the digit, then tile-local digit offsets
  uint32_t tot = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const uint32_t c = cnt[w][t];
    cnt[w][t] = tot;
    tot += c;
  }
  uint32_t total;
  const uint32_t incl = block_inclusive_scan(tot, s_waves, total);
  loc[t] = incl - tot;
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    if (rank[i] != 0xffffffffu) {
      const uint32_t d = uint32_t(k_r[i] >> a.shift) & a.mask;
      s_el[loc[d] + my[d] + rank[i]] = k_r[i];
    }
  }
  __syncthreads();
  const int64_t n_here = a.N - base < kTile ? a.N - base : kTile;
  for (int j = t; j < n_here; j += kThreads) {
    const uint64_t el = s_el[j];
    const uint32_t d = uint32_t(el >> a.shift) & a.mask;
    const uint32_t dst = goff[d] + (uint32_t(j) - loc[d]);
    if (dst < a.N) {
      a.out[dst] = el;
      if (a.next_dig) a.next_dig[dst] = uint8_t(uint32_t(el >> a.next_shift) & a.next_mask);
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

// ---------------------------------------------------------------- keys

// The key an element is counted under, as an ordered value: its masked key bits, or
// for the app-level limit (app, replica), the replica being (replica * U + user) / U.
struct KeySel {
  uint64_t mask;  // element bits of the key (per-user and per-(user, app) keys)
  bool app_level;
  int SK, Bu;
  uint32_t U;
};
__device__ inline uint64_t key_of(uint64_t e, const KeySel &k) {
  if (!k.app_level) return e & k.mask;
  const uint64_t ru = (e >> k.SK) & ((uint64_t(1) << k.Bu) - 1);
  return ((e >> (k.SK + k.Bu)) << 32) | (ru / k.U);
}

// ---------------------------------------------------------------- app-limit test

// The app limit is tested in (user, app) order.  Each record's raw reason (the user
// flag carried by the element, else the app test) goes to its stream position as one
// byte.  Those stores are scattered, so the array is first filled with the likelier
// reason (1 when most records are over the user limit, else 0) in coalesced stores
// and only the records with another reason are stored one by one.
// Called by every thread of the block.
__device__ inline uint8_t background_reason(const int32_t *n_flag, int64_t N) {
  __shared__ uint8_t s_bg;
  if (threadIdx.x < 64) {
    int64_t c = threadIdx.x < kFlagSlots ? n_flag[kFlagStride * threadIdx.x] : 0;
#pragma unroll
    for (int d = 32; d > 0; d >>= 1) c += __shfl_xor(c, d, 64);
    if (threadIdx.x == 0) s_bg = c * 2 > N ? 1 : 0;
  }
  __syncthreads();
  return s_bg;
}

__global__ void __launch_bounds__(kThreads) k_thr_fill(uint8_t *rb, int64_t N,
                                                        const int32_t *n_flag) {
  const uint32_t v = uint32_t(background_reason(n_flag, N)) * 0x01010101u;
  const uint4 q = make_uint4(v, v, v, v);
  const int64_t n16 = N >> 4;
  uint4 *r4 = reinterpret_cast<uint4 *>(rb);
  for (int64_t i = blockIdx.x * int64_t(kThreads) + threadIdx.x; i < n16;
       i += int64_t(gridDim.x) * kThreads)
    r4[i] = q;
  if (blockIdx.x == 0 && threadIdx.x < (N & 15)) rb[(n16 << 4) + threadIdx.x] = uint8_t(v);
}

struct AppTestArgs {
  const uint64_t *el;  // the app key's order (time order within a key), user flag set
  int64_t N;
  KeySel key;          // the app key
  const int32_t *t_app;
  int32_t A;
  Win win;
  uint8_t *rb;         // [N] raw reasons in stream order, filled with the background
  const int32_t *n_flag;
};

__global__ void __launch_bounds__(kThreads) k_thr_apptest(AppTestArgs a) {
  const Win win = load_win(a.win);
  const Pack &pk = win.pk;
  const uint8_t bg = background_reason(a.n_flag, a.N);
  const int64_t base = blockIdx.x * int64_t(kTile) + threadIdx.x;
  uint64_t ep[kItems];
  int64_t T[kItems];
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const int64_t p = base + i * kThreads;
    ep[i] = p < a.N ? a.el[p] : 0u;
  }
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const int64_t p = base + i * kThreads;
    const uint32_t ap = uint32_t((ep[i] >> pk.SK) >> pk.Bu);
    T[i] = (p < a.N && ap < uint32_t(a.A)) ? a.t_app[ap] : INT64_MAX;
  }
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const int64_t p = base + i * kThreads;
    if (p >= a.N) continue;
    bool fa = false;
    if (T[i] <= p) {
      const uint64_t eq = a.el[p - T[i]];
      fa = key_of(ep[i], a.key) == key_of(eq, a.key) && in_window(ep[i], eq, win);
    }
    const uint8_t code = (ep[i] & 1u) ? 1 : (fa ? 2 : 0);
    if (code != bg) a.rb[(ep[i] >> pk.SI) & pk.imask] = code;
  }
}

// ---------------------------------------------------------------- fused limit tests

constexpr int kHaloMax = 1024;              // largest user limit the fused path takes
constexpr int kFTile = 4096;                // positions tested per work-group
constexpr int kFThreads = 512;              // threads of a fused work-group
constexpr int kFSpan = kFTile + kHaloMax;   // elements held in LDS (tile and halo)

// Background of the fused path: 1 when most sampled requests whose reason is stored
// are over the user limit, else 0 (counts in slots 0 and 1 of the flag counters).
__device__ inline uint8_t fused_background(const int32_t *n_flag) {
  return int64_t(n_flag[kFlagStride]) * 2 > int64_t(n_flag[0]) ? 1 : 0;
}

struct SampleArgs {
  const uint64_t *el;  // user order
  int64_t N;
  int32_t t_user;
  uint64_t user_mask;
  Win win;
  int32_t *n_flag;
};

// The user test on every 997th position (a sample for the background's choice).
constexpr int kSampleStride = 997;
__global__ void __launch_bounds__(kThreads) k_thr_sample(SampleArgs a) {
  const Win win = load_win(a.win);
  int32_t flagged = 0, over = 0;
  const int64_t ns = (a.N + kSampleStride - 1) / kSampleStride;
  for (int64_t k = blockIdx.x * int64_t(kThreads) + threadIdx.x; k < ns;
       k += int64_t(gridDim.x) * kThreads) {
    const int64_t p = k * kSampleStride;
    const uint64_t e = a.el[p];
    if (!(e & 1u)) continue;
    ++flagged;
    if (int64_t(a.t_user) <= p) {
      const uint64_t eq = a.el[p - a.t_user];
      if (((e ^ eq) & a.user_mask) == 0 && in_window(e, eq, win)) ++over;
    }
  }
#pragma unroll
  for (int d = 32; d > 0; d >>= 1) {
    flagged += __shfl_xor(flagged, d, 64);
    over += __shfl_xor(over, d, 64);
  }
  if ((threadIdx.x & 63) == 0) {
    if (flagged) atomicAdd(a.n_flag, flagged);
    if (over) atomicAdd(a.n_flag + kFlagStride, over);
  }
}

__global__ void __launch_bounds__(kThreads) k_thr_fill_fused(uint8_t *rb, int64_t N,
                                                              const int32_t *n_flag) {
  const uint32_t v = uint32_t(fused_background(n_flag)) * 0x01010101u;
  const uint4 q = make_uint4(v, v, v, v);
  const int64_t n16 = N >> 4;
  uint4 *r4 = reinterpret_cast<uint4 *>(rb);
  for (int64_t i = blockIdx.x * int64_t(kThreads) + threadIdx.x; i < n16;
       i += int64_t(gridDim.x) * kThreads)
    r4[i] = q;
  if (blockIdx.x == 0 && threadIdx.x < (N & 15)) rb[(n16 << 4) + threadIdx.x] = uint8_t(v);
}

struct FusedArgs {
  const uint64_t *el;  // user order (each user's requests in stream order)
  int64_t N;
  int32_t t_user;      // <= kHaloMax
  const int32_t *t_app;
  int32_t A;
  int app_bits;
  uint64_t user_mask;
  Win win;
  uint8_t *rb;         // raw reasons in stream order, filled with the background
  const int32_t *n_flag;
};

// Dynamic LDS of the fused test, sized per launch for span = T_u + kFTile positions and
// A apps: the span's elements, and its positions grouped by app (a stable counting sort:
// list[rank[j]] = j, each app's positions in order).
struct FusedLds {
  uint64_t *el;        // [span]
  int32_t *tapp;       // [A] the app limits
  uint16_t *list;      // [span]
  uint16_t *rank;      // [span]
  uint16_t *cnt;       // [kFThreads / 64][A] per wave: positions of each app so far
  uint16_t *start;     // [A] first list index of each app
  uint32_t *waves;     // [kFThreads / 64] (16-byte aligned)
};
__host__ __device__ inline size_t fused_lds_bytes(int span, int A) {
  return size_t(span) * 12 + size_t(A) * 4 + size_t(kFThreads / 64) * A * 2 + size_t(A) * 2 +
         16 + size_t(kFThreads / 64) * 4;
}
__device__ inline FusedLds fused_lds(char *base, int span, int A) {
  FusedLds sm;
  sm.el = reinterpret_cast<uint64_t *>(base);
  sm.tapp = reinterpret_cast<int32_t *>(sm.el + span);
  sm.list = reinterpret_cast<uint16_t *>(sm.tapp + A);
  sm.rank = sm.list + span;
  sm.cnt = sm.rank + span;
  sm.start = sm.cnt + (kFThreads / 64) * A;
  sm.waves = reinterpret_cast<uint32_t *>(
      (reinterpret_cast<uintptr_t>(sm.start + A) + 15) & ~uintptr_t(15));
  return sm;
}

__global__ void __launch_bounds__(kFThreads) k_thr_fused(FusedArgs a) {
  extern __shared__ __align__(16) char fused_smem[];
  const Win win = load_win(a.win);
  const Pack &pk = win.pk;
  const uint8_t bg = fused_background(a.n_flag);
  const int H = a.t_user;
  const int64_t p0 = xcd_tile(blockIdx.x, gridDim.x) * int64_t(kFTile);
  const int64_t g0 = p0 - H;  // global position of el[0]
  const int span = H + kFTile;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int A = a.A;
  const FusedLds sm = fused_lds(fused_smem, span, A);
  const uint32_t amask = (1u << pk.Ba) - 1u;
  {  // every load of the span is issued before the first store to LDS
    constexpr int kIters = (kFSpan + kFThreads - 1) / kFThreads;
    uint64_t v[kIters];
#pragma unroll
    for (int i = 0; i < kIters; ++i) {
      const int j = threadIdx.x + i * kFThreads;
      const int64_t g = g0 + j;
      v[i] = (j < span && g >= 0 && g < a.N) ? a.el[g] : 0u;
    }
    constexpr int kAppIters = (1024 + kFThreads - 1) / kFThreads;  // A <= 1024
    int32_t tv[kAppIters];
#pragma unroll
    for (int i = 0; i < kAppIters; ++i) {
      const int k = threadIdx.x + i * kFThreads;
      tv[i] = k < A ? a.t_app[k] : 0;
    }
#pragma unroll
    for (int i = 0; i < kIters; ++i) {
      const int j = threadIdx.x + i * kFThreads;
      if (j < span) sm.el[j] = v[i];
    }
#pragma unroll
    for (int i = 0; i < kAppIters; ++i) {
      const int k = threadIdx.x + i * kFThreads;
      if (k < A) sm.tapp[k] = tv[i];
    }
  }
  for (int k = threadIdx.x; k < (kFThreads / 64) * A; k += kFThreads) sm.cnt[k] = 0;
  __syncthreads();
  // 1. stable ranks by app: wave w takes rows [w * rows, (w + 1) * rows) of 64 positions
  const int n_rows = (span + 63) / 64;
  const int rows = (n_rows + kFThreads / 64 - 1) / (kFThreads / 64);
  const uint64_t lt = (uint64_t(1) << lane) - 1;
  uint16_t *const my = sm.cnt + wave * A;
  for (int rw = wave * rows; rw < (wave + 1) * rows && rw < n_rows; ++rw) {
    const int j = rw * 64 + lane;
    const int64_t g = g0 + j;
    const bool valid = j < span && g >= 0 && g < a.N;
    const uint32_t ap = valid ? uint32_t(sm.el[j] >> (pk.SK + pk.Bu)) & amask : 0u;
    const uint64_t peers = digit_peers(ap, valid, a.app_bits);
    const uint32_t before = valid ? my[ap] : 0u;
    if (valid) sm.rank[j] = uint16_t(before + __popcll(peers & lt));
    if (valid && (peers & lt) == 0) my[ap] = uint16_t(before + __popcll(peers));
  }
  __syncthreads();
  // 2. each app's list start and each wave's offset within it
  uint32_t tot4 = 0;
  uint32_t tots[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {  // apps 4t .. 4t + 3 (A <= 1024 <= 4 * kFThreads)
    const int ap = threadIdx.x * 4 + q;
    uint32_t tot = 0;
    if (ap < A) {
#pragma unroll
      for (int w = 0; w < kFThreads / 64; ++w) {
        const uint32_t c = sm.cnt[w * A + ap];
        sm.cnt[w * A + ap] = uint16_t(tot);
        tot += c;
      }
    }
    tots[q] = tot;
    tot4 += tot;
  }
  uint32_t total;
  const uint32_t incl = block_inclusive_scan(tot4, sm.waves, total);
  uint32_t run = incl - tot4;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int ap = threadIdx.x * 4 + q;
    if (ap < A) sm.start[ap] = uint16_t(run);
    run += tots[q];
  }
  __syncthreads();
  // 3. final list indices
  for (int rw = wave * rows; rw < (wave + 1) * rows && rw < n_rows; ++rw) {
    const int j = rw * 64 + lane;
    const int64_t g = g0 + j;
    if (j < span && g >= 0 && g < a.N) {
      const uint32_t ap = uint32_t(sm.el[j] >> (pk.SK + pk.Bu)) & amask;
      const uint32_t idx = uint32_t(sm.start[ap]) + sm.cnt[wave * A + ap] + sm.rank[j];
      sm.rank[j] = uint16_t(idx);
      sm.list[idx] = uint16_t(j);
    }
  }
  __syncthreads();
  // 4. the tests of the tile's positions whose reason is stored
  const int64_t n_here = a.N - p0 < kFTile ? a.N - p0 : kFTile;
  for (int t = threadIdx.x; t < n_here; t += kFThreads) {
    const int64_t p = p0 + t;
    const int j = t + H;
    const uint64_t e = sm.el[j];
    if (!(e & 1u)) continue;  // a request whose own reason is not used (a later call, gated)
    uint8_t why = 0;
    if (int64_t(H) <= p) {  // the user limit: the T_u-th previous request of the user
      const uint64_t eq = sm.el[j - H];
      if (((e ^ eq) & a.user_mask) == 0 && in_window(e, eq, win)) why = 1;
    }
    if (!why) {
      const uint32_t ap = uint32_t(e >> (pk.SK + pk.Bu)) & amask;
      const int32_t ta = ap < uint32_t(A) ? sm.tapp[ap] : INT32_MAX;
      if (ta == 0) {
        why = 2;  // the request itself is over a zero limit
      } else if (ta < H) {  // (ta >= T_u: at most T_u requests of the user in the window)
        // the ta-th previous request of the app: the same user's iff the user has ta of
        // them before j; in the window only if among the last T_u - 1 positions
        const int r = int(sm.rank[j]) - ta;
        if (r >= int(sm.start[ap])) {
          const int x = sm.list[r];
          const int64_t gx = g0 + x;
          const uint64_t ex = sm.el[x];
          if (gx > p - H && ((e ^ ex) & a.user_mask) == 0 && in_window(e, ex, win)) why = 2;
        }
      }
    }
    if (why != bg) a.rb[(e >> pk.SI) & pk.imask] = why;
  }
}

// ---------------------------------------------------------------- app-level limit

// With the app limit counted over all users of an app, the user test runs on the user
// order and marks the requests over the user limit (of those whose own reason is used:
// gated, the first calls), one byte each at its stream position (the bytes zeroed
// first); the elements are then built again in stream order
// carrying that flag, so that the app passes leave each app's records in time order.
__global__ void __launch_bounds__(kThreads) k_bytes_zero(uint8_t *b, int64_t n) {
  const int64_t n16 = n >> 4;
  uint4 *b4 = reinterpret_cast<uint4 *>(b);
  for (int64_t i = blockIdx.x * int64_t(kThreads) + threadIdx.x; i < n16;
       i += int64_t(gridDim.x) * kThreads)
    b4[i] = make_uint4(0u, 0u, 0u, 0u);
  if (blockIdx.x == 0 && threadIdx.x < (n & 15)) b[(n16 << 4) + threadIdx.x] = 0;
}

__global__ void __launch_bounds__(kThreads) k_thr_user_flags(ScatterArgs a, uint8_t *flag) {
  const Win win = load_win(a.win);
  const Pack &pk = win.pk;
  for (int64_t p = blockIdx.x * int64_t(kThreads) + threadIdx.x; p < a.N;
       p += int64_t(gridDim.x) * kThreads) {
    if (int64_t(a.t_user) > p) continue;
    const uint64_t e = a.in[p];
    if (!(e & 1u)) continue;  // a request whose own reason is not used (a later call, gated)
    const uint64_t eq = a.in[p - a.t_user];
    if (((e ^ eq) & a.user_mask) == 0 && in_window(e, eq, win)) flag[(e >> pk.SI) & pk.imask] = 1;
  }
}

// ---------------------------------------------------------------- window counts (optional)

struct CountArgs {
  const uint64_t *el;  // key order in which every compared key is contiguous
  int64_t N;
  KeySel key;
  Win win;
  int32_t *cnt;        // [N] stream order
};

// cnt = p - (first position of the key whose arrival is still in the window) + 1,
// by binary search over the exact arrival times.
__global__ void __launch_bounds__(kThreads) k_thr_count(CountArgs a) {
  const Pack &pk = a.win.pk;
  for (int64_t p = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; p < a.N;
       p += int64_t(gridDim.x) * blockDim.x) {
    const uint64_t ep = a.el[p];
    const uint64_t k = key_of(ep, a.key);
    const int64_t gp = int64_t((ep >> pk.SI) & pk.imask);
    const int64_t lo_ts = a.win.ts[gp] - a.win.W;  // window is (ts - W, ts]
    int64_t l = 0, h = p;
    while (l < h) {
      const int64_t m = (l + h) >> 1;
      if (key_of(a.el[m], a.key) < k) l = m + 1; else h = m;
    }
    int64_t h2 = p;
    while (l < h2) {
      const int64_t m = (l + h2) >> 1;
      const int64_t gm = int64_t((a.el[m] >> pk.SI) & pk.imask);
      if (a.win.ts[gm] > lo_ts) h2 = m; else l = m + 1;
    }
    a.cnt[gp] = int32_t(p - l + 1);
  }
}

// ---------------------------------------------------------------- combine

struct CombineArgs {
  DevTrace t;
  const uint8_t *rb;   // [N] raw reasons in stream order
  const uint8_t *overloaded;
  bool raw;
  uint32_t *bitmap;
  uint8_t *reason;
  int64_t n_words;
};

constexpr int kCombineItems = 8;                        // consecutive records a thread
constexpr int kCombineWords = kCombineItems / 4;        // of reason bytes
constexpr int kCombineSpan = kThreads * kCombineItems;  // records per combine block

// Gated mode: a first call (head == itself) is throttled iff overloaded and over a limit;
// a later call is dropped iff its first call was.  Each thread takes 8 consecutive
// records: their reason bytes and overload flags in one 8-byte load each, their links
// in two 16-byte loads (when the link array is 16-byte aligned), the first calls' bytes
// gathered after all of those, the reasons out in one 8-byte store and the bitmap bits
// in one byte.
__global__ void __launch_bounds__(kThreads) k_thr_combine(CombineArgs a) {
  __shared__ int32_t s_rep[2];
  const int64_t N = a.t.N;
  const int64_t start = xcd_tile(blockIdx.x, gridDim.x) * kCombineSpan;
  const int64_t g0 = start + int64_t(threadIdx.x) * kCombineItems;
  const bool links = !a.raw && a.t.head != nullptr;
  if (links && threadIdx.x == 0 && start < N) {  // the replicas of the block's first and last
    const int64_t last = start + kCombineSpan < N ? start + kCombineSpan - 1 : N - 1;
    s_rep[0] = replica_of(a.t.rep_off, a.t.R, start);
    s_rep[1] = replica_of(a.t.rep_off, a.t.R, last);
  }
  __syncthreads();
  uint8_t *const bm = reinterpret_cast<uint8_t *>(a.bitmap);
  if (g0 >= N) {
    if (g0 < a.n_words * 32) bm[g0 >> 3] = 0;
    return;
  }
  const bool full = g0 + kCombineItems <= N;
  uint32_t cw[kCombineWords];  // reason bytes, four a word
  if (full) {
    const uint2 q = *reinterpret_cast<const uint2 *>(a.rb + g0);
    cw[0] = q.x;
    cw[1] = q.y;
  } else {
#pragma unroll
    for (int k = 0; k < kCombineWords; ++k) cw[k] = 0;
    for (int i = 0; i < kCombineItems; ++i)
      if (g0 + i < N) cw[i >> 2] |= uint32_t(a.rb[g0 + i]) << (8 * (i & 3));
  }
  if (!a.raw) {
    int32_t hd[kCombineItems];
    if (links) {
      if (full && (reinterpret_cast<uintptr_t>(a.t.head) & 15) == 0) {
#pragma unroll
        for (int k = 0; k < kCombineItems / 4; ++k) {
          const int4 q = reinterpret_cast<const int4 *>(a.t.head + g0)[k];
          hd[4 * k] = q.x;
          hd[4 * k + 1] = q.y;
          hd[4 * k + 2] = q.z;
          hd[4 * k + 3] = q.w;
        }
      } else {
#pragma unroll
        for (int i = 0; i < kCombineItems; ++i) hd[i] = g0 + i < N ? a.t.head[g0 + i] : 0;
      }
    }
    uint32_t ow[kCombineWords];  // own overload flags
#pragma unroll
    for (int k = 0; k < kCombineWords; ++k) ow[k] = 0xffffffffu;
    if (a.overloaded) {
      if (full) {
        const uint2 q = *reinterpret_cast<const uint2 *>(a.overloaded + g0);
        ow[0] = q.x;
        ow[1] = q.y;
      } else {
        for (int i = 0; i < kCombineItems; ++i)
          if (g0 + i < N && a.overloaded[g0 + i] == 0) ow[i >> 2] &= ~(0xffu << (8 * (i & 3)));
      }
    }
    // each record's first call: -1 itself, -2 a link out of range (reported by the
    // element pass), else its global index
    int64_t hg[kCombineItems];
#pragma unroll
    for (int i = 0; i < kCombineItems; ++i) hg[i] = -1;
    if (links) {
      // the thread's first replica: the last of the block's whose offset is <= g0
      int32_t r = s_rep[0];
      for (int32_t b = s_rep[1]; r < b;) {
        const int32_t m = (r + b + 1) >> 1;
        if (a.t.rep_off[m] <= g0)
          r = m;
        else
          b = m - 1;
      }
      int64_t lo = a.t.rep_off[r], hi = a.t.rep_off[r + 1];
#pragma unroll
      for (int i = 0; i < kCombineItems; ++i) {
        const int64_t g = g0 + i;
        if (g >= N) continue;
        while (g >= hi) {
          ++r;
          lo = hi;
          hi = a.t.rep_off[r + 1];
        }
        const int64_t h = lo + hd[i];
        if (h != g) hg[i] = (h >= lo && h < g) ? h : -2;
      }
    }
    uint8_t hr[kCombineItems], ho[kCombineItems];
#pragma unroll
    for (int i = 0; i < kCombineItems; ++i) {
      hr[i] = hg[i] >= 0 ? a.rb[hg[i]] : 0;
      ho[i] = (hg[i] >= 0 && a.overloaded) ? a.overloaded[hg[i]] : 1;
    }
#pragma unroll
    for (int i = 0; i < kCombineItems; ++i) {
      const int sh = 8 * (i & 3);
      uint32_t c = (cw[i >> 2] >> sh) & 0xffu;
      if (hg[i] >= 0)
        c = (ho[i] != 0 && hr[i] != 0) ? 3u : 0u;
      else if (hg[i] == -2)
        c = 0;
      else
        c = ((ow[i >> 2] >> sh) & 0xffu) != 0 ? c : 0u;
      cw[i >> 2] = (cw[i >> 2] & ~(0xffu << sh)) | (c << sh);
    }
  }
  uint32_t bits = 0;
#pragma unroll
  for (int i = 0; i < kCombineItems; ++i)
    bits |= (((cw[i >> 2] >> (8 * (i & 3))) & 0xffu) != 0 ? 1u : 0u) << i;
  bm[g0 >> 3] = uint8_t(bits);  // (bytes past N are zero, so are their bits)
  if (a.reason) {
    if (full && (reinterpret_cast<uintptr_t>(a.reason) & 7) == 0) {
      *reinterpret_cast<uint2 *>(a.reason + g0) = make_uint2(cw[0], cw[1]);
    } else {
      for (int i = 0; i < kCombineItems; ++i)
        if (g0 + i < N) a.reason[g0 + i] = uint8_t(cw[i >> 2] >> (8 * (i & 3)));
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

// The packed element holds the key (replica * U + user, then the app) and the record
// index: the key must fit 32 bits and key + index + flag 64 bits.
bool throttle_shape_ok(const fs_trace *t) {
  const Pack pk = make_pack(t, t->rep_off_h[t->n_replicas]);
  return pk.Bk <= 32 && pk.Bk + pk.Bi + 1 <= 64;
}

hipError_t launch_throttle(const fs_trace *t, const fs_limits *lim, const uint8_t *overloaded,
                           uint32_t flags, uint32_t *bitmap, uint8_t *reason, int32_t *cnt_user,
                           int32_t *cnt_app, void *ws, int32_t *err, hipStream_t s) {
  Layout L = layout(t);
  const Pack &pk = L.pk;
  if (!throttle_shape_ok(t)) return hipErrorInvalidValue;  // rejected by the callers first
  if (L.N == 0) return hipSuccess;
  char *w = static_cast<char *>(ws);
  uint64_t *A = reinterpret_cast<uint64_t *>(w + L.off_a);
  uint64_t *B = reinterpret_cast<uint64_t *>(w + L.off_b);
  uint32_t *hist = reinterpret_cast<uint32_t *>(w + L.off_hist);
  uint32_t *part = reinterpret_cast<uint32_t *>(w + L.off_part);
  int32_t *tapp = reinterpret_cast<int32_t *>(w + L.off_tapp);
  int32_t *sh = reinterpret_cast<int32_t *>(w + L.off_sh);
  uint8_t *dig_b = reinterpret_cast<uint8_t *>(w + L.off_dig);
  const bool raw = (flags & FS_THROTTLE_RAW) != 0;
  hipError_t e = hipMemcpyAsync(tapp, lim->t_app_h, sizeof(int32_t) * t->n_apps,
                                hipMemcpyHostToDevice, s);
  if (e != hipSuccess) return e;
  const DevTrace dt = dev_trace(t);
  hipLaunchKernelGGL(k_thr_span, dim3(1), dim3(kThreads), 0, s, dt.rep_off, dt.ts, dt.R, pk.Bq, sh);

  // digits: the user bits in passes of at most kRadixBits, then the app bits.  With a
  // power-of-two user count the key is replica << log2(U) | user, and since the stream
  // is replica-major and the sort stable, sorting the user bits alone already leaves
  // every (replica, user) run contiguous and in time order: the replica bits need no
  // pass.  The runs are then not in key order, which only the window counts rely on
  // (they binary-search a key's first position), so counts keep the full sort.
  struct Digit { int shift, width; };
  Digit dig[8];
  int nd = 0, n_user = 0;
  int user_bits = pk.Bu;
  if (!cnt_user && !cnt_app && t->n_replicas > 1 && t->n_users >= 2 &&
      (t->n_users & (t->n_users - 1)) == 0)
    user_bits = __builtin_ctz(uint32_t(t->n_users));
  for (int b0 = 0, left = user_bits; left > 0;) {
    const int passes = (left + kRadixBits - 1) / kRadixBits;
    const int wd = (left + passes - 1) / passes;
    dig[nd++] = {b0, wd};
    b0 += wd;
    left -= wd;
  }
  n_user = nd;
  for (int b0 = pk.Bu, left = pk.Ba; left > 0;) {
    const int passes = (left + kRadixBits - 1) / kRadixBits;
    const int wd = (left + passes - 1) / passes;
    dig[nd++] = {b0, wd};
    b0 += wd;
    left -= wd;
  }

  const bool app_level = lim->app_scope != 0;
  // the fused path: user bits only, both limits tested in one pass over the user order
  const bool fused = !app_level && !cnt_user && !cnt_app && lim->t_user >= 0 &&
                     lim->t_user <= kHaloMax;
  // flag bit of the first elements: the requests whose own reason is used (every one
  // raw, the first calls gated), for the fused test and the app-level user test
  const int mark = (fused || app_level) ? (raw ? 1 : 2) : 0;
  InitArgs ia{dt, pk, !raw, mark, sh, A, dig[0].shift, (1u << dig[0].width) - 1u, hist, L.tiles,
              err};
  hipLaunchKernelGGL(k_thr_init, dim3(L.tiles), dim3(kThreads), 0, s, ia);

  const Win win{lim->window_us, sh, 0, pk.Bq > 0, pk, dt.ts};

  const uint64_t user_mask = ((uint64_t(1) << pk.Bu) - 1) << pk.SK;
  uint64_t *in = A, *out = B;
  const int n_pass = fused ? n_user : nd;
  bool have_dig = false;  // the digits of this pass were written out by the last scatter
  for (int k = 0; k < n_pass; ++k) {
    const uint32_t mask = (1u << dig[k].width) - 1u;
    const int shift = pk.SK + dig[k].shift;
    bool hist_ready = false;
    if (k == n_user && app_level) {
      // user test on the user order, its flags to stream positions (one byte each, in
      // the digit buffer, which the app passes do not use), then the elements again in
      // stream order carrying them, with the first app digit's histogram
      if (cnt_user) {
        CountArgs ca{in, L.N, KeySel{user_mask, false, pk.SK, pk.Bu, 1u}, win, cnt_user};
        hipLaunchKernelGGL(k_thr_count, dim3(grid_for(L.N, kThreads)), dim3(kThreads), 0, s, ca);
      }
      hipLaunchKernelGGL(k_bytes_zero, dim3(grid_for((L.N >> 4) + 1, kThreads)), dim3(kThreads),
                         0, s, dig_b, L.N);
      ScatterArgs ua{in, out, L.N, 0, 0, nullptr, 0, lim->t_user,
                     user_mask, win, sh + kFlagStride};
      hipLaunchKernelGGL(k_thr_user_flags, dim3(grid_for(L.N, kThreads)), dim3(kThreads), 0, s,
                         ua, dig_b);
      InitArgs ia2{dt, pk, !raw, 0, sh, out, dig[k].shift, mask, hist, L.tiles, err, dig_b};
      hipLaunchKernelGGL(k_thr_init, dim3(L.tiles), dim3(kThreads), 0, s, ia2);
      uint64_t *tmp = in;
      in = out;
      out = tmp;
      hist_ready = true;
    }
    if (!hist_ready && k > 0 && have_dig)
      hipLaunchKernelGGL(k_radix_hist8, dim3(L.tiles), dim3(kThreads), 0, s, dig_b, L.N, mask,
                         hist, L.tiles);
    else if (!hist_ready && k > 0)
      hipLaunchKernelGGL(k_radix_hist, dim3(L.tiles), dim3(kThreads), 0, s, in, L.N, shift, mask,
                         hist, L.tiles);
    (void)exclusive_scan(hist, int64_t(mask + 1) * L.tiles, part, s);
    if (k == n_user && cnt_user && !app_level) {
      CountArgs ca{in, L.N, KeySel{user_mask, false, pk.SK, pk.Bu, 1u}, win, cnt_user};
      hipLaunchKernelGGL(k_thr_count, dim3(grid_for(L.N, kThreads)), dim3(kThreads), 0, s, ca);
    }
    // the next pass's digits go out with the elements, unless the app-level user test
    // builds the elements again in stream order before that pass
    have_dig = k + 1 < n_pass && !(app_level && k + 1 == n_user);
    ScatterArgs sa{in, out, L.N, shift, mask, hist, L.tiles, lim->t_user,
                   user_mask, win, sh + kFlagStride, have_dig ? dig_b : nullptr,
                   have_dig ? pk.SK + dig[k + 1].shift : 0,
                   have_dig ? (1u << dig[k + 1].width) - 1u : 0u};
    if (k == n_user && !app_level)
      hipLaunchKernelGGL(k_radix_scatter<true>, dim3(L.tiles), dim3(kThreads), 0, s, sa);
    else
      hipLaunchKernelGGL(k_radix_scatter<false>, dim3(L.tiles), dim3(kThreads), 0, s, sa);
    uint64_t *tmp = in;
    in = out;
    out = tmp;
  }
  // raw reasons to stream order in the free sort buffer
  uint8_t *rb = reinterpret_cast<uint8_t *>(out);
  if (fused) {
    const int64_t ns = (L.N + kSampleStride - 1) / kSampleStride;
    SampleArgs sa{in, L.N, lim->t_user, user_mask, win, sh + kFlagStride};
    hipLaunchKernelGGL(k_thr_sample, dim3(std::min<int64_t>((ns + kThreads - 1) / kThreads, 1024)),
                       dim3(kThreads), 0, s, sa);
    hipLaunchKernelGGL(k_thr_fill_fused, dim3(grid_for((L.N >> 4) + 1, kThreads)), dim3(kThreads),
                       0, s, rb, L.N, sh + kFlagStride);
    FusedArgs fa{in, L.N, lim->t_user, tapp, t->n_apps, pk.Ba, user_mask, win, rb,
                 sh + kFlagStride};
    const size_t lds = fused_lds_bytes(lim->t_user + kFTile, t->n_apps);
    if (lds > 65536)
      (void)hipFuncSetAttribute(reinterpret_cast<const void *>(k_thr_fused),
                                hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    hipLaunchKernelGGL(k_thr_fused, dim3(uint32_t((L.N + kFTile - 1) / kFTile)), dim3(kFThreads),
                       lds, s, fa);
  } else {  // app test in (user, app) order

    const KeySel app_key{((uint64_t(1) << pk.Bk) - 1) << pk.SK, app_level, pk.SK, pk.Bu,
                         uint32_t(t->n_users)};
    hipLaunchKernelGGL(k_thr_fill, dim3(grid_for((L.N >> 4) + 1, kThreads)), dim3(kThreads), 0, s,
                       rb, L.N, sh + kFlagStride);
    AppTestArgs aa{in, L.N, app_key, tapp, t->n_apps, win, rb, sh + kFlagStride};
    hipLaunchKernelGGL(k_thr_apptest, dim3(L.tiles), dim3(kThreads), 0, s, aa);
  }
  if (cnt_app) {
    const KeySel app_key{((uint64_t(1) << pk.Bk) - 1) << pk.SK, app_level, pk.SK, pk.Bu,
                         uint32_t(t->n_users)};
    CountArgs ca{in, L.N, app_key, win, cnt_app};
    hipLaunchKernelGGL(k_thr_count, dim3(grid_for(L.N, kThreads)), dim3(kThreads), 0, s, ca);
  }

  CombineArgs ca{dt, rb, overloaded, raw, bitmap, reason, (L.N + 31) / 32};
  hipLaunchKernelGGL(k_thr_combine, dim3((L.N + kCombineSpan - 1) / kCombineSpan), dim3(kThreads),
                     0, s, ca);
  return hipGetLastError();
}

}  // namespace fs

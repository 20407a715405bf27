// WSC scheduler steps: the global-memory kernel (its replica pass is in
// fs_sched_global.h, shared with the on-chip kernel), the state blob's initialisation
// and the launcher.
#include "fs_sched_global.h"

namespace fs {
namespace {

using namespace sched;

// Global-memory pass: resumes replicas that overflowed on chip and did not continue in
// the same launch (or runs all replicas when the engine asks for global memory only).
__global__ void __launch_bounds__(64) k_schedule_global(SchedArgs a) {
  extern __shared__ __align__(16) char gsm[];
  const int32_t r = blockIdx.x;
  if (*a.err) return;
  if (!state_header_ok(a)) return;
  RepState *rs = reinterpret_cast<RepState *>(a.state + a.L.reps) + r;
  if (!a.global_only && !rs->overflow) return;
  if (finish_if_done(a, r)) return;
  global_replica(a, r, gsm, a.oc.glds != 0, a.oc.hblk);
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
  const int32_t r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r < R) {
    RepState z = {};
    z.last_exit = -1;
    reinterpret_cast<RepState *>(state + L.reps)[r] = z;
  }
}

__global__ void k_state_users(char *state, StateLayout L, int64_t RU) {
  for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i <= RU;
       i += int64_t(gridDim.x) * blockDim.x) {
    if (i < RU) {
      reinterpret_cast<int64_t *>(state + L.u_all)[i] = 0;
      reinterpret_cast<int32_t *>(state + L.xslot_all)[i] = -1;
    }
    reinterpret_cast<uint32_t *>(state + L.seg_start)[i] = 0;
  }
}

__global__ void k_state_records(char *state, StateLayout L, int64_t N) {
  for (int64_t g = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; g < N;
       g += int64_t(gridDim.x) * blockDim.x) {
    reinterpret_cast<int8_t *>(state + L.fate)[g] = -1;
    reinterpret_cast<int32_t *>(state + L.succ)[g] = -1;
    reinterpret_cast<int32_t *>(state + L.emap)[g] = -1;
  }
}

// next-call links (succ[prev] = i) and the number of requests per (replica, user), the
// size of the user's segment (a FIFO holds at most all of its user's requests); links
// and ids are checked again before the scheduler runs.  Each block counts a tile of
// records by (replica, user) in LDS and adds each distinct key's count to global memory
// once, so a heavy user costs one global atomic per tile instead of one per request.
// When the replicas the tile spans times the users fit in the table, the count of
// (r, u) sits at (r - r0) * U + u (one LDS atomic per record); otherwise in a hash
// table (open addressing, at most half full).
constexpr int kLinkTile = 4096;
constexpr int kLinkPer = kLinkTile / 256;
constexpr int kLinkSlots = 2 * kLinkTile;
constexpr uint32_t kLinkEmpty = 0xffffffffu;

__global__ void __launch_bounds__(256) k_state_links(char *state, StateLayout L, DevTrace t) {
  __shared__ uint32_t hk[kLinkSlots], hc[kLinkSlots];
  uint32_t *cnt = reinterpret_cast<uint32_t *>(state + L.seg_start);
  const int64_t g0 = int64_t(blockIdx.x) * kLinkTile;
  const int64_t g_end = g0 + kLinkTile < t.N ? g0 + kLinkTile : t.N;
  // the tile's users (and calls and previous calls) are loaded before any is counted,
  // so that a thread's loads are in flight together
  int32_t us[kLinkPer], cs[kLinkPer], ps[kLinkPer];
#pragma unroll
  for (int k = 0; k < kLinkPer; ++k) {
    const int64_t g = g0 + k * 256 + threadIdx.x;
    us[k] = g < g_end ? t.user[g] : -1;
    cs[k] = g < g_end && t.call ? t.call[g] : 0;
    ps[k] = g < g_end && t.call ? t.prev[g] : -1;
  }
  const int32_t r0 = replica_of(t.rep_off, t.R, g0);
  const int32_t r1 = replica_of(t.rep_off, t.R, g_end - 1);
  const int64_t span = int64_t(r1 - r0 + 1) * t.U;
  const bool dense = span <= kLinkSlots;
  for (int j = threadIdx.x; j < kLinkSlots; j += 256) {
    if (!dense) hk[j] = kLinkEmpty;
    hc[j] = 0;
  }
  int32_t r = r0;
  int64_t r_beg = t.rep_off[r0], r_end = t.rep_off[r0 + 1];
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kLinkPer; ++k) {
    const int64_t g = g0 + k * 256 + threadIdx.x;
    if (g >= g_end) break;
    if (g >= r_end) {  // a later replica of the tile: search (r, r1]
      int32_t lo = r + 1, hi = r1;
      while (lo < hi) {
        const int32_t mid = (lo + hi + 1) >> 1;
        if (t.rep_off[mid] <= g)
          lo = mid;
        else
          hi = mid - 1;
      }
      r = lo;
      r_beg = t.rep_off[r];
      r_end = t.rep_off[r + 1];
    }
    const int32_t u = us[k];
    if (u >= 0 && u < t.U) {
      if (dense) {
        atomicAdd(hc + (int64_t(r - r0) * t.U + u), 1u);
      } else {
        // (replica, user) < R * U <= 2^31: fits below the empty marker
        const uint32_t key = uint32_t(int64_t(r) * t.U + u);
        uint32_t h = (key * 2654435761u) >> 19;  // top 13 bits: a slot in [0, 8192)
        while (true) {
          const uint32_t prev = atomicCAS(hk + h, kLinkEmpty, key);
          if (prev == kLinkEmpty || prev == key) {
            atomicAdd(hc + h, 1u);
            break;
          }
          h = (h + 1) & (kLinkSlots - 1);
        }
      }
    }
    const int32_t p = ps[k];
    if (cs[k] > 0 && p >= 0 && p < g - r_beg)
      reinterpret_cast<int32_t *>(state + L.succ)[r_beg + p] = int32_t(g - r_beg);
  }
  __syncthreads();
  if (dense) {
    uint32_t *base = cnt + int64_t(r0) * t.U;
    for (int j = threadIdx.x; j < span; j += 256)
      if (hc[j]) atomicAdd(base + j, hc[j]);
  } else {
    for (int j = threadIdx.x; j < kLinkSlots; j += 256)
      if (hk[j] != kLinkEmpty) atomicAdd(cnt + hk[j], hc[j]);
  }
}

// The same counts and links with one work-group per replica, for traces of many replicas
// of moderate size: the replica's counts are its own, kept in an LDS table of U entries
// and stored once at the end, without a global atomic.
constexpr int kLinkRepMinR = 512;              // replicas (work-groups) at least
constexpr int64_t kLinkRepMaxN = int64_t(1) << 16;  // records per replica at most
__global__ void __launch_bounds__(256) k_state_links_rep(char *state, StateLayout L, DevTrace t) {
  extern __shared__ uint32_t hc_rep[];  // [U]
  const int32_t r = blockIdx.x;
  const int64_t b = t.rep_off[r], e = t.rep_off[r + 1];
  for (int j = threadIdx.x; j < t.U; j += 256) hc_rep[j] = 0;
  __syncthreads();
  int32_t *succ = reinterpret_cast<int32_t *>(state + L.succ);
  for (int64_t g0 = b; g0 < e; g0 += int64_t(kLinkPer) * 256) {
    int32_t us[kLinkPer], cs[kLinkPer], ps[kLinkPer];
#pragma unroll
    for (int k = 0; k < kLinkPer; ++k) {
      const int64_t g = g0 + k * 256 + threadIdx.x;
      us[k] = g < e ? t.user[g] : -1;
      cs[k] = g < e && t.call ? t.call[g] : 0;
      ps[k] = g < e && t.call ? t.prev[g] : -1;
    }
#pragma unroll
    for (int k = 0; k < kLinkPer; ++k) {
      const int64_t g = g0 + k * 256 + threadIdx.x;
      if (g >= e) break;
      if (us[k] >= 0 && us[k] < t.U) atomicAdd(hc_rep + us[k], 1u);
      if (cs[k] > 0 && ps[k] >= 0 && ps[k] < g - b) succ[b + ps[k]] = int32_t(g - b);
    }
  }
  __syncthreads();
  uint32_t *cnt = reinterpret_cast<uint32_t *>(state + L.seg_start) + int64_t(r) * t.U;
  for (int j = threadIdx.x; j < t.U; j += 256) cnt[j] = hc_rep[j];
}

struct CheckArgs {
  DevTrace t;
  const int64_t *cost;
  const uint8_t *reason;
  const char *state;
  StateLayout L;
  int32_t *err;
};

constexpr int kCheckRows = 4;

__global__ void __launch_bounds__(256) k_sched_check(CheckArgs a) {
  const DevTrace &t = a.t;
  int32_t code = 0;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    const Header *h = reinterpret_cast<const Header *>(a.state + a.L.hdr);
    if (!(h->magic == kMagic && h->version == kVersion && h->R == t.R && h->U == t.U &&
          h->N == t.N))
      code = FS_E_STATE;
  }
  // a block checks kCheckRows rows of 256 records; every field of the rows is loaded
  // before the first test, then one search finds the first row's replica and short
  // walks the others (a row spans few replicas)
  const int64_t t0 = int64_t(blockIdx.x) * (kCheckRows * 256);
  int64_t ts[kCheckRows], tsp[kCheckRows], cst[kCheckRows];
  int32_t u[kCheckRows], ap[kCheckRows], li[kCheckRows], lo[kCheckRows], ls[kCheckRows];
  uint8_t rs[kCheckRows];
#pragma unroll
  for (int k = 0; k < kCheckRows; ++k) {
    const int64_t g = t0 + k * 256 + threadIdx.x;
    const bool in = g < t.N;
    ts[k] = in ? t.ts[g] : 0;
    tsp[k] = in && g > 0 ? t.ts[g - 1] : 0;
    u[k] = in ? t.user[g] : 0;
    ap[k] = in ? t.app[g] : 0;
    li[k] = in ? t.len_in[g] : 0;
    lo[k] = in ? t.len_out[g] : 0;
    ls[k] = in && t.len_sys ? t.len_sys[g] : 0;
    cst[k] = in ? a.cost[g] : 0;
    rs[k] = in && a.reason ? a.reason[g] : 0;
  }
  int32_t r = t0 < t.N ? replica_of(t.rep_off, t.R, t0) : 0;
  int64_t base = t.rep_off[r], r_end = t.rep_off[r + 1];
#pragma unroll
  for (int k = 0; k < kCheckRows; ++k) {
    const int64_t g = t0 + k * 256 + threadIdx.x;
    if (g >= t.N) break;
    while (r_end <= g) {
      ++r;
      base = r_end;
      r_end = t.rep_off[r + 1];
    }
    const int64_t i = g - base;
    if (u[k] < 0 || u[k] >= t.U || ap[k] < 0 || ap[k] >= t.A) code = max(code, int32_t(FS_E_RANGE));
    if (ts[k] < 0) code = max(code, int32_t(FS_E_RANGE));
    if (g > base && tsp[k] > ts[k]) code = max(code, int32_t(FS_E_ORDER));
    if (!len_ok(li[k]) || !len_ok(lo[k]) || !len_ok(ls[k])) code = max(code, int32_t(FS_E_RANGE));
    if (t.call) {
      const int32_t c = t.call[g], h = t.head[g], p = t.prev[g];
      bool ok;
      if (c == 0) {
        ok = h == i && p == -1;
      } else {
        ok = c > 0 && p >= 0 && p < i;
        if (ok) {
          const int64_t gp = base + p;
          ok = t.call[gp] == c - 1 && t.user[gp] == u[k] && t.head[gp] == h;
        }
      }
      if (!ok) code = max(code, int32_t(FS_E_RANGE));
    }
    if (cst[k] < 0 || cst[k] >= kValueLimit) code = max(code, int32_t(FS_E_RANGE));
    if (rs[k] > 2) code = max(code, int32_t(FS_E_RANGE));
  }
  if (code) raise_err(a.err, code);
}

int grid_for(int64_t n, int threads) {
  int64_t b = (n + threads - 1) / threads;
  if (b < 1) b = 1;
  if (b > 65536) b = 65536;
  return int(b);
}

}  // namespace

size_t state_bytes(const fs_trace *t) {
  return state_layout(t->n_replicas, t->n_users, t->rep_off_h[t->n_replicas]).total;
}

hipError_t launch_state_init(void *state, const fs_trace *t, hipStream_t s) {
  const int64_t N = t->rep_off_h[t->n_replicas];
  const StateLayout L = state_layout(t->n_replicas, t->n_users, N);
  char *st = static_cast<char *>(state);
  hipLaunchKernelGGL(k_state_header, dim3(1), dim3(64), 0, s, st, L, t->n_replicas, t->n_users, N);
  hipLaunchKernelGGL(k_state_reps, dim3((t->n_replicas + 255) / 256), dim3(256), 0, s, st, L,
                     t->n_replicas);
  const int64_t RU = int64_t(t->n_replicas) * t->n_users;
  hipLaunchKernelGGL(k_state_users, dim3(grid_for(RU + 1, 256)), dim3(256), 0, s, st, L, RU);
  if (N > 0) {
    hipLaunchKernelGGL(k_state_records, dim3(grid_for(N, 256)), dim3(256), 0, s, st, L, N);
    int64_t max_rep = 0;
    for (int32_t r = 0; r < t->n_replicas; ++r)
      max_rep = std::max<int64_t>(max_rep, t->rep_off_h[r + 1] - t->rep_off_h[r]);
    if (t->n_replicas >= kLinkRepMinR && t->n_users <= kLinkSlots && max_rep <= kLinkRepMaxN)
      hipLaunchKernelGGL(k_state_links_rep, dim3(t->n_replicas), dim3(256),
                         size_t(t->n_users) * sizeof(uint32_t), s, st, L, dev_trace(t));
    else
      hipLaunchKernelGGL(k_state_links, dim3((N + kLinkTile - 1) / kLinkTile), dim3(256), 0, s,
                         st, L, dev_trace(t));
  }
  // per-user first-call segments: exclusive prefix of the counts
  hipError_t e = exclusive_scan(reinterpret_cast<uint32_t *>(st + L.seg_start), RU + 1,
                                reinterpret_cast<uint32_t *>(st + L.seg_part), s);
  if (e != hipSuccess) return e;
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
  a.fcfs = (eng->flags & FS_ENGINE_FCFS) != 0;
  a.blind = (eng->flags & FS_ENGINE_BLIND) != 0;
  a.literal = (eng->flags & FS_ENGINE_LITERAL) != 0;
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
  a.oc = onchip_config(t->n_replicas, t->n_users, a.literal);
  // The global-memory kernel keeps its user table in LDS when it fits in 64 KB and
  // every replica's work-group can still be resident at once (up to four per CU on
  // the 256 CUs): a table that left some replicas waiting for a CU made the
  // 1,024-replica literal runs slower than no table.
  const size_t glds = size_t(t->n_users) * kXLdsBytesPerUser;
  const int32_t R = t->n_replicas;
  const size_t per_cu = R <= 256 ? 1 : R <= 512 ? 2 : R <= 768 ? 3 : 4;
  a.oc.glds = (glds <= 65536 && glds <= size_t(160 * 1024) / per_cu - 1024) ? 1 : 0;
  // the block minima of the two-level argmin after the table, while all fits in 64 KB
  const size_t tab = a.oc.glds ? (glds + 15) / 16 * 16 : 0;
  const int32_t nblk = (t->n_users + 63) / 64 + 1;
  const size_t hb = size_t(nblk) * kXBlockBytes;
  // an on-chip instance that continues with the global-memory pass has its own LDS
  // allocation: the table and the block minima there only if they fit in it
  {
    const size_t tab_i = (glds + 15) / 16 * 16;
    a.oc.inl_glds = tab_i <= a.oc.lds_bytes ? 1 : 0;
    a.oc.inl_hblk = (a.oc.inl_glds ? tab_i : 0) + hb <= a.oc.lds_bytes ? nblk : 0;
  }
  a.oc.hblk = tab + hb <= 65536 ? nblk : 0;
  const size_t gl_lds = tab + (a.oc.hblk ? hb : 0);

  CheckArgs ca{a.t, cost, reason, a.state, a.L, a.err};
  hipLaunchKernelGGL(k_sched_check, dim3(N > 0 ? (N + kCheckRows * 256 - 1) / (kCheckRows * 256) : 1),
                     dim3(256), 0, s, ca);
  const dim3 grid(t->n_replicas), block(64);
  if (!a.global_only) launch_onchip(a, s);
  hipLaunchKernelGGL(k_schedule_global, grid, block, gl_lds, s, a);
  return hipGetLastError();
}

}  // namespace fs

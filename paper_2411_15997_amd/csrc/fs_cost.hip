// Weighted service cost of one LLM call (Eq. 2, one term of the sum; Alg. 1 charge):
//   cost = floor(E_u * (c_in*L_I + c_sys*L_S + c_out*L_O) / 2^8)
// with Q16 coefficients c (class weight over w_aj, Eq. 1) and Q8 priority E_u.
// A pure HBM stream: each record reads app, lengths (and call, and the user when
// priorities are given: Eq. 2 reads the user only through E_i) and writes one int64.
// Four records per thread with 16-byte loads and stores.
#include "fs_device.h"
#include "fs_launch.h"

namespace fs {

struct CostArgs {
  DevTrace t;
  int32_t J;
  int64_t coef_stride, prio_stride;
  const int64_t *coef;
  const int32_t *prio;
  int64_t *cost;
  int32_t *err;
};

__device__ inline int64_t cost_one(const CostArgs &a, int64_t g, int32_t rep, int32_t app,
                                   int32_t user, int32_t call, int32_t li, int32_t ls, int32_t lo,
                                   int32_t &code) {
  if (app < 0 || app >= a.t.A || (a.prio && (user < 0 || user >= a.t.U)) || call < 0) {
    code = code > FS_E_RANGE ? code : FS_E_RANGE;
    return 0;
  }
  if (!len_ok(li) || !len_ok(ls) || !len_ok(lo)) {
    code = code > FS_E_RANGE ? code : FS_E_RANGE;
    return 0;
  }
  int32_t j = call < a.J - 1 ? call : a.J - 1;
  const int64_t *c = a.coef + rep * a.coef_stride + (int64_t(app) * a.J + j) * 3;
  int64_t c0 = __ldg(c), c1 = __ldg(c + 1), c2 = __ldg(c + 2);
  int64_t E = a.prio ? int64_t(__ldg(a.prio + rep * a.prio_stride + user)) : 256;
  if (c0 < 0 || c0 >= kCoefLimit || c1 < 0 || c1 >= kCoefLimit || c2 < 0 || c2 >= kCoefLimit ||
      E < 0 || E >= kPrioLimit) {
    code = code > FS_E_RANGE ? code : FS_E_RANGE;
    return 0;
  }
  // Each product is below 2^60, their sum below 2^62: exact in 64 bits.
  uint64_t weighted = uint64_t(li) * uint64_t(c0) + uint64_t(ls) * uint64_t(c1) +
                      uint64_t(lo) * uint64_t(c2);
  uint64_t lo64 = weighted * uint64_t(E);
  uint64_t hi64 = __umul64hi(weighted, uint64_t(E));
  // (hi:lo) >> 8 must stay below 2^62
  if (hi64 >> 6) {
    code = code > FS_E_OVERFLOW ? code : FS_E_OVERFLOW;
    return 0;
  }
  uint64_t v = (hi64 << 56) | (lo64 >> 8);
  if (v >= uint64_t(kValueLimit)) {
    code = code > FS_E_OVERFLOW ? code : FS_E_OVERFLOW;
    return 0;
  }
  return int64_t(v);
}

template <bool PER_REP, bool PRIO>
__global__ void __launch_bounds__(256) k_cost_vec4(CostArgs a, int64_t n_vec) {
  int32_t code = 0;
  for (int64_t v = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; v < n_vec;
       v += int64_t(gridDim.x) * blockDim.x) {
    int64_t g0 = v * 4;
    int4 app = __ldg(reinterpret_cast<const int4 *>(a.t.app) + v);
    int4 li = __ldg(reinterpret_cast<const int4 *>(a.t.len_in) + v);
    int4 lo = __ldg(reinterpret_cast<const int4 *>(a.t.len_out) + v);
    int4 ls = a.t.len_sys ? __ldg(reinterpret_cast<const int4 *>(a.t.len_sys) + v)
                          : make_int4(0, 0, 0, 0);
    int4 call = a.t.call ? __ldg(reinterpret_cast<const int4 *>(a.t.call) + v)
                         : make_int4(0, 0, 0, 0);
    int4 user = PRIO ? __ldg(reinterpret_cast<const int4 *>(a.t.user) + v) : make_int4(0, 0, 0, 0);
    int32_t r0 = 0, r1 = 0, r2 = 0, r3 = 0;
    if (PER_REP) {
      r0 = replica_of(a.t.rep_off, a.t.R, g0);
      r1 = r0;
      while (__ldg(a.t.rep_off + r1 + 1) <= g0 + 1) ++r1;
      r2 = r1;
      while (__ldg(a.t.rep_off + r2 + 1) <= g0 + 2) ++r2;
      r3 = r2;
      while (__ldg(a.t.rep_off + r3 + 1) <= g0 + 3) ++r3;
    }
    longlong2 out01, out23;
    out01.x = cost_one(a, g0, r0, app.x, user.x, call.x, li.x, ls.x, lo.x, code);
    out01.y = cost_one(a, g0 + 1, r1, app.y, user.y, call.y, li.y, ls.y, lo.y, code);
    out23.x = cost_one(a, g0 + 2, r2, app.z, user.z, call.z, li.z, ls.z, lo.z, code);
    out23.y = cost_one(a, g0 + 3, r3, app.w, user.w, call.w, li.w, ls.w, lo.w, code);
    reinterpret_cast<longlong2 *>(a.cost)[2 * v] = out01;
    reinterpret_cast<longlong2 *>(a.cost)[2 * v + 1] = out23;
  }
  if (code) raise_err(a.err, code);
}

template <bool PER_REP>
__global__ void __launch_bounds__(256) k_cost_scalar(CostArgs a, int64_t g_begin, int64_t g_end) {
  int32_t code = 0;
  for (int64_t g = g_begin + blockIdx.x * int64_t(blockDim.x) + threadIdx.x; g < g_end;
       g += int64_t(gridDim.x) * blockDim.x) {
    int32_t r = PER_REP ? replica_of(a.t.rep_off, a.t.R, g) : 0;
    int32_t ls = a.t.len_sys ? a.t.len_sys[g] : 0;
    int32_t call = a.t.call ? a.t.call[g] : 0;
    a.cost[g] = cost_one(a, g, r, a.t.app[g], a.prio ? a.t.user[g] : 0, call, a.t.len_in[g],
                         ls, a.t.len_out[g], code);
  }
  if (code) raise_err(a.err, code);
}

static bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

hipError_t launch_cost(const fs_trace *t, const fs_weights *w, int64_t *cost, int32_t *err,
                       hipStream_t stream) {
  CostArgs a;
  a.t = dev_trace(t);
  a.J = w->n_stages;
  a.coef_stride = w->coef_rep_stride;
  a.prio_stride = w->prio ? w->prio_rep_stride : 0;
  a.coef = w->coef;
  a.prio = w->prio;
  a.cost = cost;
  a.err = err;
  const int64_t N = a.t.N;
  if (N == 0) return hipSuccess;
  bool per_rep = (a.coef_stride != 0 || a.prio_stride != 0) && a.t.R > 1;
  bool vec = aligned16(t->app) && aligned16(t->len_in) && aligned16(t->len_out) &&
             (!a.prio || aligned16(t->user)) && aligned16(cost) &&
             (!t->len_sys || aligned16(t->len_sys)) && (!t->call || aligned16(t->call));
  int64_t n_vec = vec ? N / 4 : 0;
  const int threads = 256;
  if (n_vec > 0) {
    int64_t blocks = (n_vec + threads - 1) / threads;
    if (blocks > 65536) blocks = 65536;
    const bool pr = a.prio != nullptr;
    if (per_rep && pr)
      hipLaunchKernelGGL((k_cost_vec4<true, true>), dim3(blocks), dim3(threads), 0, stream, a, n_vec);
    else if (per_rep)
      hipLaunchKernelGGL((k_cost_vec4<true, false>), dim3(blocks), dim3(threads), 0, stream, a, n_vec);
    else if (pr)
      hipLaunchKernelGGL((k_cost_vec4<false, true>), dim3(blocks), dim3(threads), 0, stream, a, n_vec);
    else
      hipLaunchKernelGGL((k_cost_vec4<false, false>), dim3(blocks), dim3(threads), 0, stream, a, n_vec);
  }
  int64_t tail = N - n_vec * 4;
  if (tail > 0) {
    int64_t blocks = (tail + threads - 1) / threads;
    if (blocks > 65536) blocks = 65536;
    if (per_rep)
      hipLaunchKernelGGL(k_cost_scalar<true>, dim3(blocks), dim3(threads), 0, stream, a,
                         n_vec * 4, N);
    else
      hipLaunchKernelGGL(k_cost_scalar<false>, dim3(blocks), dim3(threads), 0, stream, a,
                         n_vec * 4, N);
  }
  return hipGetLastError();
}

}  // namespace fs

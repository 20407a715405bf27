"""Python binding of libfairserve.so (the FairServe policy hot path on MI355X).

Argument marshalling only: every step of the path runs in the HIP kernels of
``libfairserve.so``; torch supplies device memory and the current stream.
The functions carry the C entry points' names (include/fairserve.h).  There
is no CPU fallback: loading fails loudly when the library is missing.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libfairserve.so")

FS_OK, FS_E_ARG, FS_E_ORDER, FS_E_RANGE, FS_E_OVERFLOW, FS_E_WORKSPACE, FS_E_STATE, FS_E_HIP = range(8)
FS_THROTTLE_RAW = 1
FS_ENGINE_GLOBAL_ONLY, FS_ENGINE_FCFS, FS_ENGINE_BLIND, FS_ENGINE_LITERAL = 1, 2, 4, 8
ALIGN = 256


class FairServeError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = int(code)
        msg = _lib().fs_status_string(self.code).decode() if _LIB is not None else str(code)
        super().__init__(f"{where}: {msg} (code {code})")


# ----------------------------------------------------------------- C structs

class fs_trace(C.Structure):
    _fields_ = [("n_replicas", C.c_int32), ("n_users", C.c_int32), ("n_apps", C.c_int32),
                ("rep_off_h", C.c_void_p), ("rep_off", C.c_void_p), ("ts_us", C.c_void_p),
                ("user", C.c_void_p), ("app", C.c_void_p), ("call", C.c_void_p),
                ("head", C.c_void_p), ("prev", C.c_void_p), ("len_in", C.c_void_p),
                ("len_sys", C.c_void_p), ("len_out", C.c_void_p)]


class fs_weights(C.Structure):
    _fields_ = [("n_stages", C.c_int32), ("coef_rep_stride", C.c_int64), ("coef", C.c_void_p),
                ("prio_rep_stride", C.c_int64), ("prio", C.c_void_p)]


class fs_limits(C.Structure):
    _fields_ = [("window_us", C.c_int64), ("t_user", C.c_int32), ("t_app_h", C.c_void_p),
                ("app_scope", C.c_int32)]


class fs_engine(C.Structure):
    _fields_ = [("step_us", C.c_int64), ("cap_tokens", C.c_int64),
                ("overload_tokens", C.c_int64), ("flags", C.c_uint32)]


class fs_outputs(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("status", "admit_step", "admit_seq", "counter_after",
                                           "counter_on_arrival", "counter", "steps", "decisions",
                                           "max_gap", "err")]


class fs_metrics(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("jain", "max_gap_tokens", "svc_req_pct", "svc_int_pct",
                                           "served_users_pct", "delayed_users_pct", "throttled",
                                           "aborted_midway", "wasted_tokens")]


class fs_wstats(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("minutes", "user_req", "user_tok", "user_app_req",
                                           "user_app_tok", "rate_hist", "len_hist", "len_sum",
                                           "size_hist", "graph")]


RATE_BINS, LEN_BINS, SIZE_BINS, GRAPH_BINS = 128, 32, 64, 7

_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"libfairserve.so not built ({LIB_PATH}); run __graft_entry__.build()")
        L = C.CDLL(LIB_PATH)
        P, I32, I64, U32, SZ, S = C.c_void_p, C.c_int32, C.c_int64, C.c_uint32, C.c_size_t, C.c_void_p
        T = C.POINTER(fs_trace)
        sig = {
            "fs_cost": ([T, C.POINTER(fs_weights), P, P, S], I32),
            "fs_history_workspace": ([T, I32], SZ),
            "fs_weights_from_history": ([T, I32, I64, I32, P, P, P, P, SZ, P, S], I32),
            "fs_throttle_workspace": ([T], SZ),
            "fs_throttle": ([T, C.POINTER(fs_limits), P, U32, P, P, P, P, P, SZ, P, S], I32),
            "fs_state_bytes": ([T], SZ),
            "fs_state_init": ([P, SZ, T, S], I32),
            "fs_schedule_step": ([P, T, P, P, C.POINTER(fs_engine), C.POINTER(fs_outputs), I64, S], I32),
            "fs_run_trace_workspace": ([T], SZ),
            "fs_run_trace": ([T, C.POINTER(fs_weights), C.POINTER(fs_limits), C.POINTER(fs_engine),
                              C.POINTER(fs_outputs), P, SZ, S], I32),
            "fs_metrics_workspace": ([T], SZ),
            "fs_workload_workspace": ([T], SZ),
            "fs_workload_stats": ([T, I64, C.POINTER(fs_wstats), P, SZ, P, S], I32),
            "fs_metrics_noalloc_limit": ([], SZ),
            "fs_fairness_metrics_noalloc": ([T, P, C.POINTER(fs_outputs), C.POINTER(fs_engine),
                                             I32, C.POINTER(fs_metrics), S], I32),
            "fs_fairness_metrics": ([T, P, C.POINTER(fs_outputs), C.POINTER(fs_engine), I32,
                                     C.POINTER(fs_metrics), P, SZ, S], I32),
            "fs_coef_from_expectations": ([I32, I32, P, P, P, I64, P], I32),
            "fs_sync_status": ([S, P], I32),
            "fs_status_string": ([I32], C.c_char_p),
        }
        for name, (args, res) in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _LIB = L
    return _LIB


EXPORTED = ("fs_cost", "fs_history_workspace", "fs_weights_from_history", "fs_throttle_workspace", "fs_throttle", "fs_state_bytes", "fs_state_init",
            "fs_schedule_step", "fs_run_trace_workspace", "fs_run_trace", "fs_metrics_workspace",
            "fs_fairness_metrics", "fs_metrics_noalloc_limit", "fs_fairness_metrics_noalloc",
            "fs_workload_workspace", "fs_workload_stats",
            "fs_coef_from_expectations", "fs_sync_status", "fs_status_string")


def _check(code: int, where: str):
    if code != FS_OK:
        raise FairServeError(code, where)


def _torch():
    import torch
    return torch


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream():
    return C.c_void_p(_torch().cuda.current_stream().cuda_stream)


def _empty(shape, dtype, device):
    """Device buffer whose data pointer is 256-byte aligned (torch's allocator is)."""
    torch = _torch()
    t = torch.empty(shape, dtype=dtype, device=device)
    assert t.data_ptr() % ALIGN == 0
    return t


# ----------------------------------------------------------------- device trace

class DeviceTrace:
    """A trace resident in HBM plus its fs_trace descriptor."""

    def __init__(self, tr, device="cuda"):
        torch = _torch()
        self.n_replicas, self.n_users, self.n_apps = tr.n_replicas, tr.n_users, tr.n_apps
        self.n = int(tr.ts_us.shape[0])
        self.rep_off_h = np.ascontiguousarray(tr.rep_off, np.int64)
        def dev(a, dt):
            if a is None:
                return None
            a = np.ascontiguousarray(a, dt)
            if a.shape[0] == 0:          # keep a valid (non-null) pointer for empty traces
                a = np.zeros(1, dt)
            return torch.from_numpy(a).to(device)
        self.rep_off = dev(tr.rep_off, np.int64)
        self.ts_us = dev(tr.ts_us, np.int64)
        self.user = dev(tr.user, np.int32)
        self.app = dev(tr.app, np.int32)
        self.call = dev(tr.call, np.int32)
        self.head = dev(tr.head, np.int32)
        self.prev = dev(tr.prev, np.int32)
        self.len_in = dev(tr.len_in, np.int32)
        self.len_sys = dev(tr.len_sys, np.int32)
        self.len_out = dev(tr.len_out, np.int32)
        self.device = device
        self.s = fs_trace(self.n_replicas, self.n_users, self.n_apps, self.rep_off_h.ctypes.data,
                          *(_ptr(getattr(self, k)) for k in (
                              "rep_off", "ts_us", "user", "app", "call", "head", "prev",
                              "len_in", "len_sys", "len_out")))

    @property
    def ref(self):
        return C.byref(self.s)


def err_word(device="cuda"):
    return _empty((1,), _torch().int32, device)


def fs_sync_status(err) -> int:
    return int(_lib().fs_sync_status(_stream(), _ptr(err)))


def sync_check(err, where):
    _check(fs_sync_status(err), where)


# ----------------------------------------------------------------- entry points

def make_weights(dt: DeviceTrace, coef, prio=None, per_replica=False, prio_per_replica=False):
    """coef: [R|1][A][J][3] int64 (numpy or torch); returns (fs_weights, keep-alive tensors)."""
    torch = _torch()
    coef_t = torch.as_tensor(np.ascontiguousarray(coef, np.int64)).to(dt.device)
    J = int(coef_t.shape[-2])
    prio_t = None if prio is None else torch.as_tensor(np.ascontiguousarray(prio, np.int32)).to(dt.device)
    w = fs_weights(J, dt.n_apps * J * 3 if per_replica else 0, _ptr(coef_t),
                   dt.n_users if (prio is not None and prio_per_replica) else 0, _ptr(prio_t))
    return w, (coef_t, prio_t)


def fs_cost(dt: DeviceTrace, weights, cost=None, err=None, check=True):
    torch = _torch()
    cost = _empty((max(dt.n, 1),), torch.int64, dt.device) if cost is None else cost
    err = err_word(dt.device) if err is None else err
    _check(_lib().fs_cost(dt.ref, C.byref(weights), _ptr(cost), _ptr(err), _stream()), "fs_cost")
    if check:
        sync_check(err, "fs_cost")
    return cost


def fs_weights_from_history(dt: DeviceTrace, n_stages, K=1024, base_limit=30, coef=True,
                            limits=True, err=None, check=True):
    """Eq. 1 coefficients [A][J][3] and app limits [A] from a historical trace on the
    device; returns (stats [A][J][5], coef or None, t_app or None) as device tensors."""
    torch = _torch()
    A, J = dt.n_apps, int(n_stages)
    stats = _empty((A, J, 5), torch.int64, dt.device)
    coef_t = _empty((A, J, 3), torch.int64, dt.device) if coef else None
    t_app = _empty((A,), torch.int32, dt.device) if limits else None
    err = err_word(dt.device) if err is None else err
    wsb = int(_lib().fs_history_workspace(dt.ref, J))
    ws = _empty((wsb,), torch.uint8, dt.device) if wsb > 0 else None
    _check(_lib().fs_weights_from_history(dt.ref, J, int(K), int(base_limit), _ptr(stats),
                                          _ptr(coef_t), _ptr(t_app), _ptr(ws), wsb, _ptr(err),
                                          _stream()),
           "fs_weights_from_history")
    if check:
        sync_check(err, "fs_weights_from_history")
    return stats, coef_t, t_app


def make_limits(window_us, t_user, t_app, app_scope=0):
    t_app = np.ascontiguousarray(t_app, np.int32)
    return fs_limits(int(window_us), int(t_user), t_app.ctypes.data, int(app_scope)), t_app


def fs_throttle_workspace(dt: DeviceTrace) -> int:
    return int(_lib().fs_throttle_workspace(dt.ref))


@dataclass
class ThrottleOut:
    bitmap: object
    reason: object
    cnt_user: object
    cnt_app: object


def fs_throttle(dt: DeviceTrace, limits, overloaded=None, raw=True, want_reason=True,
                want_counts=False, ws=None, err=None, check=True, bitmap=None, reason=None):
    torch = _torch()
    lim, keep = limits
    n = dt.n
    if bitmap is None:
        bitmap = _empty(((n + 31) // 32 + 1,), torch.int32, dt.device)
    if reason is None and want_reason:
        reason = _empty((max(n, 1),), torch.uint8, dt.device)
    cu = _empty((max(n, 1),), torch.int32, dt.device) if want_counts else None
    ca = _empty((max(n, 1),), torch.int32, dt.device) if want_counts else None
    nb = fs_throttle_workspace(dt)
    ws = _empty((max(nb, 1),), torch.uint8, dt.device) if ws is None else ws
    err = err_word(dt.device) if err is None else err
    ov = None
    if overloaded is not None:
        ov = torch.as_tensor(np.ascontiguousarray(overloaded, np.uint8)).to(dt.device)
    _check(_lib().fs_throttle(dt.ref, C.byref(lim), _ptr(ov), FS_THROTTLE_RAW if raw else 0,
                              _ptr(bitmap), _ptr(reason), _ptr(cu), _ptr(ca), _ptr(ws),
                              ws.numel(), _ptr(err), _stream()), "fs_throttle")
    if check:
        sync_check(err, "fs_throttle")
    return ThrottleOut(bitmap, reason, cu, ca)


def make_engine(step_us, cap_tokens, overload_tokens, global_only=False, fcfs=False, blind=False,
                literal=False):
    """literal: the literal engine, with cap_tokens the KV-cache capacity in tokens."""
    flags = ((FS_ENGINE_GLOBAL_ONLY if global_only else 0) | (FS_ENGINE_FCFS if fcfs else 0)
             | (FS_ENGINE_BLIND if blind else 0) | (FS_ENGINE_LITERAL if literal else 0))
    return fs_engine(int(step_us), int(cap_tokens), int(overload_tokens), flags)


class Outputs:
    """Device output buffers of the scheduler and their fs_outputs descriptor."""

    def __init__(self, dt: DeviceTrace, parity=True):
        torch = _torch()
        n, R, U = max(dt.n, 1), dt.n_replicas, dt.n_users
        d = dt.device
        self.status = _empty((n,), torch.int8, d)
        self.admit_step = _empty((n,), torch.int32, d)
        self.admit_seq = _empty((n,), torch.int32, d) if parity else None
        self.counter_after = _empty((n,), torch.int64, d) if parity else None
        self.counter_on_arrival = _empty((n,), torch.int64, d) if parity else None
        self.counter = _empty((R * U,), torch.int64, d)
        self.steps = _empty((R,), torch.int64, d)
        self.decisions = _empty((R,), torch.int64, d)
        self.max_gap = _empty((R,), torch.int64, d)
        self.err = err_word(d)
        self.s = fs_outputs(*(_ptr(getattr(self, k)) for k in (
            "status", "admit_step", "admit_seq", "counter_after", "counter_on_arrival", "counter",
            "steps", "decisions", "max_gap", "err")))

    @property
    def ref(self):
        return C.byref(self.s)

    def host(self):
        out = {}
        for k in ("status", "admit_step", "admit_seq", "counter_after", "counter_on_arrival",
                  "counter", "steps", "decisions", "max_gap"):
            v = getattr(self, k)
            out[k] = None if v is None else v.cpu().numpy()
        return out


def fs_state_bytes(dt: DeviceTrace) -> int:
    return int(_lib().fs_state_bytes(dt.ref))


def fs_state_init(dt: DeviceTrace, state=None):
    torch = _torch()
    nb = fs_state_bytes(dt)
    state = _empty((nb,), torch.uint8, dt.device) if state is None else state
    _check(_lib().fs_state_init(_ptr(state), state.numel(), dt.ref, _stream()), "fs_state_init")
    return state


def fs_schedule_step(dt: DeviceTrace, state, cost, exceed_reason, engine, out: Outputs,
                     n_steps=-1, check=True):
    _check(_lib().fs_schedule_step(_ptr(state), dt.ref, _ptr(cost), _ptr(exceed_reason),
                                   C.byref(engine), out.ref, int(n_steps), _stream()),
           "fs_schedule_step")
    if check:
        sync_check(out.err, "fs_schedule_step")
    return out


def fs_run_trace_workspace(dt: DeviceTrace) -> int:
    return int(_lib().fs_run_trace_workspace(dt.ref))


def run_trace_buffers(dt: DeviceTrace):
    """Workspace for fs_run_trace and views of the cost and raw reasons it leaves there."""
    torch = _torch()
    nb = fs_run_trace_workspace(dt)
    ws = _empty((nb,), torch.uint8, dt.device)
    cost = ws[:dt.n * 8].view(torch.int64)
    off = (dt.n * 8 + ALIGN - 1) // ALIGN * ALIGN
    reason = ws[off:off + dt.n]
    return ws, cost, reason


def fs_run_trace(dt: DeviceTrace, weights, limits, engine, out: Outputs, ws, check=True):
    lim, keep = limits
    _check(_lib().fs_run_trace(dt.ref, C.byref(weights), C.byref(lim), C.byref(engine), out.ref,
                               _ptr(ws), ws.numel(), _stream()), "fs_run_trace")
    if check:
        sync_check(out.err, "fs_run_trace")
    return out


class Metrics:
    def __init__(self, dt: DeviceTrace):
        torch = _torch()
        R, d = dt.n_replicas, dt.device
        for k in ("jain", "max_gap_tokens", "svc_req_pct", "svc_int_pct", "served_users_pct",
                  "delayed_users_pct"):
            setattr(self, k, _empty((R,), torch.float64, d))
        for k in ("throttled", "aborted_midway", "wasted_tokens"):
            setattr(self, k, _empty((R,), torch.int64, d))
        self.s = fs_metrics(*(_ptr(getattr(self, k)) for k in (
            "jain", "max_gap_tokens", "svc_req_pct", "svc_int_pct", "served_users_pct",
            "delayed_users_pct", "throttled", "aborted_midway", "wasted_tokens")))

    def host(self):
        return {k: getattr(self, k).cpu().numpy() for k in (
            "jain", "max_gap_tokens", "svc_req_pct", "svc_int_pct", "served_users_pct",
            "delayed_users_pct", "throttled", "aborted_midway", "wasted_tokens")}


def fs_metrics_workspace(dt: DeviceTrace) -> int:
    return int(_lib().fs_metrics_workspace(dt.ref))


def fs_fairness_metrics(dt: DeviceTrace, cost, out: Outputs, engine, delay_steps=0, m=None,
                        ws=None, check=True):
    torch = _torch()
    m = Metrics(dt) if m is None else m
    nb = fs_metrics_workspace(dt)
    ws = _empty((max(nb, 1),), torch.uint8, dt.device) if ws is None else ws
    _check(_lib().fs_fairness_metrics(dt.ref, _ptr(cost), out.ref, C.byref(engine),
                                      int(delay_steps), C.byref(m.s), _ptr(ws), ws.numel(),
                                      _stream()), "fs_fairness_metrics")
    if check:
        sync_check(out.err, "fs_fairness_metrics")
    return m


class WorkloadStats:
    """Device outputs of fs_workload_stats and their fs_wstats descriptor."""

    FIELDS = ("minutes", "user_req", "user_tok", "user_app_req", "user_app_tok", "rate_hist",
              "len_hist", "len_sum", "size_hist", "graph")

    def __init__(self, dt: DeviceTrace, per_app=True):
        torch = _torch()
        R, U, A, d = dt.n_replicas, dt.n_users, dt.n_apps, dt.device
        e = lambda *shape: _empty(shape, torch.int64, d)
        self.minutes = e(R)
        self.user_req, self.user_tok = e(R, U), e(R, U)
        self.user_app_req = e(R, U, A) if per_app else None
        self.user_app_tok = e(R, U, A) if per_app else None
        self.rate_hist = e(R, A + 1, 2, RATE_BINS)
        self.len_hist = e(R, A, 3, LEN_BINS)
        self.len_sum = e(R, A, 3)
        self.size_hist = e(R, A, SIZE_BINS)
        self.graph = e(R, GRAPH_BINS, 5)
        self.s = fs_wstats(*(_ptr(getattr(self, k)) for k in self.FIELDS))

    def host(self):
        return {k: (None if getattr(self, k) is None else getattr(self, k).cpu().numpy())
                for k in self.FIELDS}


def fs_workload_workspace(dt: DeviceTrace) -> int:
    return int(_lib().fs_workload_workspace(dt.ref))


def fs_workload_stats(dt: DeviceTrace, minute_us=60_000_000, out=None, ws=None, err=None,
                      per_app=True, check=True):
    torch = _torch()
    out = WorkloadStats(dt, per_app) if out is None else out
    nb = fs_workload_workspace(dt)
    ws = _empty((max(nb, 1),), torch.uint8, dt.device) if ws is None else ws
    err = err_word(dt.device) if err is None else err
    _check(_lib().fs_workload_stats(dt.ref, int(minute_us), C.byref(out.s), _ptr(ws), ws.numel(),
                                    _ptr(err), _stream()), "fs_workload_stats")
    if check:
        sync_check(err, "fs_workload_stats")
    return out


def fs_metrics_noalloc_limit() -> int:
    return int(_lib().fs_metrics_noalloc_limit())


def fs_fairness_metrics_noalloc(dt: DeviceTrace, cost, out: Outputs, engine, delay_steps=0,
                                m=None, check=True):
    """fs_fairness_metrics with the library's own fixed workspace (allocates nothing but
    the Metrics outputs when `m` is not given)."""
    m = Metrics(dt) if m is None else m
    _check(_lib().fs_fairness_metrics_noalloc(dt.ref, _ptr(cost), out.ref, C.byref(engine),
                                              int(delay_steps), C.byref(m.s), _stream()),
           "fs_fairness_metrics_noalloc")
    if check:
        sync_check(out.err, "fs_fairness_metrics_noalloc")
    return m


def fs_coef_from_expectations(e_in, e_sys, e_out, K=1024):
    """Eq. 1 host helper (synchronous, host arrays): returns coef [A][J][3] int64."""
    e_in = np.ascontiguousarray(e_in, np.float64)
    A, J = e_in.shape
    e_sys = np.ascontiguousarray(e_sys, np.float64)
    e_out = np.ascontiguousarray(e_out, np.float64)
    coef = np.zeros((A, J, 3), np.int64)
    _check(_lib().fs_coef_from_expectations(A, J, e_in.ctypes.data, e_sys.ctypes.data,
                                            e_out.ctypes.data, int(K), coef.ctypes.data),
           "fs_coef_from_expectations")
    return coef


def workload_weights(wl, tr):
    """Product-side Q16 coefficient table for a workload description `wl` (any object
    with direct_coef_table(trace), expectations() and weight_K): [R|1][A][J][3] and
    whether it is per replica."""
    direct = wl.direct_coef_table(tr)
    if direct is not None:
        return direct, direct.shape[0] > 1
    e_in, e_sys, e_out = wl.expectations()
    return fs_coef_from_expectations(e_in, e_sys, e_out, wl.weight_K)[None], False

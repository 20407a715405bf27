"""ctypes wrapper around the CPU oracle (``libfs_oracle.so``).

TEST INFRASTRUCTURE ONLY: tests/, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg may import this package; the product path
never does.  Arrays are numpy arrays on the host.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from dataclasses import dataclass
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# FSO_ORACLE_LIB names another build of the same source (the sanitizer build of the
# oracle's own tests); by default the in-tree library.
LIB = os.environ.get("FSO_ORACLE_LIB") or os.path.join(HERE, "libfs_oracle.so")
SRC = os.path.join(HERE, "fs_oracle.cpp")

OK, E_ARG, E_ORDER, E_RANGE, E_OVERFLOW = 0, 1, 2, 3, 4


def build(force: bool = True, out: Optional[str] = None, sanitize: bool = False) -> str:
    """Compile the oracle with the host compiler (no GPU code).  sanitize: with
    AddressSanitizer and UndefinedBehaviorSanitizer (host code only), into `out`."""
    dst = out or LIB
    if force or not os.path.exists(dst):
        cmd = ["g++", "-O2", "-std=c++17", "-shared", "-fPIC", "-pthread", "-Wall"]
        if sanitize:
            cmd += ["-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=undefined"]
        subprocess.run(cmd + [SRC, "-o", dst + ".tmp"], check=True)
        os.replace(dst + ".tmp", dst)
    return dst


class _Trace(C.Structure):
    _fields_ = [("n_replicas", C.c_int32), ("n_users", C.c_int32), ("n_apps", C.c_int32),
                ("rep_off", C.c_void_p), ("ts_us", C.c_void_p), ("user", C.c_void_p),
                ("app", C.c_void_p), ("call", C.c_void_p), ("head", C.c_void_p),
                ("prev", C.c_void_p), ("len_in", C.c_void_p), ("len_sys", C.c_void_p),
                ("len_out", C.c_void_p)]


class _Engine(C.Structure):
    _fields_ = [("step_us", C.c_int64), ("cap_tokens", C.c_int64), ("overload_tokens", C.c_int64),
                ("flags", C.c_uint32)]


FSO_FCFS, FSO_BLIND, FSO_LITERAL = 1, 2, 4


class _Outputs(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("status", "admit_step", "admit_seq", "counter_after",
                                           "counter_on_arrival", "counter", "steps", "decisions",
                                           "max_gap")]


class _Metrics(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("jain", "max_gap_tokens", "svc_req_pct", "svc_int_pct",
                                           "served_users_pct", "delayed_users_pct", "throttled",
                                           "aborted_midway", "wasted_tokens")]


class _WStats(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("minutes", "user_req", "user_tok", "user_app_req",
                                           "user_app_tok", "rate_hist", "len_hist", "len_sum",
                                           "size_hist", "graph")]


RATE_BINS, LEN_BINS, SIZE_BINS, GRAPH_BINS = 128, 32, 64, 7

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = C.CDLL(LIB)
        L.fso_coef_from_expectations.argtypes = [C.c_int32, C.c_int32, C.c_void_p, C.c_void_p,
                                                 C.c_void_p, C.c_int64, C.c_void_p]
        L.fso_weights_from_history.argtypes = [C.POINTER(_Trace), C.c_int32, C.c_int64,
                                                C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p]
        L.fso_cost.argtypes = [C.POINTER(_Trace), C.c_int32, C.c_int64, C.c_void_p, C.c_int64,
                               C.c_void_p, C.c_void_p]
        L.fso_throttle.argtypes = [C.POINTER(_Trace), C.c_int64, C.c_int32, C.c_void_p, C.c_void_p,
                                   C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        L.fso_throttle_scoped.argtypes = [C.POINTER(_Trace), C.c_int64, C.c_int32, C.c_void_p,
                                          C.c_int32, C.c_void_p, C.c_int32, C.c_void_p,
                                          C.c_void_p, C.c_void_p, C.c_void_p]
        L.fso_simulate.argtypes = [C.POINTER(_Trace), C.c_void_p, C.c_void_p, C.POINTER(_Engine),
                                   C.c_int64, C.c_int32, C.c_int32, C.POINTER(_Outputs)]
        L.fso_workload_stats.argtypes = [C.POINTER(_Trace), C.c_int64, C.POINTER(_WStats)]
        L.fso_fairness_metrics.argtypes = [C.POINTER(_Trace), C.c_void_p, C.c_void_p, C.c_void_p,
                                           C.c_void_p, C.c_int64, C.c_int32, C.POINTER(_Metrics)]
        _lib = L
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


class OracleError(RuntimeError):
    def __init__(self, code, what):
        super().__init__(f"{what}: oracle code {code}")
        self.code = code


def _check(code, what):
    if code != OK:
        raise OracleError(code, what)


def _c(a, dt):
    return None if a is None else np.ascontiguousarray(a, dtype=dt)


class _TraceRef:
    """Keeps the contiguous arrays alive while the C struct points at them."""

    def __init__(self, tr):
        self.keep = dict(
            rep_off=_c(tr.rep_off, np.int64), ts_us=_c(tr.ts_us, np.int64),
            user=_c(tr.user, np.int32), app=_c(tr.app, np.int32), call=_c(tr.call, np.int32),
            head=_c(tr.head, np.int32), prev=_c(tr.prev, np.int32),
            len_in=_c(tr.len_in, np.int32), len_sys=_c(tr.len_sys, np.int32),
            len_out=_c(tr.len_out, np.int32))
        k = self.keep
        self.s = _Trace(tr.n_replicas, tr.n_users, tr.n_apps, *(_p(k[n]) for n in (
            "rep_off", "ts_us", "user", "app", "call", "head", "prev", "len_in", "len_sys",
            "len_out")))
        self.n = int(k["ts_us"].shape[0])


def coef_from_expectations(e_in, e_sys, e_out, K=1024):
    e_in = np.ascontiguousarray(e_in, np.float64)
    A, J = e_in.shape
    e_sys = np.ascontiguousarray(e_sys, np.float64)
    e_out = np.ascontiguousarray(e_out, np.float64)
    coef = np.zeros((A, J, 3), np.int64)
    _check(lib().fso_coef_from_expectations(A, J, _p(e_in), _p(e_sys), _p(e_out), K, _p(coef)),
           "fso_coef_from_expectations")
    return coef


@dataclass
class HistoryResult:
    stats: np.ndarray   # [A][J][5] records, first calls, sum L_I, sum L_S, sum L_O
    coef: np.ndarray    # [A][J][3] Q16
    t_app: np.ndarray   # [A]


def weights_from_history(tr, n_stages, K=1024, base_limit=30):
    """Eq. 1 coefficients and per-app limits derived from a historical trace."""
    t = _TraceRef(tr)
    A = tr.n_apps
    res = HistoryResult(np.zeros((A, n_stages, 5), np.int64), np.zeros((A, n_stages, 3), np.int64),
                        np.zeros(A, np.int32))
    _check(lib().fso_weights_from_history(C.byref(t.s), int(n_stages), int(K), int(base_limit),
                                          _p(res.stats), _p(res.coef), _p(res.t_app)),
           "fso_weights_from_history")
    return res


def cost(tr, coef, prio=None, coef_per_replica=False, prio_per_replica=False):
    """coef: [R or 1][A][J][3] int64 Q16; prio: [R or 1][U] int32 Q8 or None."""
    t = _TraceRef(tr)
    coef = np.ascontiguousarray(coef, np.int64)
    J = coef.shape[-2]
    cstride = coef.shape[1] * J * 3 if coef_per_replica else 0
    prio = _c(prio, np.int32)
    pstride = tr.n_users if (prio is not None and prio_per_replica) else 0
    out = np.zeros(t.n, np.int64)
    _check(lib().fso_cost(C.byref(t.s), J, cstride, _p(coef), pstride, _p(prio), _p(out)), "fso_cost")
    return out


@dataclass
class ThrottleResult:
    reason: np.ndarray
    bitmap: np.ndarray
    cnt_user: np.ndarray
    cnt_app: np.ndarray


def throttle(tr, window_us, t_user, t_app, overloaded=None, raw=True, counts=True,
             app_scope=0):
    """app_scope 0: the app limit per (user, app); 1: per app over all users."""
    t = _TraceRef(tr)
    t_app = np.ascontiguousarray(t_app, np.int32)
    ov = _c(overloaded, np.uint8)
    reason = np.zeros(t.n, np.uint8)
    bitmap = np.zeros((t.n + 31) // 32, np.uint32)
    cu = np.zeros(t.n, np.int32) if counts else None
    ca = np.zeros(t.n, np.int32) if counts else None
    _check(lib().fso_throttle_scoped(C.byref(t.s), int(window_us), int(t_user), _p(t_app),
                                     int(app_scope), _p(ov), 1 if raw else 0, _p(reason),
                                     _p(bitmap), _p(cu), _p(ca)), "fso_throttle")
    return ThrottleResult(reason, bitmap, cu, ca)


@dataclass
class SimResult:
    status: np.ndarray
    admit_step: np.ndarray
    admit_seq: np.ndarray
    counter_after: np.ndarray
    counter_on_arrival: np.ndarray
    counter: np.ndarray
    steps: np.ndarray
    decisions: np.ndarray
    max_gap: np.ndarray


def simulate(tr, cost_arr, exceed_reason, step_us, cap_tokens, overload_tokens, max_steps=-1,
             n_threads=1, check=False, flags=0):
    t = _TraceRef(tr)
    R, U, n = tr.n_replicas, tr.n_users, t.n
    cost_arr = np.ascontiguousarray(cost_arr, np.int64)
    er = _c(exceed_reason, np.uint8)
    res = SimResult(np.zeros(n, np.int8), np.zeros(n, np.int32), np.zeros(n, np.int32),
                    np.zeros(n, np.int64), np.zeros(n, np.int64), np.zeros(R * U, np.int64),
                    np.zeros(R, np.int64), np.zeros(R, np.int64), np.zeros(R, np.int64))
    o = _Outputs(*(_p(getattr(res, f)) for f in ("status", "admit_step", "admit_seq",
                                                  "counter_after", "counter_on_arrival", "counter",
                                                  "steps", "decisions", "max_gap")))
    e = _Engine(int(step_us), int(cap_tokens), int(overload_tokens), int(flags))
    _check(lib().fso_simulate(C.byref(t.s), _p(cost_arr), _p(er), C.byref(e), int(max_steps),
                              int(n_threads), 1 if check else 0, C.byref(o)), "fso_simulate")
    return res


@dataclass
class MetricsResult:
    jain: np.ndarray
    max_gap_tokens: np.ndarray
    svc_req_pct: np.ndarray
    svc_int_pct: np.ndarray
    served_users_pct: np.ndarray
    delayed_users_pct: np.ndarray
    throttled: np.ndarray
    aborted_midway: np.ndarray
    wasted_tokens: np.ndarray


def fairness_metrics(tr, cost_arr, status, admit_step, max_gap, step_us, delay_steps=0):
    t = _TraceRef(tr)
    R = tr.n_replicas
    f = lambda: np.zeros(R, np.float64)
    i = lambda: np.zeros(R, np.int64)
    res = MetricsResult(f(), f(), f(), f(), f(), f(), i(), i(), i())
    m = _Metrics(*(_p(getattr(res, n)) for n in MetricsResult.__dataclass_fields__))
    cost_arr = np.ascontiguousarray(cost_arr, np.int64)
    status = np.ascontiguousarray(status, np.int8)
    admit_step = np.ascontiguousarray(admit_step, np.int32)
    mg = _c(max_gap, np.int64)
    _check(lib().fso_fairness_metrics(C.byref(t.s), _p(cost_arr), _p(status), _p(admit_step),
                                      _p(mg), int(step_us), int(delay_steps), C.byref(m)),
           "fso_fairness_metrics")
    return res


def weights_for(wl, tr):
    """Oracle-side Q16 coefficient table [R|1][A][J][3] and whether it is per replica."""
    direct = wl.direct_coef_table(tr)
    if direct is not None:
        return direct, direct.shape[0] > 1
    e_in, e_sys, e_out = wl.expectations()
    return coef_from_expectations(e_in, e_sys, e_out, wl.weight_K)[None], False


def run_workload(wl, tr, n_threads=1, check=False, max_steps=-1, counts=False):
    """cost -> raw throttle -> step simulation -> metrics, all on the oracle."""
    coef, per_rep = weights_for(wl, tr)
    c = cost(tr, coef, coef_per_replica=per_rep)
    th = throttle(tr, wl.window_us, wl.t_user, wl.t_app, raw=True, counts=counts)
    sim = simulate(tr, c, th.reason, wl.step_us, wl.cap_tokens, wl.overload_tokens,
                   max_steps=max_steps, n_threads=n_threads, check=check)
    met = fairness_metrics(tr, c, sim.status, sim.admit_step, sim.max_gap, wl.step_us)
    return c, th, sim, met


@dataclass
class WorkloadStats:
    minutes: np.ndarray       # [R]
    user_req: np.ndarray      # [R][U]
    user_tok: np.ndarray      # [R][U]
    user_app_req: np.ndarray  # [R][U][A]
    user_app_tok: np.ndarray  # [R][U][A]
    rate_hist: np.ndarray     # [R][A+1][2][RATE_BINS]
    len_hist: np.ndarray      # [R][A][3][LEN_BINS]
    len_sum: np.ndarray       # [R][A][3]
    size_hist: np.ndarray     # [R][A][SIZE_BINS]
    graph: np.ndarray         # [R][GRAPH_BINS][5]


def workload_stats(tr, minute_us=60_000_000):
    """The workload analysis of Sec. 3 (Figs. 2-5, Table 2), per replica."""
    t = _TraceRef(tr)
    R, U, A = tr.n_replicas, tr.n_users, tr.n_apps
    z = lambda *shape: np.zeros(shape, np.int64)
    res = WorkloadStats(z(R), z(R, U), z(R, U), z(R, U, A), z(R, U, A),
                        z(R, A + 1, 2, RATE_BINS), z(R, A, 3, LEN_BINS), z(R, A, 3),
                        z(R, A, SIZE_BINS), z(R, GRAPH_BINS, 5))
    w = _WStats(*(_p(getattr(res, f)) for f in WorkloadStats.__dataclass_fields__))
    _check(lib().fso_workload_stats(C.byref(t.s), int(minute_us), C.byref(w)),
           "fso_workload_stats")
    return res

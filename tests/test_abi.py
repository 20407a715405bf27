"""The C-ABI library loads and exports every entry point include/fairserve.h declares;
host-only behaviour (argument checks, the Eq. 1 helper) needs no GPU."""
import ctypes as C
import os
import re

import numpy as np
import pytest

import oracle
import paper_2411_15997_amd as fs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            src = open(os.path.join(ROOT, "include", fn)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names |= set(re.findall(r"\b(fs_[a-z_0-9]+)\s*\(", src))
    return names


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert {"fs_cost", "fs_throttle", "fs_schedule_step", "fs_run_trace",
            "fs_fairness_metrics"} <= names
    lib = C.CDLL(fs.LIB_PATH)
    for n in sorted(names):
        assert hasattr(lib, n), n
    assert set(fs.EXPORTED) == names


def test_status_strings():
    lib = fs._lib()
    for code in range(8):
        assert lib.fs_status_string(code)


def test_coef_helper_matches_oracle_and_worked_example():
    rng = np.random.default_rng(0)
    for A, J in ((2, 1), (8, 1), (32, 20)):
        e_in = rng.uniform(1, 5000, (A, J))
        e_sys = rng.uniform(0, 500, (A, J))
        e_out = rng.uniform(1, 2000, (A, J))
        got = fs.fs_coef_from_expectations(e_in, e_sys, e_out, 1024)
        want = oracle.coef_from_expectations(e_in, e_sys, e_out, 1024)
        assert (got == want).all()
    c = fs.fs_coef_from_expectations(np.array([[10.0], [50.0]]), np.zeros((2, 1)), np.zeros((2, 1)))
    assert c[0, 0, 0] == round(2 ** 26 / 10) and c[1, 0, 0] == round(2 ** 26 / 50)
    with pytest.raises(fs.FairServeError) as e:
        fs.fs_coef_from_expectations(np.zeros((1, 1)), np.zeros((1, 1)), np.zeros((1, 1)))
    assert e.value.code == fs.FS_E_ARG


def test_synchronous_argument_errors_need_no_gpu():
    lib = fs._lib()
    assert lib.fs_cost(None, None, None, None, None) == fs.FS_E_ARG
    t = fs.fs_trace(0, 1, 1, None, None, None, None, None, None, None, None, None, None, None)
    assert lib.fs_throttle_workspace(C.byref(t)) == 0
    assert lib.fs_state_bytes(C.byref(t)) == 0
    rep = np.array([0, 4], np.int64)
    t2 = fs.fs_trace(1, 2, 2, rep.ctypes.data, 16, 16, 16, 16, None, None, None, 16, None, 16)
    w = fs.fs_weights(0, 0, 16, 0, None)          # zero stages
    assert lib.fs_cost(C.byref(t2), C.byref(w), 16, 16, None) == fs.FS_E_ARG
    t3 = fs.fs_trace(1, 2, 2, rep.ctypes.data, 16, 16, 16, 16, 16, None, None, 16, None, 16)
    w2 = fs.fs_weights(1, 0, 16, 0, None)         # call without head/prev
    assert lib.fs_cost(C.byref(t3), C.byref(w2), 16, 16, None) == fs.FS_E_ARG
    eng = fs.fs_engine(0, 10, 10, 0)               # zero step length
    out = fs.fs_outputs(*([16] * 10))
    assert lib.fs_schedule_step(256, C.byref(t2), 16, None, C.byref(eng), C.byref(out), -1,
                                None) == fs.FS_E_ARG
    t_app = np.array([-1, 3], np.int32)            # negative limit
    lim = fs.fs_limits(1000, 5, t_app.ctypes.data)
    assert lib.fs_throttle(C.byref(t2), C.byref(lim), None, 1, 16, None, None, None, 256, 1 << 20,
                           16, None) == fs.FS_E_ARG
    t_app2 = np.array([1, 3], np.int32)
    lim2 = fs.fs_limits(1000, 5, t_app2.ctypes.data)
    assert lib.fs_throttle(C.byref(t2), C.byref(lim2), None, 1, 16, None, None, None, 256, 0,
                           16, None) == fs.FS_E_WORKSPACE
    lim3 = fs.fs_limits(1000, 5, t_app2.ctypes.data, 2)   # app_scope must be 0 or 1
    assert lib.fs_throttle(C.byref(t2), C.byref(lim3), None, 1, 16, None, None, None, 256,
                           1 << 20, 16, None) == fs.FS_E_ARG


def test_history_arguments_and_workspace_need_no_gpu():
    lib = fs._lib()
    rep = np.array([0, 4000], np.int64)
    t = fs.fs_trace(1, 2, 2, rep.ctypes.data, 16, 16, 16, 16, None, None, None, 16, None, 16)
    ws = lib.fs_history_workspace(C.byref(t), 3)
    # one partial table row (2 apps x 3 stages x 5 int64) per work-group of the LDS path
    assert ws > 0 and ws % (2 * 3 * 5 * 8) == 0
    assert lib.fs_history_workspace(C.byref(t), 0) == 0
    assert lib.fs_weights_from_history(C.byref(t), 3, 0, 30, 256, None, None, 256, ws, 16,
                                       None) == fs.FS_E_ARG          # K = 0
    assert lib.fs_weights_from_history(C.byref(t), 3, 1024, -1, 256, None, None, 256, ws, 16,
                                       None) == fs.FS_E_ARG          # negative base limit
    assert lib.fs_weights_from_history(C.byref(t), 3, 1024, 30, None, None, None, 256, ws, 16,
                                       None) == fs.FS_E_ARG          # no stats buffer
    assert lib.fs_weights_from_history(C.byref(t), 3, 1024, 30, 256, None, None, 256, ws - 1,
                                       16, None) == fs.FS_E_WORKSPACE


def test_throttle_key_space_limit_needs_no_gpu():
    """fs_throttle packs (replica * U + user, app) into 32 key bits and the record index
    beside them: a larger key space is FS_E_ARG from fs_throttle and fs_run_trace (before
    anything is enqueued) and a zero workspace size, not a HIP error."""
    lib = fs._lib()
    rep = np.array([0, 4], np.int64)
    # 2^22 users (22 bits) x 1024 apps (10 bits) = 32 bits: accepted
    ok = fs.fs_trace(1, 1 << 22, 1024, rep.ctypes.data, 16, 16, 16, 16, None, None, None, 16,
                     None, 16)
    assert lib.fs_throttle_workspace(C.byref(ok)) > 0
    assert lib.fs_run_trace_workspace(C.byref(ok)) > 0
    # one more user bit: 33 key bits
    big = fs.fs_trace(1, (1 << 22) + 1, 1024, rep.ctypes.data, 16, 16, 16, 16, None, None, None,
                      16, None, 16)
    assert lib.fs_throttle_workspace(C.byref(big)) == 0
    assert lib.fs_run_trace_workspace(C.byref(big)) == 0
    t_app = np.ones(1024, np.int32)
    lim = fs.fs_limits(1000, 5, t_app.ctypes.data)
    assert lib.fs_throttle(C.byref(big), C.byref(lim), None, 1, 16, None, None, None, 256,
                           1 << 40, 16, None) == fs.FS_E_ARG
    coef = 256
    w = fs.fs_weights(1, 0, coef, 0, None)
    eng = fs.fs_engine(10, 10, 10, 0)
    out = fs.fs_outputs(*([16] * 10))
    assert lib.fs_run_trace(C.byref(big), C.byref(w), C.byref(lim), C.byref(eng), C.byref(out),
                            256, 1 << 40, None) == fs.FS_E_ARG
    # replicas x users multiply: 2^12 replicas x 2^11 users x 2^9 apps = 32 bits, one more
    # replica makes 33
    rep2 = np.zeros((1 << 12) + 2, np.int64)
    r_ok = fs.fs_trace(1 << 12, 1 << 11, 512, rep2[:(1 << 12) + 1].ctypes.data, 16, 16, 16, 16,
                       None, None, None, 16, None, 16)
    assert lib.fs_throttle_workspace(C.byref(r_ok)) > 0
    r_big = fs.fs_trace((1 << 12) + 1, 1 << 11, 512, rep2.ctypes.data, 16, 16, 16, 16, None,
                        None, None, 16, None, 16)
    assert lib.fs_throttle_workspace(C.byref(r_big)) == 0

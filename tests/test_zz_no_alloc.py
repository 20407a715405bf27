"""fs_fairness_metrics_noalloc: the metrics with the library's own fixed workspace (for
callers that cannot allocate) against fs_fairness_metrics with a caller workspace, on
two calls in a row whose second input is smaller (the fixed workspace keeps the first
call's contents, so the second shows it is cleared), through the C-ABI; and the
synchronous rejection of a trace whose workspace exceeds the fixed size."""
import ctypes as C

import numpy as np
import pytest
import torch

import paper_2411_15997_amd as fs
from gpu_common import say
from tiny import random_trace

STEP_US = 50


def _outputs(tr, rng):
    n = tr.n
    cost = rng.integers(0, 10 ** 9, n).astype(np.int64)
    status = rng.choice(np.array([0, 0, 0, 1, 2, 3], np.int8), n)
    admit_step = np.where(status == 0, tr.ts_us // STEP_US + rng.integers(0, 4, n),
                          -1).astype(np.int32)
    max_gap = rng.integers(0, 2 ** 40, tr.n_replicas).astype(np.int64)
    dt = fs.DeviceTrace(tr)
    out = fs.Outputs(dt, parity=False)
    out.status[:n].copy_(torch.as_tensor(status))
    out.admit_step[:n].copy_(torch.as_tensor(admit_step))
    out.max_gap.copy_(torch.as_tensor(max_gap))
    return dt, out, torch.as_tensor(cost).to(dt.device)


@pytest.mark.gpu
def test_noalloc_metrics_match_two_calls():
    rng = np.random.default_rng(2024)
    eng = fs.make_engine(STEP_US, 1000, 1000)
    # first call: many users (the per-wave hash aggregation), 3 replicas of 9,000 records;
    # second: fewer users (per-replica LDS tables), 2 replicas of 700 records
    for U, n, R in ((5000, 9000, 3), (300, 700, 2)):
        tr = random_trace(rng, n, U, 3, 20 * n, multi=True, n_replicas=R)
        say("noalloc metrics", U, n, R)
        dt, out, cost = _outputs(tr, rng)
        ref = fs.fs_fairness_metrics(dt, cost, out, eng, 1).host()
        got = fs.fs_fairness_metrics_noalloc(dt, cost, out, eng, 1).host()
        for k in ("throttled", "aborted_midway", "wasted_tokens"):
            assert (got[k] == ref[k]).all(), k
        for k in ("jain", "max_gap_tokens", "svc_req_pct", "svc_int_pct", "served_users_pct",
                  "delayed_users_pct"):
            np.testing.assert_allclose(got[k], ref[k], rtol=1e-9, atol=0, err_msg=k)


def test_noalloc_metrics_rejects_a_trace_beyond_the_limit():
    """Checked on the host before anything is enqueued (no GPU needed)."""
    lib = fs._lib()
    limit = int(lib.fs_metrics_noalloc_limit())
    assert limit == 32 << 20
    # the workspace holds 4 bytes per request: 9M requests need more than 32 MiB
    rep = np.array([0, 9_000_000], np.int64)
    t = fs.fs_trace(1, 8, 2, rep.ctypes.data, 16, 16, 16, 16, None, None, None, 16, None, 16)
    assert lib.fs_metrics_workspace(C.byref(t)) > limit
    eng = fs.fs_engine(10, 10, 10, 0)
    out = fs.fs_outputs(*([16] * 10))
    m = fs.fs_metrics(*([16] * 9))
    assert lib.fs_fairness_metrics_noalloc(C.byref(t), 16, C.byref(out), C.byref(eng), 0,
                                           C.byref(m), None) == fs.FS_E_WORKSPACE
    rep2 = np.array([0, 1_000_000], np.int64)
    t2 = fs.fs_trace(1, 8, 2, rep2.ctypes.data, 16, 16, 16, 16, None, None, None, 16, None, 16)
    assert lib.fs_metrics_workspace(C.byref(t2)) <= limit

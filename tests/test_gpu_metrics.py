"""fs_fairness_metrics on arbitrary scheduler outputs: statuses and admission steps are
drawn at random, so interactions end half served (aborted midway, wasted tokens) and
users are delayed.  Counts are compared exactly and the fp64 ratios within 1e-9
relative against the oracle, on both of the kernel's paths: per-replica user tables in
LDS (up to 4,096 users) and the global-memory aggregation (more users), with replicas
that are empty, shorter than one work-group's chunk of 8,192 requests, or span chunks."""
import numpy as np
import pytest

import oracle
import paper_2411_15997_amd as fs
from gpu_common import say
from tiny import random_trace
import tracegen as tg

pytestmark = pytest.mark.gpu

STEP_US = 50


def _check(tr, rng, delay):
    import torch
    n = tr.n
    cost = rng.integers(0, 10 ** 6, n).astype(np.int64)
    status = rng.choice(np.array([0, 0, 0, 1, 2, 3], np.int8), n)
    admit_step = np.where(status == 0, tr.ts_us // STEP_US + rng.integers(0, 4, n),
                          -1).astype(np.int32)
    max_gap = rng.integers(0, 2 ** 40, tr.n_replicas).astype(np.int64)
    dt = fs.DeviceTrace(tr)
    out = fs.Outputs(dt, parity=False)
    if n:
        out.status[:n].copy_(torch.as_tensor(status))
        out.admit_step[:n].copy_(torch.as_tensor(admit_step))
    out.max_gap.copy_(torch.as_tensor(max_gap))
    eng = fs.make_engine(STEP_US, 1000, 1000)
    cost_d = torch.as_tensor(cost).to(dt.device)
    m = fs.fs_fairness_metrics(dt, cost_d, out, eng, delay).host()
    mo = oracle.fairness_metrics(tr, cost, status, admit_step, max_gap, STEP_US, delay)
    for k in ("throttled", "aborted_midway", "wasted_tokens"):
        assert (m[k] == getattr(mo, k)).all(), k
    for k in ("jain", "max_gap_tokens", "svc_req_pct", "svc_int_pct", "served_users_pct",
              "delayed_users_pct"):
        np.testing.assert_allclose(m[k], getattr(mo, k), rtol=1e-9, atol=0, err_msg=k)
    return mo


@pytest.mark.parametrize("U,sizes", [
    (300, [0, 1, 8191, 8193, 20000]),   # LDS tables, chunks spanning replicas
    (4096, [30000, 5000]),              # the largest LDS table
    (5000, [7000, 0, 12000]),           # global-memory aggregation
])
@pytest.mark.parametrize("delay", [0, 2])
def test_metrics_random_outputs(U, sizes, delay):
    rng = np.random.default_rng(U + 7 * delay + len(sizes))
    tr = tg.concat([random_trace(rng, n, U, 3, 40 * max(n, 1), multi=True, max_tok=50)
                    for n in sizes])
    say("metrics", U, sizes, delay)
    mo = _check(tr, rng, delay)
    assert (mo.aborted_midway > 0).sum() >= 1 and (mo.wasted_tokens > 0).sum() >= 1


@pytest.mark.parametrize("U", [300, 5000])
def test_metrics_single_call_interactions(U):
    """Traces without interaction links (every request its own interaction): nothing can
    be aborted midway; both paths."""
    rng = np.random.default_rng(90 + U)
    tr = tg.concat([random_trace(rng, n, U, 2, 40 * n, multi=False, max_tok=50)
                    for n in (9000, 3, 16384)])
    assert tr.call is None
    say("metrics single-call", U)
    mo = _check(tr, rng, 1)
    assert (mo.aborted_midway == 0).all() and (mo.wasted_tokens == 0).all()


def _gpu_metrics(tr, cost, status, admit_step, max_gap, step_us):
    import torch
    n = tr.n
    dt = fs.DeviceTrace(tr)
    out = fs.Outputs(dt, parity=False)
    out.status[:n].copy_(torch.as_tensor(status))
    out.admit_step[:n].copy_(torch.as_tensor(admit_step))
    out.max_gap.copy_(torch.as_tensor(max_gap))
    eng = fs.make_engine(step_us, 1000, 1000)
    return fs.fs_fairness_metrics(dt, torch.as_tensor(cost).to(dt.device), out, eng, 0).host()


@pytest.mark.parametrize("U", [4, 5000])
def test_metrics_charged_service_limit(U):
    """Admitted costs near 2^62 (both aggregation paths): below a replica total of 2^62
    the GPU's Jain index matches the oracle, at 2^62 both report an overflow, and an
    admitted cost out of range is a range error on both sides."""
    q = 1 << 60
    n = 8
    tr = tg.Trace(2, U, 1, np.array([0, 4, 8], np.int64), np.zeros(n, np.int64),
                  np.array([0, 1, 2, 3] * 2, np.int32) % U, np.zeros(n, np.int32), None, None,
                  None, np.ones(n, np.int32), None, np.zeros(n, np.int32))
    st = np.zeros(n, np.int8)
    adm = np.zeros(n, np.int32)
    mg = np.zeros(2, np.int64)
    ok = np.array([3 * q - 1, q - 1, 0, 0, q - 1, q - 1, q - 1, q - 1], np.int64)
    want = oracle.fairness_metrics(tr, ok, st, adm, mg, 10)
    got = _gpu_metrics(tr, ok, st, adm, mg, 10)
    np.testing.assert_allclose(got["jain"], want.jain, rtol=1e-9, atol=0)
    for bad, code in ((np.array([q, q, q, q, 1, 1, 1, 1], np.int64), fs.FS_E_OVERFLOW),
                      (np.array([(1 << 62) - 1] * 8, np.int64), fs.FS_E_OVERFLOW),
                      (np.array([1, 1, 1, 1, 1, -1, 1, 1], np.int64), fs.FS_E_RANGE)):
        with pytest.raises(oracle.OracleError) as oe:
            oracle.fairness_metrics(tr, bad, st, adm, mg, 10)
        with pytest.raises(fs.FairServeError) as ge:
            _gpu_metrics(tr, bad, st, adm, mg, 10)
        assert ge.value.code == oe.value.code == code

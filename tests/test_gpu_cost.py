"""Parity of fs_cost (Eq. 2 per call) with the oracle, bit-exact."""
import numpy as np
import pytest

import oracle
import paper_2411_15997_amd as fs
from gpu_common import say, workload_trace
from tiny import random_trace
import tracegen as tg

pytestmark = pytest.mark.gpu


def _gpu_cost(tr, coef, prio=None, per_rep=False, prio_per_rep=False):
    dt = fs.DeviceTrace(tr)
    w, keep = fs.make_weights(dt, coef, prio, per_rep, prio_per_rep)
    return fs.fs_cost(dt, w).cpu().numpy()


@pytest.mark.parametrize("name,kw", [
    ("c1_small", {}),
    ("c2_replicas", dict(replicas=3, records=20011)),
    ("c4_sweep", dict(replicas=16, records=5003)),
    ("c5_tenant", dict(records=100003, users=20000)),
])
def test_cost_workloads(name, kw):
    wl, tr = workload_trace(name, **kw)
    say("cost", name, tr.n)
    coef, per_rep = fs.workload_weights(wl, tr)
    ocoef, _ = oracle.weights_for(wl, tr)
    assert (coef == ocoef).all()
    got = _gpu_cost(tr, coef, per_rep=per_rep)
    want = oracle.cost(tr, ocoef, coef_per_replica=per_rep)
    assert (got == want).all()


def test_cost_with_priorities_and_ragged_tail():
    rng = np.random.default_rng(7)
    tr = random_trace(rng, 1003, 50, 5, 10 ** 6, multi=True, max_tok=70000, n_replicas=3)
    coef = rng.integers(0, 1 << 30, size=(3, 5, 4, 3)).astype(np.int64)
    prio = rng.integers(0, 1 << 12, size=(3, 50)).astype(np.int32)
    got = _gpu_cost(tr, coef, prio, per_rep=True, prio_per_rep=True)
    want = oracle.cost(tr, coef, prio, coef_per_replica=True, prio_per_replica=True)
    assert (got == want).all()
    for n in (1, 2, 3, 5, 7):
        sub = tr.replica(0)
        small = tg.Trace(1, sub.n_users, sub.n_apps, np.array([0, n], np.int64),
                         *(None if getattr(sub, k) is None else getattr(sub, k)[:n] for k in (
                             "ts_us", "user", "app", "call", "head", "prev", "len_in", "len_sys",
                             "len_out")))
        small.call = None; small.head = None; small.prev = None
        assert (_gpu_cost(small, coef[:1]) == oracle.cost(small, coef[:1])).all()


def test_cost_full_weight_sweep():
    """The weight-sweep workload at full size (20.48M calls, one table per replica)."""
    wl, tr = workload_trace("c4_sweep")
    say("cost full", tr.n)
    coef, per_rep = fs.workload_weights(wl, tr)
    got = _gpu_cost(tr, coef, per_rep=per_rep)
    want = oracle.cost(tr, coef, coef_per_replica=per_rep)
    assert (got == want).all()


def test_cost_errors_match_oracle():
    rng = np.random.default_rng(8)
    tr = random_trace(rng, 64, 4, 2, 1000, multi=False)
    coef = np.full((1, 2, 1, 3), 1 << 16, np.int64)
    bad_user = tg.Trace(**{**tr.__dict__, "user": tr.user.copy()})
    bad_user.user[10] = 4
    big = coef.copy(); big[0, 1, 0, 0] = 1 << 36
    huge = np.full((1, 2, 1, 3), (1 << 36) - 1, np.int64)
    prio = np.full((1, 4), 65535, np.int32)
    lens = tg.Trace(**{**tr.__dict__, "len_in": np.full(64, (1 << 24) - 1, np.int32)})
    unit = np.full((1, 4), 256, np.int32)
    for t, c, p, code in ((bad_user, coef, unit, fs.FS_E_RANGE), (tr, big, None, fs.FS_E_RANGE),
                          (lens, huge, prio, fs.FS_E_OVERFLOW)):
        with pytest.raises(oracle.OracleError) as oe:
            oracle.cost(t, c, p)
        with pytest.raises(fs.FairServeError) as ge:
            _gpu_cost(t, c, p)
        assert ge.value.code == oe.value.code == code
    # Eq. 2 reads the user only through its priority: without priorities the user id is
    # not read, on either side
    assert (_gpu_cost(bad_user, coef, None) == oracle.cost(bad_user, coef, None)).all()


def test_cost_empty_trace():
    tr = tg.Trace(1, 1, 1, np.array([0, 0], np.int64), np.zeros(0, np.int64), np.zeros(0, np.int32),
                  np.zeros(0, np.int32), None, None, None, np.zeros(0, np.int32), None,
                  np.zeros(0, np.int32))
    dt = fs.DeviceTrace(tr)
    w, keep = fs.make_weights(dt, np.ones((1, 1, 1, 3), np.int64))
    fs.fs_cost(dt, w)

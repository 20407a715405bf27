"""fs_workload_stats (the workload analysis of Sec. 3: Fig. 2 rates per user overall
and per application, Figs. 3-5 lengths and calls per application, Table 2 graph rows)
against the oracle, bit-exact: random multi-replica traces with empty replicas and
interactions, the workload recipes at reduced size, and the large-tenant and
weight-sweep workloads at full size."""
import numpy as np
import pytest

import oracle
import paper_2411_15997_amd as fs
from gpu_common import say, workload_trace
from tiny import random_trace
import tracegen as tg

pytestmark = pytest.mark.gpu

FIELDS = ("minutes", "user_req", "user_tok", "user_app_req", "user_app_tok", "rate_hist",
          "len_hist", "len_sum", "size_hist", "graph")


def _compare(tr, minute=60_000_000, per_app=True):
    dt = fs.DeviceTrace(tr)
    got = fs.fs_workload_stats(dt, minute, per_app=per_app).host()
    want = oracle.workload_stats(tr, minute)
    for k in FIELDS:
        if got[k] is None:
            continue
        w = getattr(want, k)
        bad = np.argwhere(got[k].reshape(w.shape) != w)
        assert bad.size == 0, f"{k}: {len(bad)} mismatches, first {bad[:3].tolist()}"


@pytest.mark.parametrize("seed", range(8))
def test_random_traces(seed):
    rng = np.random.default_rng(900 + seed)
    parts = []
    for _ in range(int(rng.integers(1, 5))):
        n = int(rng.choice([0, 1, 7, 300, 3000]))
        parts.append(random_trace(rng, n, int(rng.integers(1, 40)), int(rng.integers(1, 6)),
                                  int(rng.integers(1, 10 ** 6)), multi=bool(rng.integers(0, 2)),
                                  max_tok=int(rng.choice([0, 3, 5000]))))
    U = max(p.n_users for p in parts)
    A = max(p.n_apps for p in parts)
    parts = [tg.Trace(**{**p.__dict__, "n_users": U, "n_apps": A}) for p in parts]
    multi = [p.call is not None for p in parts]
    if any(multi) and not all(multi):
        parts = [p if p.call is not None else tg.Trace(**{
            **p.__dict__, "call": np.zeros(p.n, np.int32), "head": np.arange(p.n, dtype=np.int32),
            "prev": np.full(p.n, -1, np.int32)}) for p in parts]
    tr = tg.concat(parts)
    say("workload stats random", seed, tr.n_replicas, tr.n)
    _compare(tr, minute=int(rng.choice([1, 1000, 60_000])), per_app=bool(seed % 2))


@pytest.mark.parametrize("seed", range(6))
def test_random_many_replicas(seed):
    """256 or more replicas whose (user, app) tables fit in LDS: one work-group per
    replica does every accumulation (empty and one-request replicas, interactions or
    none, system tokens or none, tables from a few entries to about 9,000)."""
    rng = np.random.default_rng(950 + seed)
    R = int(rng.integers(256, 300))
    U = int(rng.choice([1, 7, 300, 1100]))
    A = int(rng.integers(1, 9))
    multi = bool(seed % 2)
    parts = [random_trace(rng, int(rng.choice([0, 1, 20, 300])), U, A,
                          int(rng.integers(1, 10 ** 6)), multi=multi,
                          max_tok=int(rng.choice([0, 3, 5000]))) for _ in range(R)]
    tr = tg.concat(parts)
    if seed % 3 == 0:
        tr = tg.Trace(**{**tr.__dict__, "len_sys": None})
    say("workload stats many replicas", seed, tr.n_replicas, tr.n_users, tr.n_apps, tr.n)
    _compare(tr, minute=int(rng.choice([1, 1000, 60_000])), per_app=bool(seed % 2))


@pytest.mark.parametrize("U,A", [(1100, 8), (1400, 8)])
def test_many_replicas_length_table_copies(U, A):
    """The per-replica work-group keeps copies of the per-app length sums and histograms
    when LDS allows (1,100 users x 8 apps) and a single one when the (user, app) table
    leaves no room for them (1,400 x 8)."""
    rng = np.random.default_rng(990 + U)
    parts = [random_trace(rng, int(rng.choice([0, 1, 40, 200])), U, A,
                          int(rng.integers(1, 10 ** 6)), multi=True, max_tok=5000)
             for _ in range(260)]
    tr = tg.concat(parts)
    say("workload stats length copies", U, A, tr.n)
    _compare(tr, minute=60_000, per_app=True)


def test_errors_many_replicas():
    rng = np.random.default_rng(5)
    tr = random_trace(rng, 40, 6, 3, 1000, multi=True, n_replicas=260)
    bad = tg.Trace(**{**tr.__dict__, "user": tr.user.copy(), "head": tr.head.copy()})
    bad.user[int(tr.rep_off[17]) + 3] = 6
    later = np.nonzero(tr.call[int(tr.rep_off[30]):int(tr.rep_off[31])] > 0)[0]
    if later.size:
        bad.head[int(tr.rep_off[30]) + int(later[0])] = int(later[0]) + 1  # ahead of itself
    with pytest.raises(oracle.OracleError) as oe:
        oracle.workload_stats(bad)
    with pytest.raises(fs.FairServeError) as ge:
        fs.fs_workload_stats(fs.DeviceTrace(bad))
    assert ge.value.code == oe.value.code == fs.FS_E_RANGE


@pytest.mark.parametrize("name,kw", [("c1_small", {}), ("c2_replicas", dict(replicas=5, records=20000)),
                                     ("c4_sweep", dict(replicas=40)), ("c4_sweep", dict(replicas=300)),
                                     ("c5_tenant", dict(records=200_003, users=30_000))])
def test_workload_recipes(name, kw):
    wl, tr = workload_trace(name, **kw)
    say("workload stats", name, tr.n)
    _compare(tr)


@pytest.mark.parametrize("name", ["c5_tenant", "c4_sweep"])
def test_full_size(name):
    wl, tr = workload_trace(name)
    say("workload stats full", name, tr.n)
    _compare(tr)


def test_errors_match_oracle():
    rng = np.random.default_rng(3)
    tr = random_trace(rng, 50, 4, 2, 1000, multi=True)
    bad_user = tg.Trace(**{**tr.__dict__, "user": tr.user.copy()})
    bad_user.user[7] = 4
    neg_ts = tg.Trace(**{**tr.__dict__, "ts_us": tr.ts_us - 10 ** 9})
    for t in (bad_user, neg_ts):
        with pytest.raises(oracle.OracleError) as oe:
            oracle.workload_stats(t)
        with pytest.raises(fs.FairServeError) as ge:
            fs.fs_workload_stats(fs.DeviceTrace(t))
        assert ge.value.code == oe.value.code == fs.FS_E_RANGE

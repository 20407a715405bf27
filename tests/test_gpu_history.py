"""Parity of fs_weights_from_history (Eq. 1 from a history's sample means, and the app
limits scaled by the mean calls per interaction) with the oracle, bit-exact."""
import numpy as np
import pytest

import oracle
from gpu_common import say, workload_trace
from tiny import random_trace
import tracegen as tg
import paper_2411_15997_amd as fs

pytestmark = pytest.mark.gpu


def _gpu(tr, J, K=1024, base=30, coef=True, limits=True):
    dt = fs.DeviceTrace(tr)
    st, c, t = fs.fs_weights_from_history(dt, J, K=K, base_limit=base, coef=coef, limits=limits)
    return (st.cpu().numpy(), None if c is None else c.cpu().numpy(),
            None if t is None else t.cpu().numpy())


def _check(tr, J, K=1024, base=30):
    st, c, t = _gpu(tr, J, K, base)
    o = oracle.weights_from_history(tr, J, K=K, base_limit=base)
    assert (st == o.stats).all()
    assert (c == o.coef).all(), np.argwhere(c != o.coef)[:5]
    assert (t == o.t_app).all()
    return o


@pytest.mark.parametrize("seed", range(6))
def test_random_histories(seed):
    rng = np.random.default_rng(200 + seed)
    n = int(rng.integers(1, 20000))
    A = int(rng.integers(1, 40))
    tr = random_trace(rng, n, 5, A, 1000, multi=bool(seed % 3), max_tok=int(rng.integers(1, 5000)),
                      n_replicas=int(rng.integers(1, 4)))
    J = int(rng.integers(1, 6))
    say("history random", seed, tr.n, A, J)
    _check(tr, J, K=int(rng.integers(1, 1 << 20)), base=int(rng.integers(0, 200)))


def test_ragged_sizes_and_no_system_tokens():
    rng = np.random.default_rng(21)
    for n in (1, 2, 3, 4, 5, 63, 64, 65, 1023, 1024, 1025):
        tr = random_trace(rng, n, 3, 3, 50, multi=True, max_tok=300)
        _check(tr, 3)
        nosys = tg.Trace(**{**tr.__dict__, "len_sys": None})
        _check(nosys, 2)


def test_table_too_large_for_lds():
    # 1024 apps x 8 stages = 8192 groups: accumulated in global memory
    rng = np.random.default_rng(22)
    tr = random_trace(rng, 30000, 4, 1024, 1000, multi=True, max_tok=2000)
    say("history global table", tr.n)
    _check(tr, 8)


def test_empty_groups_and_optional_outputs():
    rng = np.random.default_rng(23)
    tr = random_trace(rng, 500, 3, 2, 100, multi=True, max_tok=100)
    tr = tg.Trace(**{**tr.__dict__, "n_apps": 6})     # apps 2..5 have no history
    o = _check(tr, 5)
    assert (o.stats[2:, :, 0] == 0).all()
    st, c, t = _gpu(tr, 5, coef=False, limits=False)
    assert c is None and t is None and (st == o.stats).all()


@pytest.mark.parametrize("name,kw,J", [
    ("c2_replicas", dict(replicas=8, records=100_000), 1),
    ("c5_tenant", dict(records=1_000_003, users=30_000), 20),
    ("c4_sweep", dict(replicas=64), 1),
])
def test_workload_histories(name, kw, J):
    wl, tr = workload_trace(name, **kw)
    say("history", name, tr.n)
    _check(tr, J, K=wl.weight_K, base=30)


def test_errors_match_oracle():
    rng = np.random.default_rng(24)
    tr = random_trace(rng, 300, 3, 2, 100, multi=True, max_tok=50)
    bad = tg.Trace(**{**tr.__dict__, "app": tr.app.copy()})
    bad.app[17] = 5
    with pytest.raises(oracle.OracleError) as oe:
        oracle.weights_from_history(bad, 2)
    with pytest.raises(fs.FairServeError) as ge:
        _gpu(bad, 2)
    assert ge.value.code == oe.value.code == fs.FS_E_RANGE
    big = tg.Trace(**{**tr.__dict__, "len_in": np.ones_like(tr.len_in),
                      "len_sys": np.zeros_like(tr.len_in), "len_out": np.zeros_like(tr.len_in)})
    with pytest.raises(fs.FairServeError) as ge:
        _gpu(big, 1, K=1 << 20)       # coefficient 2^37 for system tokens
    assert ge.value.code == fs.FS_E_RANGE
    with pytest.raises(fs.FairServeError) as ge:
        _gpu(tr, 1, K=0)
    assert ge.value.code == fs.FS_E_ARG

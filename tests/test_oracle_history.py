"""Pins of the oracle's offline derivation of weights and app limits from a history
(Eq. 1 with sample means; the app limit scaled by the mean calls per interaction).

Each pin reaches the result by another route than the oracle's own formula:
numpy group sums, the double-precision Eq. 1 routine on exactly representable means,
the paper's worked example (Sec. 3), hand-derived half-even ties, metamorphic
relations (pooling, duplication), closed forms of the limit, and the law of large
numbers on a workload with known expectations.
"""
import numpy as np
import pytest

import oracle
from tiny import random_trace
import tracegen as tg
from tracegen import Trace, concat


def _trace(app, call, lin, lsys, lout, n_apps, head=None, prev=None):
    n = len(app)
    call = None if call is None else np.asarray(call, np.int32)
    if call is not None and head is None:
        # chains in stream order: call j follows the last record with call j - 1
        head = np.zeros(n, np.int32)
        prev = np.full(n, -1, np.int32)
        last = {}
        for i in range(n):
            if call[i] == 0:
                head[i] = i
            else:
                prev[i] = last[int(call[i]) - 1]
                head[i] = head[prev[i]]
            last[int(call[i])] = i
    return Trace(1, 1, n_apps, np.array([0, n], np.int64), np.arange(n, dtype=np.int64),
                 np.zeros(n, np.int32), np.asarray(app, np.int32), call,
                 None if call is None else np.asarray(head, np.int32),
                 None if call is None else np.asarray(prev, np.int32),
                 np.asarray(lin, np.int32), None if lsys is None else np.asarray(lsys, np.int32),
                 np.asarray(lout, np.int32))


@pytest.mark.parametrize("seed", range(5))
def test_stats_are_group_sums(seed):
    rng = np.random.default_rng(seed)
    J = int(rng.integers(1, 5))
    tr = random_trace(rng, int(rng.integers(1, 400)), 4, int(rng.integers(1, 6)), 100,
                      multi=True, max_tok=1000, n_replicas=int(rng.integers(1, 4)))
    h = oracle.weights_from_history(tr, J)
    j = np.minimum(tr.call, J - 1)
    key = tr.app.astype(np.int64) * J + j
    G = tr.n_apps * J
    want = np.stack([np.bincount(key, minlength=G),
                     np.bincount(key, weights=(tr.call == 0), minlength=G),
                     np.bincount(key, weights=tr.len_in, minlength=G),
                     np.bincount(key, weights=tr.len_sys, minlength=G),
                     np.bincount(key, weights=tr.len_out, minlength=G)], axis=1)
    assert (h.stats.reshape(G, 5) == want.astype(np.int64)).all()


def test_constant_lengths_match_the_eq1_routine():
    """With constant lengths per (app, stage) the sample means are exact, so the
    history route and the double-precision Eq. 1 routine must agree exactly."""
    rng = np.random.default_rng(7)
    A, J = 5, 3
    L = rng.integers(1, 3000, size=(A, J, 3))
    rows = []
    for a in range(A):
        for j in range(J):
            rows += [(a, j)] * int(rng.integers(1, 9))
    rows.sort(key=lambda r: r[1])   # every stage-j record after some stage j-1 record
    app = [a for a, _ in rows]
    call = [j for _, j in rows]
    lin = [L[a, j, 0] for a, j in rows]
    lsys = [L[a, j, 1] for a, j in rows]
    lout = [L[a, j, 2] for a, j in rows]
    tr = _trace(app, call, lin, lsys, lout, A)
    h = oracle.weights_from_history(tr, J, K=1024)
    e = oracle.coef_from_expectations(L[..., 0].astype(float), L[..., 1].astype(float),
                                      L[..., 2].astype(float), 1024)
    assert (h.coef == e).all()


def test_worked_example_from_history():
    """Sec. 3's example: apps whose requests average 10 and 50 tokens; 5 tokens then
    give 50 % and 10 % of the normalised service."""
    lin = [4, 16, 10, 35, 65, 50]      # app 0 averages 10, app 1 averages 50
    tr = _trace([0, 0, 0, 1, 1, 1], None, lin, None, [0] * 6, 2)
    K = 1024
    h = oracle.weights_from_history(tr, 1, K=K)
    probe = Trace(1, 2, 2, np.array([0, 2], np.int64), np.zeros(2, np.int64),
                  np.array([0, 1], np.int32), np.array([0, 1], np.int32), None, None, None,
                  np.array([5, 5], np.int32), None, np.zeros(2, np.int32))
    frac = oracle.cost(probe, h.coef[None]) / float(1 << 16) / K
    assert abs(frac[0] - 0.5) <= 5 * 2.0 ** -16 and abs(frac[1] - 0.1) <= 5 * 2.0 ** -16


def test_half_even_ties_by_hand():
    """K = 1: coefficient = 65536 n x / D.  D = 2^17 makes n = 1, 3, 5 land on
    0.5, 1.5, 2.5 for x = 1 (-> 0, 2, 2) and on 1, 3, 5 for x = 2."""
    for n, want in ((1, 0), (3, 2), (5, 2)):
        lin = [131072] + [0] * (n - 1)
        tr = _trace([0] * n, None, lin, None, [0] * n, 1)
        h = oracle.weights_from_history(tr, 1, K=1)
        assert h.coef[0, 0].tolist() == [want, n, want]
    # system tokens weigh twice: D = 2 * 65536 from one system-token count of 65536
    tr = _trace([0], None, [0], [65536], [0], 1)
    assert oracle.weights_from_history(tr, 1, K=1).coef[0, 0].tolist() == [0, 1, 0]


def test_empty_groups_pool_the_app_then_the_history():
    rng = np.random.default_rng(3)
    tr = random_trace(rng, 300, 3, 3, 100, multi=True, max_tok=500)
    # app 2 never reaches stage >= 2, app 1 disappears entirely
    keep = ~((tr.app == 1) | ((tr.app == 2) & (tr.call >= 2)))
    # dropping records must keep chains valid: drop whole interactions instead
    bad_heads = set(tr.head[~keep].tolist())
    keep = np.array([h not in bad_heads for h in tr.head])
    idx = np.nonzero(keep)[0]
    remap = -np.ones(tr.n, np.int64)
    remap[idx] = np.arange(idx.size)
    sub = Trace(1, tr.n_users, 3, np.array([0, idx.size], np.int64), tr.ts_us[idx],
                tr.user[idx], tr.app[idx], tr.call[idx], remap[tr.head[idx]].astype(np.int32),
                np.where(tr.prev[idx] >= 0, remap[np.maximum(tr.prev[idx], 0)], -1).astype(np.int32),
                tr.len_in[idx], tr.len_sys[idx], tr.len_out[idx])
    J = 4
    h = oracle.weights_from_history(sub, J)
    per_app = oracle.weights_from_history(sub, 1)           # J = 1 pools each app's stages
    assert (h.stats[2, 2:, 0] == 0).all() and (h.stats[1, :, 0] == 0).all()
    for j in range(2, J):
        assert (h.coef[2, j] == per_app.coef[2, 0]).all()
    one_app = Trace(**{**sub.__dict__, "app": np.zeros_like(sub.app)})
    pooled = oracle.weights_from_history(one_app, 1)          # one app pools everything
    for j in range(J):
        assert (h.coef[1, j] == pooled.coef[0, 0]).all()
    # no tokens at all: w = K, coefficients 2^16 x
    z = _trace([0, 0], None, [0, 0], None, [0, 0], 1)
    assert oracle.weights_from_history(z, 2, K=77).coef.tolist() == [[[65536, 131072, 65536]] * 2]


def test_duplicated_history_keeps_weights_and_limits():
    rng = np.random.default_rng(5)
    tr = random_trace(rng, 200, 4, 3, 100, multi=True, max_tok=900)
    h1 = oracle.weights_from_history(tr, 3, base_limit=17)
    h2 = oracle.weights_from_history(concat([tr, tr]), 3, base_limit=17)
    assert (h2.stats == 2 * h1.stats).all()
    assert (h2.coef == h1.coef).all() and (h2.t_app == h1.t_app).all()


def test_limits_closed_form():
    # app 0: interactions of exactly 3 calls; app 1: of 1 and 2 calls (mean 1.5);
    # app 2: 7 calls over 3 interactions (mean 7/3)
    calls = {0: [[0, 1, 2]] * 4, 1: [[0], [0, 1]] * 3, 2: [[0, 1, 2], [0, 1], [0, 1]]}
    trs = []
    for a, inters in calls.items():
        for c in inters:
            trs.append(_trace([a] * len(c), c, [1] * len(c), None, [1] * len(c), 3))
    tr = concat(trs)
    h = oracle.weights_from_history(tr, 1, base_limit=30)
    assert h.t_app.tolist() == [90, 45, 70]
    assert oracle.weights_from_history(tr, 1, base_limit=1).t_app.tolist() == [3, 2, 3]
    # an app with no first call keeps the base limit
    z = _trace([0, 0], None, [1, 1], None, [1, 1], 2)
    assert oracle.weights_from_history(z, 1, base_limit=12).t_app.tolist() == [12, 12]


def test_large_history_recovers_the_expectations():
    """Law of large numbers: coefficients from a long synthetic history approach the
    ones computed from the generator's nominal expectations (within 10 %: the token
    lognormals are clipped, which lowers the largest means by a few per cent), and the
    limits approach ceil(30 E[m_a]).  Swapping token classes or apps misses by far more."""
    wl = tg.scaled(tg.WORKLOADS["c2_replicas"], replicas=4, records=100_000)
    tr = tg.generate(wl)
    h = oracle.weights_from_history(tr, 1, K=wl.weight_K, base_limit=30)
    e_in, e_sys, e_out = wl.expectations()
    exact = oracle.coef_from_expectations(e_in, e_sys, e_out, wl.weight_K)
    rel = np.abs(h.coef - exact) / exact
    assert rel.max() < 0.10, rel.max()
    lim = np.asarray(wl.t_app, float)
    assert (np.abs(h.t_app - lim) <= 0.05 * lim + 1).all(), (h.t_app, lim)


def test_errors():
    tr = _trace([0, 1], None, [1, 2], None, [3, 4], 2)
    with pytest.raises(oracle.OracleError) as e:
        oracle.weights_from_history(tr, 1, K=0)
    assert e.value.code == oracle.E_ARG
    bad = _trace([0, 2], None, [1, 2], None, [3, 4], 2)
    with pytest.raises(oracle.OracleError) as e:
        oracle.weights_from_history(bad, 1)
    assert e.value.code == oracle.E_RANGE
    # a coefficient of 2^37 (K = 2^20, x = 2, w = 1)
    big = _trace([0], None, [1], None, [0], 1)
    with pytest.raises(oracle.OracleError) as e:
        oracle.weights_from_history(big, 1, K=1 << 20)
    assert e.value.code == oracle.E_RANGE
    # a limit above INT32_MAX: base 2^31 - 1 and two calls per interaction
    two = _trace([0, 0], [0, 1], [1, 1], None, [1, 1], 1)
    with pytest.raises(oracle.OracleError) as e:
        oracle.weights_from_history(two, 1, base_limit=2 ** 31 - 1)
    assert e.value.code == oracle.E_RANGE

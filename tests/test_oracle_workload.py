"""Pins of the oracle's workload analysis (Sec. 3: Fig. 2 request and token rates per
user overall and per application, Figs. 3-5 lengths and calls per application,
Table 2 graph sizes): a hand-built trace with known rates, brute force on tiny random
traces, invariants that tie the outputs together, and Table 2's request shares recovered
from the large-tenant generator, whose interaction sizes are drawn from that table."""
import numpy as np
import pytest

import oracle
import tracegen as tg
from tiny import random_trace
from tracegen import Trace

MIN = 60_000_000


def _bin_ratio(x, M):
    """Rate bin by its definition: 0 for x = 0, else 64 + the largest k with M 2^k <= x."""
    if x == 0:
        return 0
    k = 0
    if M <= x:
        while M * 2 ** (k + 1) <= x:
            k += 1
    else:
        k = -1
        while x * 2 ** (-k) < M:
            k -= 1
    return 64 + k


def _graph_bin(s):
    for b, hi in enumerate((1, 10, 20, 30, 40, 50)):
        if s <= hi:
            return b
    return 6


def test_rates_of_a_hand_built_trace():
    """User 0 sends 3 requests in each of 4 minutes (RPM 3, bin 64 + 1); user 1 one
    request (RPM 1/4, bin 64 - 2); user 2 none (no bin).  Tokens: 10 per request of user 0
    (TPM 30: bin 64 + 4), 0 for user 1 (bin 0)."""
    ts, user = [], []
    for m in range(4):
        for j in range(3):
            ts.append(m * MIN + 1000 * j)
            user.append(0)
    ts.append(2 * MIN + 5)
    user.append(1)
    order = np.argsort(np.array(ts), kind="stable")
    ts = np.array(ts, np.int64)[order]
    user = np.array(user, np.int32)[order]
    n = ts.size
    li = np.where(user == 0, 6, 0).astype(np.int32)
    lo = np.where(user == 0, 4, 0).astype(np.int32)
    tr = Trace(1, 3, 1, np.array([0, n], np.int64), ts, user, np.zeros(n, np.int32), None, None,
               None, li, None, lo)
    st = oracle.workload_stats(tr, MIN)
    assert st.minutes[0] == 4
    assert list(st.user_req[0]) == [12, 1, 0] and list(st.user_tok[0]) == [120, 0, 0]
    rpm, tpm = st.rate_hist[0, 1, 0], st.rate_hist[0, 1, 1]   # overall row (A = 1)
    assert rpm[65] == 1 and rpm[62] == 1 and rpm.sum() == 2
    assert tpm[68] == 1 and tpm[0] == 1 and tpm.sum() == 2
    assert (st.rate_hist[0, 0] == st.rate_hist[0, 1]).all()     # one app: the same users
    # lengths: 12 records of L_I = 6 (bin 3), one of 0 (bin 0); L_S absent (bin 0)
    assert st.len_hist[0, 0, 0, 3] == 12 and st.len_hist[0, 0, 0, 0] == 1
    assert st.len_hist[0, 0, 1, 0] == 13 and st.len_sum[0, 0].tolist() == [72, 0, 48]
    # every record a single-call interaction: Table 2's first row only
    assert st.size_hist[0, 0, 0] == 13 and st.size_hist[0].sum() == 13
    assert st.graph[0, 0].tolist() == [13, 13, 72, 48, 0] and st.graph[0, 1:].sum() == 0


@pytest.mark.parametrize("seed", range(6))
def test_brute_force_tiny(seed):
    rng = np.random.default_rng(500 + seed)
    R, U, A = 2, 4, 3
    tr = random_trace(rng, int(rng.integers(1, 40)), U, A, 5 * 60, multi=True, max_tok=9,
                      n_replicas=R)
    minute = 60
    st = oracle.workload_stats(tr, minute)
    for r in range(R):
        a0, a1 = int(tr.rep_off[r]), int(tr.rep_off[r + 1])
        n = a1 - a0
        M = (max(tr.ts_us[a0:a1]) // minute + 1) if n else 0
        assert st.minutes[r] == M
        req = np.zeros((U, A), np.int64); tok = np.zeros((U, A), np.int64)
        size = {}
        for i in range(n):
            g = a0 + i
            u, a = tr.user[g], tr.app[g]
            req[u, a] += 1
            tok[u, a] += int(tr.len_in[g]) + int(tr.len_sys[g]) + int(tr.len_out[g])
            h = i if tr.call[g] == 0 else int(tr.head[g])
            size[h] = size.get(h, 0) + 1
        assert (st.user_app_req[r] == req).all() and (st.user_app_tok[r] == tok).all()
        assert (st.user_req[r] == req.sum(1)).all() and (st.user_tok[r] == tok.sum(1)).all()
        want = np.zeros((A + 1, 2, 128), np.int64)
        for u in range(U):
            if req[u].sum():
                want[A, 0, _bin_ratio(int(req[u].sum()), M)] += 1
                want[A, 1, _bin_ratio(int(tok[u].sum()), M)] += 1
            for a in range(A):
                if req[u, a]:
                    want[a, 0, _bin_ratio(int(req[u, a]), M)] += 1
                    want[a, 1, _bin_ratio(int(tok[u, a]), M)] += 1
        assert (st.rate_hist[r] == want).all()
        gr = np.zeros((7, 5), np.int64); sh = np.zeros((A, 64), np.int64)
        for i in range(n):
            g = a0 + i
            h = i if tr.call[g] == 0 else int(tr.head[g])
            b = _graph_bin(size[h])
            if h == i:
                gr[b, 0] += 1
                sh[tr.app[g], min(size[h], 64) - 1] += 1
            gr[b, 1] += 1
            gr[b, 2] += tr.len_in[g]; gr[b, 3] += tr.len_out[g]; gr[b, 4] += tr.len_sys[g]
        assert (st.graph[r] == gr).all() and (st.size_hist[r] == sh).all()
        lh = np.zeros((A, 3, 32), np.int64)
        for i in range(n):
            g = a0 + i
            for x, L in enumerate((tr.len_in[g], tr.len_sys[g], tr.len_out[g])):
                lh[tr.app[g], x, 0 if L == 0 else int(L).bit_length()] += 1
        assert (st.len_hist[r] == lh).all()


@pytest.mark.parametrize("name", ["c2_replicas", "c5_tenant"])
def test_invariants_on_workload_recipes(name):
    base = tg.WORKLOADS[name]
    wl = tg.scaled(base, replicas=min(base.n_replicas, 3), records=20_000)
    tr = tg.generate(wl)
    st = oracle.workload_stats(tr)
    A = tr.n_apps
    for r in range(tr.n_replicas):
        n = int(tr.rep_off[r + 1] - tr.rep_off[r])
        assert st.user_req[r].sum() == n
        assert (st.user_app_req[r].sum(1) == st.user_req[r]).all()
        assert (st.user_app_tok[r].sum(1) == st.user_tok[r]).all()
        active = int((st.user_req[r] > 0).sum())
        assert st.rate_hist[r, A, 0].sum() == st.rate_hist[r, A, 1].sum() == active
        for a in range(A):
            assert st.rate_hist[r, a, 0].sum() == int((st.user_app_req[r, :, a] > 0).sum())
        assert (st.len_hist[r].sum(axis=(0, 2)) == n).all()
        assert st.graph[r, :, 1].sum() == n and st.graph[r, :, 0].sum() == st.size_hist[r].sum()
        sizes = np.arange(1, 65)
        assert (st.size_hist[r][:, :63] * sizes[:63]).sum() + 0 <= n
        # the graph rows of sizes 1..63 are sums of the size histogram
        for b, (lo, hi) in enumerate(((1, 1), (2, 10), (11, 20), (21, 30), (31, 40), (41, 50))):
            assert st.graph[r, b, 0] == st.size_hist[r][:, lo - 1:hi].sum()
        assert st.graph[r, :, 2].sum() == st.len_sum[r, :, 0].sum()
        assert st.graph[r, :, 3].sum() == st.len_sum[r, :, 2].sum()
        assert st.graph[r, :, 4].sum() == st.len_sum[r, :, 1].sum()


def test_table2_request_shares_from_the_large_tenant_generator():
    """The large-tenant recipe draws interaction sizes so that the share of requests in
    interactions of 1, 2-10 and 11-20 calls follows Table 2 (73.22 %, 26.09 %, 0.50 %,
    renormalised over those rows); the analysis recovers them from 400k requests."""
    wl = tg.scaled(tg.WORKLOADS["c5_tenant"], records=400_000, users=20_000)
    tr = tg.generate(wl)
    st = oracle.workload_stats(tr)
    share = st.graph[0, :, 1] / tr.n * 100.0
    tot = 73.22 + 26.09 + 0.50
    assert abs(share[0] - 100 * 73.22 / tot) < 0.6
    assert abs(share[1] - 100 * 26.09 / tot) < 0.6
    assert abs(share[2] - 100 * 0.50 / tot) < 0.15
    assert share[3:].sum() == 0


def test_errors():
    tr = Trace(1, 2, 1, np.array([0, 2], np.int64), np.array([1, 2], np.int64),
               np.array([0, 2], np.int32), np.zeros(2, np.int32), None, None, None,
               np.ones(2, np.int32), None, np.ones(2, np.int32))
    with pytest.raises(oracle.OracleError) as e:
        oracle.workload_stats(tr)
    assert e.value.code == oracle.E_RANGE
    with pytest.raises(oracle.OracleError) as e:
        oracle.workload_stats(Trace(**{**tr.__dict__, "user": np.zeros(2, np.int32)}), 0)
    assert e.value.code == oracle.E_ARG

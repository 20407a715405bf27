"""Pins for the CPU oracle: checks against what the paper and the mathematics fix.

- hand-worked schedules, window counts and costs (tests/golden, each cited);
- the paper's worked example of application-normalised service (Sec. 3);
- closed forms: a single user is served FIFO with counters equal to prefix
  sums of cost; with everything queued at once and single calls, the order is
  the weighted-fair-queueing start-tag merge;
- invariances: with equal weights for all apps the schedule ignores app labels;
- brute force: the naive model (tests/naive_model.py) on exhaustive and random
  tiny traces;
- Jain's index special cases; the paper's invariants (oracle check mode).
"""
import itertools

import numpy as np
import pytest

import oracle
import naive_model as nm
from tiny import load_golden, random_trace, trace_from_case
import tracegen as tg
from tracegen import Trace, concat

# ---------------------------------------------------------------- golden cases


@pytest.mark.parametrize("case", load_golden("hand_traces.json")["cases"], ids=lambda c: c["name"])
def test_hand_traces(case):
    tr = trace_from_case(case)
    cost = np.asarray(case["cost"], np.int64)
    reason = np.asarray(case["reason"], np.uint8)
    res = oracle.simulate(tr, cost, reason, case["tau"], case["C"], case["theta"], check=True)
    for key in ("status", "admit_step", "admit_seq", "counter_after", "counter_on_arrival",
                "counter"):
        assert res.__dict__[key].tolist() == case[key], key
    assert int(res.steps[0]) == case["steps"]
    assert int(res.decisions[0]) == case["decisions"]
    assert int(res.max_gap[0]) == case["max_gap"]
    # the brute-force model agrees on the same hand case
    nres = nm.simulate(tr, cost, reason, case["tau"], case["C"], case["theta"])
    assert nres.status == case["status"] and nres.counter_after == case["counter_after"]


def test_window_counts_golden():
    g = load_golden("window_counts.json")
    n = len(g["ts"])
    tr = Trace(1, g["U"], g["A"], np.array([0, n], np.int64), np.asarray(g["ts"], np.int64),
               np.asarray(g["user"], np.int32), np.asarray(g["app"], np.int32),
               None, None, None, None, None, None)
    res = oracle.throttle(tr, g["W"], g["t_user"], g["t_app"], raw=True)
    assert res.cnt_user.tolist() == g["cnt_user"]
    assert res.cnt_app.tolist() == g["cnt_app"]
    assert res.reason.tolist() == g["raw"]
    gated = oracle.throttle(tr, g["W"], g["t_user"], g["t_app"], overloaded=g["overloaded"],
                            raw=False)
    assert gated.reason.tolist() == g["gated"]
    bits = [(int(gated.bitmap[i // 32]) >> (i % 32)) & 1 for i in range(n)]
    assert bits == [int(x != 0) for x in g["gated"]]


@pytest.mark.parametrize("case", load_golden("cost_cases.json")["cases"])
def test_cost_golden(case):
    tr = Trace(1, 1, 1, np.array([0, 1], np.int64), np.zeros(1, np.int64), np.zeros(1, np.int32),
               np.zeros(1, np.int32), None, None, None, np.array([case["L"][0]], np.int32),
               np.array([case["L"][1]], np.int32), np.array([case["L"][2]], np.int32))
    coef = np.asarray(case["coef"], np.int64).reshape(1, 1, 1, 3)
    prio = np.array([[case["E"]]], np.int32)
    if case["cost"] == "overflow":
        with pytest.raises(oracle.OracleError) as e:
            oracle.cost(tr, coef, prio=prio)
        assert e.value.code == oracle.E_OVERFLOW
    else:
        assert oracle.cost(tr, coef, prio=prio).tolist() == [case["cost"]]


# ------------------------------------------------- the paper's worked example


def test_worked_example_application_normalised_service():
    """Sec. 3: apps A and B with mean request lengths 10 and 50; after 5 tokens each,
    users of A and B have received 50 % and 10 % of their service, so B's user is
    the less served and is picked next."""
    K = 1024
    coef = oracle.coef_from_expectations(np.array([[10.0], [50.0]]), np.zeros((2, 1)),
                                         np.zeros((2, 1)), K)
    tr = Trace(1, 2, 2, np.array([0, 2], np.int64), np.array([0, 0], np.int64),
               np.array([0, 1], np.int32), np.array([0, 1], np.int32), None, None, None,
               np.array([5, 5], np.int32), None, np.array([0, 0], np.int32))
    c = oracle.cost(tr, coef[None])
    frac = c / float(1 << 16) / K
    assert abs(frac[0] - 0.5) <= 5 * 2.0 ** -16 and abs(frac[1] - 0.1) <= 5 * 2.0 ** -16
    # both users keep a second request queued (so no lift evens them out): after one
    # request each, B's user has the smaller counter and is served first
    tr2 = Trace(1, 2, 2, np.array([0, 4], np.int64), np.array([0, 0, 0, 0], np.int64),
                np.array([0, 1, 0, 1], np.int32), np.array([0, 1, 0, 1], np.int32), None, None,
                None, np.array([5, 5, 5, 5], np.int32), None, np.zeros(4, np.int32))
    c2 = oracle.cost(tr2, coef[None])
    res = oracle.simulate(tr2, c2, None, 10, 10, 10 ** 9, check=True)
    # step 0 serves both (10 tokens of budget); at step 1 user 1 (app B) has the smaller counter
    assert res.admit_step.tolist() == [0, 0, 1, 1]
    assert res.admit_seq[3] < res.admit_seq[2]


def test_eq1_weights_and_class_factors():
    """Eq. 1 with alpha, beta, gamma = 1, 2, 1: system tokens cost twice input tokens,
    and the coefficient scales as 1 / w_aj."""
    e_in = np.array([[100.0, 30.0]])
    e_sys = np.array([[50.0, 0.0]])
    e_out = np.array([[20.0, 10.0]])
    c = oracle.coef_from_expectations(e_in, e_sys, e_out, 1024)
    w = np.array([100 + 2 * 50 + 20, 30 + 0 + 10], float)
    for j in range(2):
        assert abs(c[0, j, 0] - 2 ** 26 / w[j]) <= 0.5
        assert abs(c[0, j, 1] - 2 * 2 ** 26 / w[j]) <= 0.5
        assert c[0, j, 0] == c[0, j, 2]
    with pytest.raises(oracle.OracleError):
        oracle.coef_from_expectations(np.zeros((1, 1)), np.zeros((1, 1)), np.zeros((1, 1)))


# -------------------------------------------------------------- closed forms


def test_single_user_fifo_prefix_sums():
    rng = np.random.default_rng(1)
    for _ in range(20):
        n = int(rng.integers(1, 60))
        ts = np.sort(rng.integers(0, 500, n)).astype(np.int64)
        tok = rng.integers(1, 9, n).astype(np.int32)
        cost = rng.integers(0, 1000, n).astype(np.int64)
        tr = Trace(1, 1, 1, np.array([0, n], np.int64), ts, np.zeros(n, np.int32),
                   np.zeros(n, np.int32), None, None, None, tok, None, np.zeros(n, np.int32))
        res = oracle.simulate(tr, cost, None, 10, int(rng.integers(1, 12)), 10 ** 9, check=True)
        assert res.admit_seq.tolist() == list(range(n))          # FIFO
        assert res.counter_after.tolist() == np.cumsum(cost).tolist()
        assert int(res.counter[0]) == int(cost.sum())
        assert (res.status == 0).all()


def test_wfq_start_tag_merge():
    """All single-call requests queued in step 0 and no later arrivals: the
    admission order is the merge of each user's start tags u_k + sum of its earlier
    costs, ties to the lower user id (weighted fair queueing)."""
    rng = np.random.default_rng(2)
    for _ in range(30):
        U = int(rng.integers(1, 6))
        n = int(rng.integers(1, 40))
        user = rng.integers(0, U, n).astype(np.int32)
        cost = rng.integers(1, 50, n).astype(np.int64)
        tok = rng.integers(1, 5, n).astype(np.int32)
        tr = Trace(1, U, 1, np.array([0, n], np.int64), np.zeros(n, np.int64), user,
                   np.zeros(n, np.int32), None, None, None, tok, None, np.zeros(n, np.int32))
        res = oracle.simulate(tr, cost, None, 10, int(rng.integers(1, 10)), 10 ** 9, check=True)
        tags = []
        acc = {}
        for i in range(n):       # every counter starts at 0 and every lift is to 0
            k = int(user[i])
            tags.append((acc.get(k, 0), k, i))
            acc[k] = acc.get(k, 0) + int(cost[i])
        expected = [i for (_, _, i) in sorted(tags)]
        assert np.argsort(res.admit_seq).tolist() == expected


def test_equal_weights_ignore_app_labels():
    """With the same coefficients for every app the charge depends on tokens only,
    so relabelling apps changes nothing (the VTC special case of WSC)."""
    rng = np.random.default_rng(3)
    for _ in range(10):
        tr = random_trace(rng, 80, 4, 3, 400, multi=True)
        coef = np.tile(np.array([3 << 16, 5 << 16, 7 << 16], np.int64), (1, 3, 1, 1))
        c1 = oracle.cost(tr, coef)
        perm = rng.permutation(3).astype(np.int32)
        tr2 = Trace(**{**tr.__dict__, "app": perm[tr.app]})
        c2 = oracle.cost(tr2, coef)
        assert (c1 == c2).all()
        r1 = oracle.simulate(tr, c1, None, 25, 9, 10 ** 9, check=True)
        r2 = oracle.simulate(tr2, c2, None, 25, 9, 10 ** 9, check=True)
        assert (r1.admit_seq == r2.admit_seq).all() and (r1.counter == r2.counter).all()


def test_sliding_window_infinite_window_is_rank_limit():
    """W beyond the trace span: a request exceeds a limit T iff its rank within
    its key (counting itself) exceeds T."""
    rng = np.random.default_rng(4)
    tr = random_trace(rng, 300, 5, 3, 1000, multi=False)
    res = oracle.throttle(tr, 10 ** 9, 7, [3, 4, 5], raw=True)
    ru, ra = {}, {}
    for i in range(tr.n):
        k = int(tr.user[i]); a = int(tr.app[i])
        ru[k] = ru.get(k, 0) + 1
        ra[(k, a)] = ra.get((k, a), 0) + 1
        want = 1 if ru[k] > 7 else (2 if ra[(k, a)] > [3, 4, 5][a] else 0)
        assert res.reason[i] == want


# --------------------------------------------------------------- brute force


def _run_both(tr, step_us, C, theta, W, t_user, t_app, coef, overloaded=None, flags=0):
    c = oracle.cost(tr, coef)
    assert c.tolist() == nm.cost(tr, coef)
    th = oracle.throttle(tr, W, t_user, t_app, raw=True)
    cu, ca = nm.window_counts(tr, W)
    assert th.cnt_user.tolist() == cu and th.cnt_app.tolist() == ca
    assert th.reason.tolist() == nm.throttle_raw(tr, W, t_user, t_app)
    gated = oracle.throttle(tr, W, t_user, t_app, overloaded=overloaded, raw=False)
    assert gated.reason.tolist() == nm.throttle_gated(tr, W, t_user, t_app, overloaded)
    r = oracle.simulate(tr, c, th.reason, step_us, C, theta, check=True, flags=flags)
    n = nm.simulate(tr, c, th.reason, step_us, C, theta, flags=flags)
    for key in ("status", "admit_step", "admit_seq", "counter_after", "counter_on_arrival",
                "counter", "steps", "decisions", "max_gap"):
        assert getattr(r, key).tolist() == getattr(n, key), key
    return r


# the default policy, first-come first-served order, interaction-blind limits, and both
# (with overload_tokens = -1 the latter is the request-rate-limit policy); then the
# literal engine under the default policy and under the rate-limit policy
POLICY_FLAGS = (0, oracle.FSO_FCFS, oracle.FSO_BLIND, oracle.FSO_FCFS | oracle.FSO_BLIND,
                oracle.FSO_LITERAL, oracle.FSO_LITERAL | oracle.FSO_FCFS | oracle.FSO_BLIND)


def test_naive_equals_oracle_exhaustive_tiny():
    """Every 3-request trace over 2 users, arrival steps {0,1}, tokens {1,3},
    first-call limits hit or not, chained or not, at two overload thresholds."""
    coef = np.array([[[[1 << 16, 0, 1 << 16]]]], np.int64)
    count = 0
    for users in itertools.product(range(2), repeat=3):
        for steps in itertools.product(range(2), repeat=3):
            if list(steps) != sorted(steps):
                continue
            for toks in itertools.product((1, 3), repeat=3):
                for link in (False, True):
                    n = 3
                    call = np.zeros(n, np.int32); head = np.arange(n, dtype=np.int32)
                    prev = np.full(n, -1, np.int32)
                    if link and users[2] == users[0]:
                        call[2], head[2], prev[2] = 1, 0, 0
                    elif link:
                        continue
                    tr = Trace(1, 2, 1, np.array([0, n], np.int64),
                               np.asarray(steps, np.int64) * 10, np.asarray(users, np.int32),
                               np.zeros(n, np.int32), call, head, prev,
                               np.asarray(toks, np.int32), None, np.zeros(n, np.int32))
                    for theta in (-1, 1):
                        for flags in POLICY_FLAGS:
                            # T_app = 0 makes every first call exceed; T_user = 1 flags repeats
                            _run_both(tr, 10, 2, theta, 15, 1, [0], coef, flags=flags)
                            count += 1
    assert count > 100


def test_naive_equals_oracle_literal_engine_exhaustive():
    """The literal engine on every 3-request trace over 2 users, arrival steps {0,1},
    input tokens {1,3}, output tokens {0,2}, chained or not, at two KV capacities."""
    coef = np.array([[[[1 << 16, 0, 3 << 16]]]], np.int64)
    count = 0
    for users in itertools.product(range(2), repeat=3):
        for steps in itertools.product(range(2), repeat=3):
            if list(steps) != sorted(steps):
                continue
            for toks in itertools.product((1, 3), repeat=3):
                for outs in itertools.product((0, 2), repeat=3):
                    for link in (False, True):
                        n = 3
                        call = np.zeros(n, np.int32); head = np.arange(n, dtype=np.int32)
                        prev = np.full(n, -1, np.int32)
                        if link and users[2] == users[0]:
                            call[2], head[2], prev[2] = 1, 0, 0
                        elif link:
                            continue
                        tr = Trace(1, 2, 1, np.array([0, n], np.int64),
                                   np.asarray(steps, np.int64) * 10, np.asarray(users, np.int32),
                                   np.zeros(n, np.int32), call, head, prev,
                                   np.asarray(toks, np.int32), None, np.asarray(outs, np.int32))
                        for kv in (4, 7):
                            for flags in (oracle.FSO_LITERAL, oracle.FSO_LITERAL | oracle.FSO_FCFS):
                                _run_both(tr, 10, kv, 1, 15, 1, [0], coef, flags=flags)
                                count += 1
    assert count > 500


def test_literal_engine_closed_forms():
    """Charge at finish (Alg. 1, execution stream): counters do not move between a step's
    admissions, so the least-served user's whole queue goes first; a call holds its KV
    tokens until its last output token; an oversized call runs alone."""
    L = oracle.FSO_LITERAL
    coef = np.array([[[[1 << 16, 0, 1 << 16]]]], np.int64)
    # two users, three one-token requests each, all at step 0, ample KV
    n = 6
    users = np.array([0, 1, 0, 1, 0, 1], np.int32)
    tr = Trace(1, 2, 1, np.array([0, n], np.int64), np.zeros(n, np.int64), users,
               np.zeros(n, np.int32), None, None, None, np.ones(n, np.int32), None,
               np.zeros(n, np.int32))
    c = oracle.cost(tr, coef)
    lit = oracle.simulate(tr, c, None, 10, 100, 10 ** 9, check=True, flags=L)
    assert lit.admit_seq.tolist() == [0, 3, 1, 4, 2, 5]     # user 0's queue, then user 1's
    assert lit.counter.tolist() == [3 << 16, 3 << 16]
    eager = oracle.simulate(tr, c, None, 10, 100, 10 ** 9, check=True)
    assert eager.admit_seq.tolist() == [0, 1, 2, 3, 4, 5]   # charged at admission: alternate
    # one user, calls of 1 input + L_O output tokens, KV for one call at a time
    outs = np.array([3, 1, 2, 5], np.int32)
    n = 4
    tr = Trace(1, 1, 1, np.array([0, n], np.int64), np.zeros(n, np.int64), np.zeros(n, np.int32),
               np.zeros(n, np.int32), None, None, None, np.ones(n, np.int32), None, outs)
    c = oracle.cost(tr, coef)
    # KV of 1 token: every call is oversized and runs alone, starting the step after the
    # previous one decoded its last token
    r = oracle.simulate(tr, c, None, 10, 1, 10 ** 9, check=True, flags=L)
    assert r.admit_step.tolist() == [0, 3, 4, 6]
    assert r.counter_after.tolist() == np.cumsum(c).tolist()
    assert r.steps.tolist() == [11]                          # the last call decodes in step 10
    # KV of 6 (footprints 4, 2, 3, 6): calls 0 and 1 fit at step 0; call 1 finishes in
    # step 0 and call 0 in step 2, so call 2 waits for step 3, call 3 for call 2's finish
    r = oracle.simulate(tr, c, None, 10, 6, 10 ** 9, check=True, flags=L)
    assert r.admit_step.tolist() == [0, 0, 3, 5]
    assert r.counter_after.tolist() == [c[1] + c[0], c[1], c[0] + c[1] + c[2], int(np.sum(c))]
    assert r.steps.tolist() == [10]
    # an oversized call (10 tokens > KV 5) runs when nothing else does
    tr2 = Trace(1, 1, 1, np.array([0, 3], np.int64), np.zeros(3, np.int64), np.zeros(3, np.int32),
                np.zeros(3, np.int32), None, None, None, np.array([1, 8, 1], np.int32), None,
                np.array([1, 2, 1], np.int32))
    c2 = oracle.cost(tr2, coef)
    r2 = oracle.simulate(tr2, c2, None, 10, 5, 10 ** 9, check=True, flags=L)
    assert r2.admit_step.tolist() == [0, 1, 3]


@pytest.mark.parametrize("seed", range(6))
def test_naive_equals_oracle_random(seed):
    rng = np.random.default_rng(100 + seed)
    for _ in range(40):
        U = int(rng.integers(1, 4)); A = int(rng.integers(1, 3))
        n = int(rng.integers(1, 25))
        tr = random_trace(rng, n, U, A, int(rng.integers(1, 120)), multi=bool(rng.integers(0, 2)))
        coef = rng.integers(0, 4, size=(1, A, 1, 3)).astype(np.int64) << 14
        ov = rng.integers(0, 2, size=n).astype(np.uint8)
        _run_both(tr, int(rng.integers(1, 30)), int(rng.integers(1, 12)),
                  int(rng.integers(-1, 10)), int(rng.integers(1, 60)), int(rng.integers(0, 4)),
                  rng.integers(0, 4, size=A).tolist(), coef, overloaded=ov,
                  flags=POLICY_FLAGS[seed % len(POLICY_FLAGS)])


def test_naive_equals_oracle_small_workload():
    """The first small workload's recipe at 400 requests (the naive model is quadratic)."""
    wl = tg.scaled(tg.WORKLOADS["c1_small"], records=400)
    tr = tg.generate(wl)
    coef, _ = oracle.weights_for(wl, tr)
    _run_both(tr, wl.step_us, wl.cap_tokens, wl.overload_tokens, wl.window_us, wl.t_user,
              wl.t_app, coef)


@pytest.mark.parametrize("seed", range(4))
def test_app_level_limit_brute_force(seed):
    """The app limit counted per application over all users (the app-level rate limit),
    against counts by brute force over all earlier requests."""
    rng = np.random.default_rng(40 + seed)
    for _ in range(25):
        A = int(rng.integers(1, 4))
        tr = random_trace(rng, int(rng.integers(1, 60)), int(rng.integers(1, 5)), A,
                          int(rng.integers(1, 200)), multi=bool(seed % 2))
        W, tu = int(rng.integers(1, 80)), int(rng.integers(0, 6))
        ta = rng.integers(0, 6, size=A).tolist()
        th = oracle.throttle(tr, W, tu, ta, raw=True, app_scope=1)
        cu, ca = nm.window_counts(tr, W, app_scope=1)
        assert th.cnt_user.tolist() == cu and th.cnt_app.tolist() == ca
        assert th.reason.tolist() == nm.throttle_raw(tr, W, tu, ta, app_scope=1)
        # with one user the two scopes agree
        if tr.n_users == 1:
            th0 = oracle.throttle(tr, W, tu, ta, raw=True)
            assert th0.reason.tolist() == th.reason.tolist()


def test_fcfs_serves_in_arrival_order():
    """First come, first served without throttling: every request is admitted and the
    admission sequence is the stream order (closed form), whatever the counters say."""
    rng = np.random.default_rng(31)
    for _ in range(20):
        tr = random_trace(rng, int(rng.integers(5, 80)), int(rng.integers(1, 6)), 2,
                          int(rng.integers(1, 400)), multi=True)
        c = rng.integers(0, 1000, tr.n).astype(np.int64)
        r = oracle.simulate(tr, c, None, int(rng.integers(1, 40)), int(rng.integers(1, 10)),
                            10 ** 9, check=True, flags=oracle.FSO_FCFS)
        assert (r.status == 0).all()
        assert r.admit_seq.tolist() == list(range(tr.n))
        assert (np.diff(r.admit_step) >= 0).all()


def _rate_limit_fates(tr, raw):
    """Interaction-blind limits, always on: a call over a limit is dropped with its
    reason, and every later call of an interaction with a dropped call is dropped (3)."""
    out = np.zeros(tr.n, np.int8)
    for g in range(tr.n):
        if tr.call is not None and tr.call[g] > 0 and out[int(tr.prev[g])] != 0:
            out[g] = 3
        else:
            out[g] = raw[g]
    return out


def test_rate_limit_policy_fates_closed_form():
    rng = np.random.default_rng(32)
    for _ in range(30):
        tr = random_trace(rng, int(rng.integers(5, 90)), int(rng.integers(1, 5)), 2,
                          int(rng.integers(1, 300)), multi=True)
        W, tu, ta = int(rng.integers(1, 100)), int(rng.integers(0, 5)), [2, 3]
        raw = oracle.throttle(tr, W, tu, ta, raw=True).reason
        c = np.ones(tr.n, np.int64)
        for flags in (oracle.FSO_BLIND, oracle.FSO_FCFS | oracle.FSO_BLIND):
            r = oracle.simulate(tr, c, raw, 10, 4, -1, check=True, flags=flags)
            assert r.status.tolist() == _rate_limit_fates(tr, raw).tolist()


def test_rate_limit_policy_aborts_interactions_midway():
    """An interaction whose second call goes over the user limit: interaction-blind
    limits serve its first call and drop the second (an interaction aborted midway,
    its served tokens wasted); the paper's policy exempts the second call."""
    # user 0: interaction A = (call 0 at t=0, call 1 at t=10), a single request at t=1
    tr = Trace(1, 1, 1, np.array([0, 3], np.int64), np.array([0, 1, 10], np.int64),
               np.zeros(3, np.int32), np.zeros(3, np.int32), np.array([0, 0, 1], np.int32),
               np.array([0, 1, 0], np.int32), np.array([-1, -1, 0], np.int32),
               np.array([4, 2, 3], np.int32), None, np.zeros(3, np.int32))
    raw = oracle.throttle(tr, 100, 1, [100], raw=True).reason
    assert raw.tolist() == [0, 1, 1]
    c = np.array([5, 5, 5], np.int64)
    rpm = oracle.simulate(tr, c, raw, 10, 100, -1, flags=oracle.FSO_FCFS | oracle.FSO_BLIND)
    fs = oracle.simulate(tr, c, raw, 10, 100, -1)
    assert rpm.status.tolist() == [0, 1, 1] and fs.status.tolist() == [0, 1, 0]
    m_rpm = oracle.fairness_metrics(tr, c, rpm.status, rpm.admit_step, rpm.max_gap, 10)
    m_fs = oracle.fairness_metrics(tr, c, fs.status, fs.admit_step, fs.max_gap, 10)
    assert m_rpm.aborted_midway[0] == 1 and m_rpm.wasted_tokens[0] == 4
    assert m_fs.aborted_midway[0] == 0 and m_fs.wasted_tokens[0] == 0


def test_bounded_runs_are_prefixes():
    """Simulating s steps gives exactly the decisions of the first s steps of a full run."""
    rng = np.random.default_rng(5)
    tr = random_trace(rng, 120, 4, 2, 300, multi=True)
    c = oracle.cost(tr, np.full((1, 2, 1, 3), 1 << 15, np.int64))
    full = oracle.simulate(tr, c, None, 10, 4, 6, check=True)
    for s in (0, 1, 5, 17, int(full.steps[0])):
        part = oracle.simulate(tr, c, None, 10, 4, 6, max_steps=s)
        in_prefix = (full.admit_step >= 0) & (full.admit_step < s)
        assert ((part.admit_step >= 0) == in_prefix).all()
        assert (part.admit_seq[in_prefix] == full.admit_seq[in_prefix]).all()
        assert (part.counter_after[in_prefix] == full.counter_after[in_prefix]).all()
        assert int(part.decisions[0]) == int(in_prefix.sum())


# --------------------------------------------------------------- invariants


def test_bounded_gap_between_continuously_backlogged_users():
    """Single-call traces: for users f, g continuously backlogged since t0,
    u_f - u_g <= max(u_f(t0) - u_g(t0), c_max)."""
    rng = np.random.default_rng(6)
    for _ in range(15):
        tr = random_trace(rng, 60, 4, 1, 150, multi=False, max_tok=4)
        c = rng.integers(0, 40, tr.n).astype(np.int64)
        res = nm.simulate(tr, c, None, 10, 3, 10 ** 9, record_states=True)
        cmax = int(c.max())
        states = res.trace_of_counters
        for a in range(len(states)):
            for b in range(a, len(states)):
                sa, sb = states[a][2], states[b][2]
                common = set(sa) & set(sb)
                # continuously backlogged: present in every state between a and b
                for st in states[a:b + 1]:
                    common &= set(st[2])
                for f in common:
                    for g in common:
                        assert sb[f] - sb[g] <= max(sa[f] - sa[g], cmax)


def test_invariants_on_workload_recipes():
    """Oracle check mode (throttled only while overloaded, counters monotone, every
    unthrottled request served once, queue fronts are first calls) on scaled recipes."""
    for name in ("c1_small", "c2_replicas", "c4_sweep", "c5_tenant"):
        wl = tg.scaled(tg.WORKLOADS[name], replicas=min(2, tg.WORKLOADS[name].n_replicas),
                       records=5000)
        tr = tg.generate(wl)
        c, th, sim, met = oracle.run_workload(wl, tr, check=True)
        assert (met.aborted_midway == 0).all() and (met.wasted_tokens == 0).all()
        assert ((sim.status >= 0) & (sim.status <= 3)).all()


def test_jain_special_cases():
    n = 4
    tr = Trace(1, n, 1, np.array([0, n], np.int64), np.zeros(n, np.int64),
               np.arange(n, dtype=np.int32), np.zeros(n, np.int32), None, None, None,
               np.ones(n, np.int32), None, np.zeros(n, np.int32))
    st = np.zeros(n, np.int8); adm = np.zeros(n, np.int32)
    eq = oracle.fairness_metrics(tr, np.full(n, 7, np.int64), st, adm, None, 10)
    assert eq.jain[0] == 1.0
    one = oracle.fairness_metrics(tr, np.array([9, 0, 0, 0], np.int64), st, adm, None, 10)
    assert abs(one.jain[0] - 1.0 / n) < 1e-15
    two = oracle.fairness_metrics(tr, np.array([1, 3, 0, 0], np.int64), st, adm, None, 10)
    assert abs(two.jain[0] - 16.0 / (4 * 10)) < 1e-15


def test_jain_near_the_charged_service_limit():
    """Costs near 2^62: the replica's total charged service decides.  Below 2^62 the sums
    are exact (Jain's index of equal shares is 1, of a 3:1 split 0.8 by hand); at 2^62 or
    more the call reports an overflow instead of a wrapped sum; an admitted cost outside
    [0, 2^62) is a range error."""
    n = 4
    tr = Trace(1, n, 1, np.array([0, n], np.int64), np.zeros(n, np.int64),
               np.array([0, 1, 2, 3], np.int32), np.zeros(n, np.int32), None, None, None,
               np.ones(n, np.int32), None, np.zeros(n, np.int32))
    st = np.zeros(n, np.int8); adm = np.zeros(n, np.int32)
    q = 1 << 60
    eq = oracle.fairness_metrics(tr, np.array([q - 1] * 4, np.int64), st, adm, None, 10)
    assert eq.jain[0] == 1.0
    # two users share 2^62 - 1 as 3:1 (the other two are dropped): J = 4^2 / (4 * 10) * ...
    st2 = np.array([0, 0, 1, 1], np.int8)
    x, y = 3 * q - 1, q - 1        # total 2^62 - 2
    m = oracle.fairness_metrics(tr, np.array([x, y, 5, 5], np.int64), st2, adm, None, 10)
    want = float(x + y) ** 2 / (4.0 * (float(x) ** 2 + float(y) ** 2))
    assert abs(m.jain[0] - want) < 1e-15 and abs(want - 16.0 / 40.0) < 1e-12
    with pytest.raises(oracle.OracleError) as e:    # total exactly 2^62
        oracle.fairness_metrics(tr, np.array([q] * 4, np.int64), st, adm, None, 10)
    assert e.value.code == oracle.E_OVERFLOW
    big = (1 << 62) - 1                              # four of them would wrap 64 bits
    with pytest.raises(oracle.OracleError) as e:
        oracle.fairness_metrics(tr, np.array([big] * 4, np.int64), st, adm, None, 10)
    assert e.value.code == oracle.E_OVERFLOW
    with pytest.raises(oracle.OracleError) as e:     # an admitted cost out of range
        oracle.fairness_metrics(tr, np.array([1, -1, 1, 1], np.int64), st, adm, None, 10)
    assert e.value.code == oracle.E_RANGE


def test_served_experience_metrics_by_hand():
    # two interactions of user 0 (one throttled), one of user 1 served late
    tr = Trace(1, 2, 1, np.array([0, 4], np.int64), np.array([0, 0, 5, 20], np.int64),
               np.array([0, 0, 0, 1], np.int32), np.zeros(4, np.int32),
               np.array([0, 0, 1, 0], np.int32), np.array([0, 1, 0, 3], np.int32),
               np.array([-1, -1, 0, -1], np.int32), np.array([2, 2, 2, 2], np.int32), None,
               np.zeros(4, np.int32))
    status = np.array([0, 1, 0, 0], np.int8)
    adm = np.array([0, -1, 0, 4], np.int32)
    m = oracle.fairness_metrics(tr, np.array([5, 5, 5, 5], np.int64), status, adm,
                                np.array([3 << 16]), 10, delay_steps=1)
    assert m.svc_req_pct[0] == 75.0 and abs(m.svc_int_pct[0] - 200.0 / 3) < 1e-12
    assert m.served_users_pct[0] == 100.0 and m.delayed_users_pct[0] == 50.0
    assert m.throttled[0] == 1 and m.aborted_midway[0] == 0 and m.wasted_tokens[0] == 0
    assert m.max_gap_tokens[0] == 3.0
    # an interaction served halfway wastes its served tokens
    status2 = np.array([0, 0, 3, 0], np.int8)
    m2 = oracle.fairness_metrics(tr, np.full(4, 5, np.int64), status2, adm, None, 10)
    assert m2.aborted_midway[0] == 1 and m2.wasted_tokens[0] == 2


# --------------------------------------------------------------- errors


def test_error_codes():
    tr = Trace(1, 2, 1, np.array([0, 2], np.int64), np.array([5, 4], np.int64),
               np.array([0, 1], np.int32), np.zeros(2, np.int32), None, None, None,
               np.ones(2, np.int32), None, np.ones(2, np.int32))
    with pytest.raises(oracle.OracleError) as e:
        oracle.throttle(tr, 10, 1, [1])
    assert e.value.code == oracle.E_ORDER
    tr2 = Trace(**{**tr.__dict__, "ts_us": np.array([4, 5], np.int64),
                   "user": np.array([0, 2], np.int32)})
    with pytest.raises(oracle.OracleError) as e:
        oracle.throttle(tr2, 10, 1, [1])
    assert e.value.code == oracle.E_RANGE
    tr3 = Trace(**{**tr.__dict__, "ts_us": np.array([4, 5], np.int64)})
    with pytest.raises(oracle.OracleError) as e:
        oracle.simulate(tr3, np.array([1, -1], np.int64), None, 10, 5, 5)
    assert e.value.code == oracle.E_RANGE
    with pytest.raises(oracle.OracleError) as e:
        oracle.simulate(tr3, np.array([1, 1 << 61], np.int64) * np.array([1, 2]), None, 10, 5, 5)
    assert e.value.code == oracle.E_RANGE
    tr4 = Trace(**{**tr3.__dict__, "user": np.array([0, 0], np.int32)})
    with pytest.raises(oracle.OracleError) as e:
        oracle.simulate(tr4, np.array([(1 << 62) - 1, 1], np.int64), None, 10, 5, 5)
    assert e.value.code == oracle.E_OVERFLOW
    oracle.simulate(tr4, np.array([(1 << 62) - 2, 1], np.int64), None, 10, 5, 5)


def test_generator_is_seeded_and_shaped():
    wl = tg.WORKLOADS["c1_small"]
    a, b = tg.generate(wl), tg.generate(wl)
    assert a.sha256() == b.sha256()
    assert a.n == 2000 and (np.diff(a.ts_us) >= 0).all() and a.ts_us.max() < 60_000_000
    frac7 = (a.user == 7).mean()
    assert 0.8 < frac7 < 0.9       # user 7 draws 20 / (20 + 7 * 0.5) = 0.85 of the requests
    wl2 = tg.scaled(tg.WORKLOADS["c2_replicas"], replicas=2, records=3000)
    t2 = tg.generate(wl2)
    assert t2.n == 6000 and t2.call.max() <= 19
    for r in range(2):
        s = t2.replica(r)
        i = np.arange(s.n)
        later = s.call > 0
        assert (s.prev[later] < i[later]).all() and (s.user[s.prev[later]] == s.user[later]).all()
        assert (s.head[~later] == i[~later]).all()

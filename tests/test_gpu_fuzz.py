"""Randomised parity sweep: small random traces (several replicas, multi-call
interactions, random limits, capacities and overload thresholds) through the raw
throttle and the scheduler in every engine and policy mode, on the on-chip path, the
global-memory path and in resumed chunks of steps, bit-exact against the oracle."""
import numpy as np
import pytest

import oracle
from gpu_common import compare_sim, gpu_schedule, gpu_throttle, say
from tiny import random_trace
import tracegen as tg

pytestmark = pytest.mark.gpu


def _case(seed):
    rng = np.random.default_rng(1000 + seed)
    R = int(rng.integers(1, 7))
    U = int(rng.choice([1, 3, 17, 64, 65, 200]))
    A = int(rng.integers(1, 5))
    multi = bool(rng.integers(0, 2))  # (interaction links are all set or all absent)
    reps = []
    for _ in range(R):
        n = int(rng.choice([0, 1, 50, 700, 2500, 8000]))
        span = int(rng.integers(1, 4 * max(n, 1) * 10))
        reps.append(random_trace(rng, n, U, A, span, multi=multi, max_tok=int(rng.integers(1, 40))))
    tr = tg.concat(reps)
    W = int(rng.integers(1, 2000))
    t_user = int(rng.choice([0, 3, 20, 2 ** 31 - 1]))
    t_app = [int(x) for x in rng.integers(0, 15, A)]
    step = int(rng.integers(1, 200))
    literal = bool(rng.integers(0, 3) == 0)
    cap = int(rng.integers(1, 300)) if not literal else int(rng.integers(40, 2000))
    theta = int(rng.choice([-1, 0, 50, 10 ** 9]))
    fcfs, blind = bool(rng.integers(0, 2)), bool(rng.integers(0, 2))
    mode = int(rng.integers(0, 3))  # 0 on chip, 1 global memory only, 2 in chunks of steps
    cost = rng.integers(0, 5000, tr.n).astype(np.int64)
    return tr, W, t_user, t_app, step, literal, cap, theta, fcfs, blind, mode, cost, rng


@pytest.mark.parametrize("seed", range(300))
def test_random_throttle_and_schedule(seed):
    tr, W, t_user, t_app, step, literal, cap, theta, fcfs, blind, mode, cost, rng = _case(seed)
    say("fuzz", seed, tr.n_replicas, tr.n_users, tr.n, literal, fcfs, blind, mode)
    o_th = oracle.throttle(tr, W, t_user, t_app, raw=True, counts=False)
    g_th = gpu_throttle(tr, W, t_user, t_app, raw=True, counts=False)
    assert (g_th["reason"] == o_th.reason).all()
    flags = ((oracle.FSO_FCFS if fcfs else 0) | (oracle.FSO_BLIND if blind else 0) |
             (oracle.FSO_LITERAL if literal else 0))
    o = oracle.simulate(tr, cost, o_th.reason, step, cap, theta, flags=flags)
    chunks = int(rng.integers(1, 40)) if mode == 2 else None
    g = gpu_schedule(tr, cost, o_th.reason, step, cap, theta, chunks=chunks,
                     global_only=(mode == 1), fcfs=fcfs, blind=blind, literal=literal)
    compare_sim(g, o)


@pytest.mark.parametrize("seed", range(80))
def test_random_wide_keys(seed):
    """Costs from a few tokens' worth up to 2^40, so that the counters of the backlogged
    users spread over more than 2^31 (the on-chip scheduler then compares full keys, also
    when it takes a step's admissions together)."""
    tr, W, t_user, t_app, step, literal, cap, theta, fcfs, blind, mode, _, rng = _case(7000 + seed)
    fcfs = fcfs and seed % 4 == 0
    blind = blind and seed % 4 == 1
    bits = rng.integers(0, 41, tr.n)
    cost = (rng.integers(0, 1 << 20, tr.n).astype(np.int64) << 20) >> (40 - bits)
    say("fuzz wide", seed, tr.n_replicas, tr.n_users, tr.n, literal, fcfs, blind, mode)
    o_th = oracle.throttle(tr, W, t_user, t_app, raw=True, counts=False)
    flags = ((oracle.FSO_FCFS if fcfs else 0) | (oracle.FSO_BLIND if blind else 0) |
             (oracle.FSO_LITERAL if literal else 0))
    o = oracle.simulate(tr, cost, o_th.reason, step, cap, theta, flags=flags)
    chunks = int(rng.integers(1, 40)) if mode == 2 else None
    g = gpu_schedule(tr, cost, o_th.reason, step, cap, theta, chunks=chunks,
                     global_only=(mode == 1), fcfs=fcfs, blind=blind, literal=literal)
    compare_sim(g, o)


@pytest.mark.parametrize("seed", range(150))
def test_random_throttle_modes(seed):
    """Gated (random overload flags or always overloaded) and raw, per-(user, app) and
    app-level limits, with the window counts."""
    from gpu_common import bits_of
    tr, W, t_user, t_app, *_, rng = _case(5000 + seed)
    raw = bool(rng.integers(0, 2))
    scope = int(rng.integers(0, 2))
    ov = None if rng.integers(0, 2) else rng.integers(0, 2, tr.n).astype(np.uint8)
    say("fuzz throttle", seed, tr.n, raw, scope, ov is None)
    o = oracle.throttle(tr, W, t_user, t_app, overloaded=ov, raw=raw, counts=True,
                        app_scope=scope)
    g = gpu_throttle(tr, W, t_user, t_app, ov, raw, True, scope)
    assert (g["reason"] == o.reason).all()
    assert (bits_of(g["bitmap"], tr.n) == bits_of(o.bitmap, tr.n)).all()
    assert (g["cnt_user"] == o.cnt_user).all() and (g["cnt_app"] == o.cnt_app).all()


@pytest.mark.parametrize("seed", range(100))
def test_random_cost(seed):
    """Random Q16 coefficient tables (shared or per replica, 1 to 20 stages) and Q8
    priorities (none, shared or per replica)."""
    import torch
    import paper_2411_15997_amd as fs
    tr, *_, rng = _case(9000 + seed)
    R, A, U = tr.n_replicas, tr.n_apps, tr.n_users
    J = int(rng.choice([1, 2, 20]))
    per_rep = bool(rng.integers(0, 2))
    coef = rng.integers(0, 1 << int(rng.choice([8, 17, 30])), (R if per_rep else 1, A, J, 3))
    pmode = int(rng.integers(0, 3))  # 0 none, 1 shared, 2 per replica
    prio = (None if pmode == 0 else
            rng.integers(0, 1 << 12, (R if pmode == 2 else 1, U)).astype(np.int32))
    say("fuzz cost", seed, tr.n, J, per_rep, pmode)
    o = oracle.cost(tr, coef, prio if pmode else None, coef_per_replica=per_rep,
                    prio_per_replica=pmode == 2)
    dt = fs.DeviceTrace(tr)
    w, keep = fs.make_weights(dt, coef, prio if pmode else None, per_rep, pmode == 2)
    c = fs.fs_cost(dt, w, cost=torch.empty(tr.n, dtype=torch.int64, device=dt.device))
    assert (c.cpu().numpy() == o).all()


@pytest.mark.parametrize("seed", range(60))
def test_random_history(seed):
    """fs_weights_from_history on random histories (several replicas pooled, 1 to 20
    stages, random K and base limit)."""
    import paper_2411_15997_amd as fs
    tr, *_, rng = _case(12000 + seed)
    J = int(rng.choice([1, 3, 20]))
    K = int(rng.integers(1, 1 << 20))
    base = int(rng.integers(0, 200))
    say("fuzz history", seed, tr.n, J, K, base)
    o = oracle.weights_from_history(tr, J, K=K, base_limit=base)
    dt = fs.DeviceTrace(tr)
    st, c, t = fs.fs_weights_from_history(dt, J, K=K, base_limit=base)
    assert (st.cpu().numpy() == o.stats).all()
    assert (c.cpu().numpy() == o.coef).all()
    assert (t.cpu().numpy() == o.t_app).all()


@pytest.mark.parametrize("seed", range(60))
def test_random_metrics(seed):
    """fs_fairness_metrics on random outputs of random traces; every fourth case with
    5,000 users (the global-memory aggregation)."""
    import torch
    import paper_2411_15997_amd as fs
    tr, W, t_user, t_app, step, *_, rng = _case(15000 + seed)
    if seed % 4 == 3:
        tr = tg.Trace(**{**tr.__dict__, "n_users": 5000,
                         "user": (tr.user * 997 + 13) % 5000})
    n = tr.n
    cost = rng.integers(0, 10 ** 6, n).astype(np.int64)
    status = rng.choice(np.array([0, 0, 1, 2, 3], np.int8), n)
    admit_step = np.where(status == 0, tr.ts_us // step + rng.integers(0, 3, n),
                          -1).astype(np.int32)
    max_gap = rng.integers(0, 2 ** 40, tr.n_replicas).astype(np.int64)
    delay = int(rng.integers(0, 3))
    say("fuzz metrics", seed, n, tr.n_users, delay)
    mo = oracle.fairness_metrics(tr, cost, status, admit_step, max_gap, step, delay)
    dt = fs.DeviceTrace(tr)
    out = fs.Outputs(dt, parity=False)
    if n:
        out.status[:n].copy_(torch.as_tensor(status))
        out.admit_step[:n].copy_(torch.as_tensor(admit_step))
    out.max_gap.copy_(torch.as_tensor(max_gap))
    eng = fs.make_engine(step, 1000, 1000)
    m = fs.fs_fairness_metrics(dt, torch.as_tensor(cost).to(dt.device), out, eng, delay).host()
    for k in ("throttled", "aborted_midway", "wasted_tokens"):
        assert (m[k] == getattr(mo, k)).all(), k
    for k in ("jain", "max_gap_tokens", "svc_req_pct", "svc_int_pct", "served_users_pct",
              "delayed_users_pct"):
        np.testing.assert_allclose(m[k], getattr(mo, k), rtol=1e-9, atol=0, err_msg=k)

"""The paper's comparison policies on the same kernels, bit-exact against the oracle:
first come first served, interaction-blind limits, both together with the limits
always on (the request-rate-limit policy), the WSC-only ablation (no limits) and the
virtual token counter (equal coefficients, no limits)."""
import numpy as np
import pytest

import oracle
import paper_2411_15997_amd as fs
from gpu_common import compare_sim, gpu_schedule, say, workload_trace
from tiny import random_trace
import tracegen as tg

pytestmark = pytest.mark.gpu

MODES = {"fcfs": oracle.FSO_FCFS, "blind": oracle.FSO_BLIND,
         "rate_limit": oracle.FSO_FCFS | oracle.FSO_BLIND}


def _run(tr, cost, reason, step, cap, theta, flags, **kw):
    o = oracle.simulate(tr, cost, reason, step, cap, theta, flags=flags)
    g = gpu_schedule(tr, cost, reason, step, cap, theta, fcfs=bool(flags & oracle.FSO_FCFS),
                     blind=bool(flags & oracle.FSO_BLIND), **kw)
    compare_sim(g, o)
    return g, o


@pytest.mark.parametrize("mode", list(MODES))
def test_many_tiny_replicas(mode):
    rng = np.random.default_rng(70 + len(mode))
    reps = [random_trace(rng, int(rng.integers(1, 40)), int(rng.integers(1, 5)), 2,
                         int(rng.integers(1, 300)), multi=True, max_tok=6) for _ in range(300)]
    tr = tg.concat(reps)
    cost = rng.integers(0, 50, tr.n).astype(np.int64)
    reason = rng.integers(0, 3, tr.n).astype(np.uint8)
    for theta in (-1, 4):
        say("policy tiny", mode, theta, tr.n)
        _run(tr, cost, reason, 20, 6, theta, MODES[mode])


def _workload(name, **kw):
    wl, tr = workload_trace(name, **kw)
    coef, per_rep = fs.workload_weights(wl, tr)
    return wl, tr, oracle.cost(tr, coef, coef_per_replica=per_rep)


@pytest.mark.parametrize("chunks,global_only", [(None, False), (None, True), (97, False)])
def test_rate_limit_policy_replica_workload(chunks, global_only):
    """Per-user request limit, always on, interaction-blind, first come first served."""
    wl, tr, c = _workload("c2_replicas", replicas=3, records=20000)
    raw = oracle.throttle(tr, wl.window_us, wl.t_user, [2 ** 31 - 1] * tr.n_apps,
                          counts=False).reason
    say("rate limit", tr.n, chunks, global_only)
    g, o = _run(tr, c, raw, wl.step_us, wl.cap_tokens, -1, MODES["rate_limit"], chunks=chunks,
                global_only=global_only)
    assert (o.status == 3).any()  # interactions abandoned midway


def test_fcfs_and_blind_overflow_to_global_memory():
    """More backlogged users than fit on chip, under both new rules."""
    rng = np.random.default_rng(71)
    tr = random_trace(rng, 5000, 300, 2, 3000, multi=True, max_tok=8)
    c = rng.integers(1, 1000, tr.n).astype(np.int64)
    reason = rng.integers(0, 3, tr.n).astype(np.uint8)
    for flags in MODES.values():
        _run(tr, c, reason, 100, 30, 10 ** 9, flags)
        _run(tr, c, reason, 100, 30, 40, flags)


@pytest.mark.parametrize("policy", ["wsc_only", "virtual_token_counter"])
def test_unlimited_policies(policy):
    """No limits (the WSC-only ablation); with equal coefficients for every app, the
    virtual token counter."""
    wl, tr = workload_trace("c2_replicas", replicas=3, records=20000)
    if policy == "wsc_only":
        coef, per_rep = fs.workload_weights(wl, tr)
    else:
        coef, per_rep = np.full((1, tr.n_apps, 1, 3), 1 << 16, np.int64), False
    c = oracle.cost(tr, coef, coef_per_replica=per_rep)
    big = 2 ** 31 - 1
    raw = oracle.throttle(tr, wl.window_us, big, [big] * tr.n_apps, counts=False).reason
    assert not raw.any()
    _run(tr, c, raw, wl.step_us, wl.cap_tokens, wl.overload_tokens, 0)


def test_rate_limit_policy_wastes_tokens_fs_does_not():
    """The paper's comparison on a synthetic replica: interaction-blind limits abort
    interactions midway and waste their served tokens; the paper's policy aborts none."""
    wl, tr, c = _workload("c2_replicas", replicas=2, records=30000)
    dt = fs.DeviceTrace(tr)
    import torch
    cost_d = torch.as_tensor(c).cuda()
    raw_rpm = oracle.throttle(tr, wl.window_us, wl.t_user, [2 ** 31 - 1] * tr.n_apps,
                              counts=False).reason
    raw_fs = oracle.throttle(tr, wl.window_us, wl.t_user, wl.t_app, counts=False).reason
    res = {}
    for name, raw, theta, fl in (("rpm", raw_rpm, -1, MODES["rate_limit"]),
                                 ("fs", raw_fs, wl.overload_tokens, 0)):
        o = oracle.simulate(tr, c, raw, wl.step_us, wl.cap_tokens, theta, flags=fl)
        eng = fs.make_engine(wl.step_us, wl.cap_tokens, theta, fcfs=bool(fl & 1), blind=bool(fl & 2))
        out = fs.Outputs(dt)
        st = fs.fs_state_init(dt)
        fs.fs_schedule_step(dt, st, cost_d, torch.as_tensor(raw).cuda(), eng, out, -1)
        m = fs.fs_fairness_metrics(dt, cost_d, out, eng, 0).host()
        mo = oracle.fairness_metrics(tr, c, o.status, o.admit_step, o.max_gap, wl.step_us)
        for k in ("throttled", "aborted_midway", "wasted_tokens"):
            assert (m[k] == getattr(mo, k)).all(), (name, k)
        for k in ("jain", "svc_req_pct", "svc_int_pct", "served_users_pct", "delayed_users_pct"):
            np.testing.assert_allclose(m[k], getattr(mo, k), rtol=1e-9, err_msg=f"{name} {k}")
        res[name] = m
    assert (res["rpm"]["aborted_midway"] > 0).all() and (res["rpm"]["wasted_tokens"] > 0).all()
    assert (res["fs"]["aborted_midway"] == 0).all() and (res["fs"]["wasted_tokens"] == 0).all()

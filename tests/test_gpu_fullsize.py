"""Full-size parity: each workload at its real size, in the launch configuration the
benchmark times (fs_run_trace + fs_fairness_metrics, or fs_throttle for the
throttle-only stream), compared bit-exact with the oracle (fp64 metrics to 1e-9)."""
import numpy as np
import pytest

import oracle
import paper_2411_15997_amd as fs
from gpu_common import bits_of, compare_sim, gpu_throttle, say, workload_trace

pytestmark = pytest.mark.gpu


def _full_path(name):
    wl, tr = workload_trace(name)
    say("full path", name, tr.n)
    dt = fs.DeviceTrace(tr)
    coef, per_rep = fs.workload_weights(wl, tr)
    w, keep = fs.make_weights(dt, coef, None, per_rep)
    lim = fs.make_limits(wl.window_us, wl.t_user, wl.t_app)
    eng = fs.make_engine(wl.step_us, wl.cap_tokens, wl.overload_tokens)
    out = fs.Outputs(dt)
    ws, cost_view, reason_view = fs.run_trace_buffers(dt)
    fs.fs_run_trace(dt, w, lim, eng, out, ws)
    m = fs.fs_fairness_metrics(dt, cost_view, out, eng).host()
    h = out.host()
    gcost = cost_view.cpu().numpy()
    greason = reason_view.cpu().numpy()
    del ws, out, dt
    say("  gpu done; oracle")
    c, th, sim, met = oracle.run_workload(wl, tr, n_threads=16)
    assert (gcost == c).all()
    assert (greason == th.reason).all()
    n = tr.n
    compare_sim({k: (v[:n] if v is not None and k not in ("counter", "steps", "decisions",
                                                          "max_gap") else v)
                 for k, v in h.items()}, sim)
    for k in ("jain", "max_gap_tokens", "svc_req_pct", "svc_int_pct", "served_users_pct",
              "delayed_users_pct"):
        np.testing.assert_allclose(m[k], getattr(met, k), rtol=1e-9, atol=0, err_msg=k)
    for k in ("throttled", "aborted_midway", "wasted_tokens"):
        assert (m[k] == getattr(met, k)).all(), k
    say("  ok:", int(h["decisions"].sum()), "admissions")


def test_full_small():
    _full_path("c1_small")


def test_full_replica_workload():
    """64 replicas x 256 users x 8 apps, 6.4M requests: the benchmark's default line."""
    _full_path("c2_replicas")


def test_full_weight_sweep():
    """1,024 replicas x 1,024 users, 20.48M requests, one weight pair per replica."""
    _full_path("c4_sweep")


def test_full_large_tenant():
    """1 replica, 100,000 users, 10M requests over 24 h (counters in global memory)."""
    _full_path("c5_tenant")


def test_full_throttle_stream():
    """The 50M-request throttle-only stream: overload forced on, bitmap bit-exact."""
    wl, tr = workload_trace("c3_throttle")
    say("throttle full", tr.n)
    g = gpu_throttle(tr, wl.window_us, wl.t_user, wl.t_app, raw=False, counts=False)
    say("  gpu done; oracle")
    o = oracle.throttle(tr, wl.window_us, wl.t_user, wl.t_app, raw=False, counts=False)
    assert (g["reason"] == o.reason).all()
    nw = (tr.n + 31) // 32
    assert (g["bitmap"][:nw] == o.bitmap[:nw]).all()
    say("  ok:", int((o.reason > 0).sum()), "throttled")


NO_LIMIT = 2 ** 31 - 1


@pytest.mark.parametrize("policy", ["rpm", "literal"])
def test_full_replica_workload_policy_and_engine(policy):
    """The 64 x 256 x 8 replica workload (6.4M requests) as the benchmark runs it with
    --policy rpm (per-user limit always on, interaction-blind, first come first served)
    or --engine literal (20 ms decode steps, 2^22 KV tokens per replica), through
    fs_run_trace and fs_fairness_metrics, bit-exact with the oracle."""
    wl, tr = workload_trace("c2_replicas")
    say("full", policy, tr.n)
    if policy == "rpm":
        t_user, t_app, theta = wl.t_user, [NO_LIMIT] * tr.n_apps, -1
        fcfs, blind, literal = True, True, False
        step_us, cap = wl.step_us, wl.cap_tokens
    else:
        t_user, t_app, theta = wl.t_user, list(wl.t_app), wl.overload_tokens
        fcfs, blind, literal = False, False, True
        step_us, cap = 20_000, 1 << 22
    dt = fs.DeviceTrace(tr)
    coef, per_rep = fs.workload_weights(wl, tr)
    w, keep = fs.make_weights(dt, coef, None, per_rep)
    lim = fs.make_limits(wl.window_us, t_user, t_app)
    eng = fs.make_engine(step_us, cap, theta, fcfs=fcfs, blind=blind, literal=literal)
    out = fs.Outputs(dt)
    ws, cost_view, reason_view = fs.run_trace_buffers(dt)
    fs.fs_run_trace(dt, w, lim, eng, out, ws)
    m = fs.fs_fairness_metrics(dt, cost_view, out, eng).host()
    h = out.host()
    gcost, greason = cost_view.cpu().numpy(), reason_view.cpu().numpy()
    del ws, out, dt
    say("  gpu done; oracle")
    ocoef, oper = oracle.weights_for(wl, tr)
    c = oracle.cost(tr, ocoef, coef_per_replica=oper)
    th = oracle.throttle(tr, wl.window_us, t_user, t_app, raw=True, counts=False)
    flags = ((oracle.FSO_FCFS if fcfs else 0) | (oracle.FSO_BLIND if blind else 0) |
             (oracle.FSO_LITERAL if literal else 0))
    sim = oracle.simulate(tr, c, th.reason, step_us, cap, theta, n_threads=16, flags=flags)
    met = oracle.fairness_metrics(tr, c, sim.status, sim.admit_step, sim.max_gap, step_us)
    assert (gcost == c).all()
    assert (greason == th.reason).all()
    n = tr.n
    compare_sim({k: (v[:n] if v is not None and k not in ("counter", "steps", "decisions",
                                                          "max_gap") else v)
                 for k, v in h.items()}, sim)
    for k in ("jain", "max_gap_tokens", "svc_req_pct", "svc_int_pct", "served_users_pct",
              "delayed_users_pct"):
        np.testing.assert_allclose(m[k], getattr(met, k), rtol=1e-9, atol=0, err_msg=k)
    for k in ("throttled", "aborted_midway", "wasted_tokens"):
        assert (m[k] == getattr(met, k)).all(), k
    if policy == "rpm":
        assert met.aborted_midway.sum() > 0
    say("  ok:", int(h["decisions"].sum()), "admissions")

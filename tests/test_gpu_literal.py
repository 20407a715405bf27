"""The literal engine (prefill at admission, one output token per step, KV-cache
capacity, charge at finish) on the GPU, bit-exact against the oracle."""
import numpy as np
import pytest

import oracle
import paper_2411_15997_amd as fs
from gpu_common import compare_sim, gpu_schedule, say, workload_trace
from tiny import random_trace
import tracegen as tg

pytestmark = pytest.mark.gpu

L = oracle.FSO_LITERAL
MODES = {"literal": L, "literal_rate_limit": L | oracle.FSO_FCFS | oracle.FSO_BLIND,
         "literal_fcfs": L | oracle.FSO_FCFS}


def _run(tr, cost, reason, step, kv, theta, flags, **kw):
    o = oracle.simulate(tr, cost, reason, step, kv, theta, flags=flags,
                        max_steps=kw.get("n_steps", -1))
    g = gpu_schedule(tr, cost, reason, step, kv, theta, fcfs=bool(flags & oracle.FSO_FCFS),
                     blind=bool(flags & oracle.FSO_BLIND), literal=True, **kw)
    compare_sim(g, o, decided_only=kw.get("n_steps", -1) >= 0)
    return g, o


@pytest.mark.parametrize("global_only", [False, True])
@pytest.mark.parametrize("mode", list(MODES))
def test_many_tiny_replicas(mode, global_only):
    rng = np.random.default_rng(80 + len(mode))
    reps = [random_trace(rng, int(rng.integers(1, 40)), int(rng.integers(1, 5)), 2,
                         int(rng.integers(1, 300)), multi=True, max_tok=6) for _ in range(300)]
    tr = tg.concat(reps)
    cost = rng.integers(0, 50, tr.n).astype(np.int64)
    reason = rng.integers(0, 3, tr.n).astype(np.uint8)
    for kv, theta in ((4, -1), (9, 4), (40, 10 ** 9)):
        say("literal tiny", mode, global_only, kv, theta, tr.n)
        _run(tr, cost, reason, 20, kv, theta, MODES[mode], global_only=global_only)


@pytest.mark.parametrize("chunks", [None, 3])
def test_running_batch_larger_than_on_chip(chunks):
    """Thousands of calls running at once: the on-chip batch fills and the replica
    continues in global memory, in the middle of a step's admissions (and, in chunks,
    resumes from the saved batch)."""
    rng = np.random.default_rng(91)
    reps = []
    for _ in range(3):
        n = 5000
        ts = np.sort(rng.integers(0, 40, size=n)).astype(np.int64)
        user = rng.integers(0, 30, size=n).astype(np.int32)
        reps.append(tg.Trace(1, 30, 1, np.array([0, n], np.int64), ts, user,
                             np.zeros(n, np.int32), None, None, None,
                             rng.integers(1, 20, n).astype(np.int32), None,
                             rng.integers(30, 120, n).astype(np.int32)))
    tr = tg.concat(reps)
    cost = rng.integers(1, 1 << 20, tr.n).astype(np.int64)
    say("literal big batch", tr.n, chunks)
    _run(tr, cost, None, 10, 10 ** 9, 10 ** 9, L, chunks=chunks)


def test_oversized_calls_and_zero_output():
    # calls larger than the KV cache run alone; calls with no output finish at once
    rng = np.random.default_rng(90)
    reps = []
    for _ in range(64):
        t = random_trace(rng, int(rng.integers(5, 60)), 3, 2, 200, multi=True, max_tok=9)
        t.len_out[rng.random(t.n) < 0.3] = 0
        reps.append(t)
    tr = tg.concat(reps)
    cost = rng.integers(1, 1000, tr.n).astype(np.int64)
    say("literal oversized", tr.n)
    _run(tr, cost, None, 7, 12, 10 ** 9, L)


def _workload(name, **kw):
    wl, tr = workload_trace(name, **kw)
    coef, per_rep = fs.workload_weights(wl, tr)
    return wl, tr, oracle.cost(tr, coef, coef_per_replica=per_rep)


def test_small_workload():
    """The 1-replica, 8-user workload with a 10 ms decode step and a 64k-token KV cache."""
    wl, tr, c = _workload("c1_small")
    raw = oracle.throttle(tr, wl.window_us, wl.t_user, wl.t_app, counts=False).reason
    say("literal c1", tr.n)
    g, o = _run(tr, c, raw, 10_000, 65536, 65536, L)
    assert (o.status == 0).sum() > 0


@pytest.mark.parametrize("chunks", [None, 997])
def test_replica_workload(chunks):
    """Four replicas of the 256-user workload, 20 ms decode steps, a 2^20-token KV cache;
    resumed every 997 steps the run must equal one call."""
    wl, tr, c = _workload("c2_replicas", replicas=4, records=15000)
    raw = oracle.throttle(tr, wl.window_us, wl.t_user, wl.t_app, counts=False).reason
    say("literal c2", tr.n, chunks)
    g, o = _run(tr, c, raw, 20_000, 1 << 20, 1 << 20, L, chunks=chunks)
    assert (o.status > 0).any() and (o.status == 0).any()


def test_without_optional_outputs():
    wl, tr, c = _workload("c2_replicas", replicas=4, records=15000)
    raw = oracle.throttle(tr, wl.window_us, wl.t_user, wl.t_app, counts=False).reason
    say("literal no optional outputs", tr.n)
    _run(tr, c, raw, 20_000, 1 << 20, 1 << 20, L, parity=False)


def test_bounded_run_is_a_prefix():
    wl, tr, c = _workload("c2_replicas", replicas=2, records=8000)
    raw = oracle.throttle(tr, wl.window_us, wl.t_user, wl.t_app, counts=False).reason
    for n_steps in (1, 5000, 40000):
        say("literal bounded", n_steps)
        _run(tr, c, raw, 20_000, 1 << 19, 1 << 19, L, n_steps=n_steps)


def test_large_tenant_slice():
    """One replica with many users and multi-call interactions (charges of queued users
    and of idle users both happen at finish)."""
    wl, tr, c = _workload("c5_tenant", records=60_000, users=5000)
    raw = oracle.throttle(tr, wl.window_us, wl.t_user, wl.t_app, counts=False).reason
    say("literal c5 slice", tr.n)
    _run(tr, c, raw, 40_000, 1 << 21, 1 << 21, L)

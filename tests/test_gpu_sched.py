"""Parity of the WSC scheduler (fs_schedule_step / fs_run_trace) with the oracle, bit-exact."""
import numpy as np
import pytest
import torch

import oracle
import paper_2411_15997_amd as fs
from gpu_common import compare_sim, gpu_schedule, gpu_throttle, say, workload_trace
from tiny import load_golden, random_trace, trace_from_case
import tracegen as tg

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("case", load_golden("hand_traces.json")["cases"], ids=lambda c: c["name"])
def test_hand_traces(case):
    tr = trace_from_case(case)
    g = gpu_schedule(tr, case["cost"], case["reason"], case["tau"], case["C"], case["theta"])
    for k in ("status", "admit_step", "admit_seq", "counter_after", "counter_on_arrival", "counter"):
        assert g[k].tolist() == case[k], k
    assert int(g["steps"][0]) == case["steps"] and int(g["max_gap"][0]) == case["max_gap"]


def _batch_of_random(rng, count, n_max, U_max, multi=True):
    reps = []
    for _ in range(count):
        n = int(rng.integers(1, n_max))
        reps.append(random_trace(rng, n, int(rng.integers(1, U_max)), 2, int(rng.integers(1, 400)),
                                 multi=multi, max_tok=6))
    # all replicas share U = max; user ids stay valid
    return tg.concat(reps)


@pytest.mark.parametrize("seed", range(3))
def test_many_tiny_replicas_one_launch(seed):
    """Hundreds of random tiny traces, each a replica of one launch."""
    rng = np.random.default_rng(50 + seed)
    tr = _batch_of_random(rng, 400, 40, 5)
    cost = rng.integers(0, 50, tr.n).astype(np.int64)
    reason = rng.integers(0, 3, tr.n).astype(np.uint8)
    step, cap, theta = int(rng.integers(1, 40)), int(rng.integers(1, 12)), int(rng.integers(-1, 8))
    say("sched tiny", seed, tr.n)
    o = oracle.simulate(tr, cost, reason, step, cap, theta)
    g = gpu_schedule(tr, cost, reason, step, cap, theta)
    compare_sim(g, o)


@pytest.mark.parametrize("seed,multi", [(0, True), (1, True), (2, False)])
def test_many_replicas_counted_per_replica(seed, multi):
    """Enough replicas (at least 512, each of at most 2^16 requests) that the state's
    per-(replica, user) counts and next-call links are taken one work-group a replica."""
    rng = np.random.default_rng(70 + seed)
    tr = _batch_of_random(rng, 700, 60, 9, multi=multi)
    cost = rng.integers(0, 50, tr.n).astype(np.int64)
    reason = rng.integers(0, 3, tr.n).astype(np.uint8)
    step, cap, theta = int(rng.integers(1, 40)), int(rng.integers(1, 12)), int(rng.integers(-1, 8))
    say("sched per-replica counts", seed, tr.n_replicas, tr.n)
    o = oracle.simulate(tr, cost, reason, step, cap, theta)
    g = gpu_schedule(tr, cost, reason, step, cap, theta)
    compare_sim(g, o)


def _run_workload(wl, tr, global_only=False):
    coef, per_rep = fs.workload_weights(wl, tr)
    c = oracle.cost(tr, coef, coef_per_replica=per_rep)
    th = oracle.throttle(tr, wl.window_us, wl.t_user, wl.t_app, counts=False)
    o = oracle.simulate(tr, c, th.reason, wl.step_us, wl.cap_tokens, wl.overload_tokens,
                        n_threads=8)
    g = gpu_schedule(tr, c, th.reason, wl.step_us, wl.cap_tokens, wl.overload_tokens,
                     global_only=global_only)
    return g, o, c, th


@pytest.mark.parametrize("name,kw", [
    ("c1_small", {}),
    ("c2_replicas", dict(replicas=4)),
    ("c4_sweep", dict(replicas=64)),
    ("c5_tenant", dict(records=400_003, users=40_000)),
])
def test_workloads_schedule(name, kw):
    wl, tr = workload_trace(name, **kw)
    say("sched", name, tr.n)
    g, o, _, _ = _run_workload(wl, tr)
    compare_sim(g, o)


@pytest.mark.parametrize("mode", ["fs", "fcfs", "blind", "literal"])
def test_users_sharing_low_bits(mode):
    """User ids spread so that groups of users share their low 12 bits: the on-chip
    kernel's per-user tables for matching the arrival window collide often (and then
    match users bit by bit), and must give the same schedule in every engine mode."""
    wl, tr = workload_trace("c2_replicas", replicas=4, records=15000)
    spread = (tr.user % 3) + 4096 * (tr.user // 3)
    tr = tg.Trace(**{**tr.__dict__, "user": spread.astype(np.int32),
                     "n_users": int(spread.max()) + 1})
    say("sched colliding users", mode, tr.n, tr.n_users)
    if mode == "fs":
        g, o, _, _ = _run_workload(wl, tr)
    else:
        coef, per_rep = fs.workload_weights(wl, tr)
        c = oracle.cost(tr, coef, coef_per_replica=per_rep)
        th = oracle.throttle(tr, wl.window_us, wl.t_user, wl.t_app, counts=False)
        flags = {"fcfs": oracle.FSO_FCFS, "blind": oracle.FSO_BLIND | oracle.FSO_FCFS,
                 "literal": oracle.FSO_LITERAL}[mode]
        step, cap = (20_000, 1 << 20) if mode == "literal" else (wl.step_us, wl.cap_tokens)
        o = oracle.simulate(tr, c, th.reason, step, cap, wl.overload_tokens, flags=flags)
        g = gpu_schedule(tr, c, th.reason, step, cap, wl.overload_tokens,
                         fcfs=bool(flags & oracle.FSO_FCFS), blind=bool(flags & oracle.FSO_BLIND),
                         literal=mode == "literal")
    compare_sim(g, o)
    assert (o.status == 0).any() and (o.status > 0).any()


@pytest.mark.parametrize("name,kw", [("c2_replicas", dict(replicas=4, records=15000)),
                                     ("c4_sweep", dict(replicas=16))])
def test_without_optional_outputs(name, kw):
    """Without admit_seq, counter_after and counter_on_arrival (the kernel then skips
    the work that only feeds them) the remaining outputs are unchanged."""
    wl, tr = workload_trace(name, **kw)
    coef, per_rep = fs.workload_weights(wl, tr)
    c = oracle.cost(tr, coef, coef_per_replica=per_rep)
    th = oracle.throttle(tr, wl.window_us, wl.t_user, wl.t_app, counts=False)
    o = oracle.simulate(tr, c, th.reason, wl.step_us, wl.cap_tokens, wl.overload_tokens,
                        n_threads=8)
    say("sched no optional outputs", name, tr.n)
    g = gpu_schedule(tr, c, th.reason, wl.step_us, wl.cap_tokens, wl.overload_tokens,
                     parity=False)
    assert g["admit_seq"] is None and g["counter_on_arrival"] is None
    compare_sim(g, o)


def test_global_memory_path_matches():
    wl, tr = workload_trace("c2_replicas", replicas=2, records=20000)
    g, o, _, _ = _run_workload(wl, tr, global_only=True)
    compare_sim(g, o)


@pytest.mark.parametrize("literal", [False, True])
def test_global_memory_path_many_replicas_many_users(literal):
    """800 replicas of 800 users: the global-memory kernel's user table would not let
    every replica's work-group be resident at once, so it keeps the table in HBM."""
    rng = np.random.default_rng(63 + literal)
    reps = [random_trace(rng, int(rng.integers(1, 30)), 800, 2, 400, multi=True, max_tok=6)
            for _ in range(800)]
    tr = tg.concat(reps)
    cost = rng.integers(0, 100, tr.n).astype(np.int64)
    reason = rng.integers(0, 3, tr.n).astype(np.uint8)
    say("global many replicas", literal, tr.n)
    cap = 40 if literal else 8  # (the literal engine's KV capacity)
    o = oracle.simulate(tr, cost, reason, 20, cap, 6, flags=oracle.FSO_LITERAL if literal else 0)
    g = gpu_schedule(tr, cost, reason, 20, cap, 6, global_only=True, literal=literal)
    compare_sim(g, o)


def test_onchip_overflow_resumes_in_global_memory():
    """More backlogged users and queued requests than fit on chip: with no
    throttling and a tiny capacity the queue grows to thousands of requests."""
    rng = np.random.default_rng(60)
    n, U = 6000, 700
    ts = np.sort(rng.integers(0, 2000, n)).astype(np.int64)
    user = rng.integers(0, U, n).astype(np.int32)
    tr = tg.Trace(1, U, 1, np.array([0, n], np.int64), ts, user, np.zeros(n, np.int32), None, None,
                  None, rng.integers(1, 9, n).astype(np.int32), None, np.zeros(n, np.int32))
    cost = rng.integers(1, 1000, n).astype(np.int64)
    o = oracle.simulate(tr, cost, None, 100, 40, 10 ** 9)
    g = gpu_schedule(tr, cost, None, 100, 40, 10 ** 9)
    compare_sim(g, o)
    # and with chained calls (later calls pile up as pending entries)
    tr2 = random_trace(rng, 5000, 300, 2, 3000, multi=True, max_tok=8)
    c2 = rng.integers(1, 1000, tr2.n).astype(np.int64)
    o2 = oracle.simulate(tr2, c2, None, 100, 30, 10 ** 9)
    g2 = gpu_schedule(tr2, c2, None, 100, 30, 10 ** 9)
    compare_sim(g2, o2)


@pytest.mark.parametrize("chunk", [1, 7, 250])
def test_stepwise_equals_one_call(chunk):
    """k calls of fs_schedule_step give the outputs of a single call (checkpoint/resume)."""
    wl, tr = workload_trace("c2_replicas", replicas=2, records=8000)
    coef, per_rep = fs.workload_weights(wl, tr)
    c = oracle.cost(tr, coef, coef_per_replica=per_rep)
    th = oracle.throttle(tr, wl.window_us, wl.t_user, wl.t_app, counts=False)
    o = oracle.simulate(tr, c, th.reason, wl.step_us, wl.cap_tokens, wl.overload_tokens)
    g = gpu_schedule(tr, c, th.reason, wl.step_us, wl.cap_tokens, wl.overload_tokens, chunks=chunk)
    compare_sim(g, o)


def test_bounded_run_matches_oracle_prefix():
    wl, tr = workload_trace("c1_small")
    coef, _ = fs.workload_weights(wl, tr)
    c = oracle.cost(tr, coef)
    th = oracle.throttle(tr, wl.window_us, wl.t_user, wl.t_app, counts=False)
    for s in (1, 13, 100):
        o = oracle.simulate(tr, c, th.reason, wl.step_us, wl.cap_tokens, wl.overload_tokens,
                            max_steps=s)
        g = gpu_schedule(tr, c, th.reason, wl.step_us, wl.cap_tokens, wl.overload_tokens, n_steps=s)
        compare_sim(g, o, decided_only=True)


def test_counter_overflow_reported():
    n = 3
    tr = tg.Trace(1, 1, 1, np.array([0, n], np.int64), np.zeros(n, np.int64), np.zeros(n, np.int32),
                  np.zeros(n, np.int32), None, None, None, np.ones(n, np.int32), None,
                  np.zeros(n, np.int32))
    cost = np.array([(1 << 61), (1 << 61) - 1, 1], np.int64)
    with pytest.raises(oracle.OracleError) as oe:
        oracle.simulate(tr, cost, None, 10, 100, 100)
    with pytest.raises(fs.FairServeError) as ge:
        gpu_schedule(tr, cost, None, 10, 100, 100)
    assert ge.value.code == oe.value.code == fs.FS_E_OVERFLOW


@pytest.mark.parametrize("users", [1, 2])
def test_counter_overflow_reported_on_chip(users):
    """Counters that reach 2^62 through many admissions of packable costs (below 2^40): the
    on-chip kernel's single-user pass (one user) and batched admissions (two users) stop
    before the overflowing admission, and the error is the oracle's."""
    n = users * ((1 << 22) + 1)
    z32 = np.zeros(n, np.int32)
    user = (np.arange(n) % users).astype(np.int32)
    tr = tg.Trace(1, users, 1, np.array([0, n], np.int64), np.zeros(n, np.int64), user, z32,
                  None, None, None, np.ones(n, np.int32), None, z32)
    cost = np.full(n, (1 << 40) - 1, np.int64)
    say("sched overflow on chip", users, n)
    with pytest.raises(oracle.OracleError) as oe:
        oracle.simulate(tr, cost, None, 10, 1 << 30, 1 << 40)
    with pytest.raises(fs.FairServeError) as ge:
        gpu_schedule(tr, cost, None, 10, 1 << 30, 1 << 40)
    assert ge.value.code == oe.value.code == fs.FS_E_OVERFLOW


def test_run_trace_and_metrics_full_path():
    """fs_run_trace (cost + raw throttle + steps) and fs_fairness_metrics end to end."""
    wl, tr = workload_trace("c2_replicas", replicas=3, records=30000)
    dt = fs.DeviceTrace(tr)
    coef, per_rep = fs.workload_weights(wl, tr)
    w, keep = fs.make_weights(dt, coef, None, per_rep)
    lim = fs.make_limits(wl.window_us, wl.t_user, wl.t_app)
    eng = fs.make_engine(wl.step_us, wl.cap_tokens, wl.overload_tokens)
    out = fs.Outputs(dt)
    ws, cost_view, reason_view = fs.run_trace_buffers(dt)
    fs.fs_run_trace(dt, w, lim, eng, out, ws)
    m = fs.fs_fairness_metrics(dt, cost_view, out, eng, delay_steps=0).host()
    c, th, sim, met = oracle.run_workload(wl, tr, n_threads=8)
    assert (cost_view.cpu().numpy() == c).all()
    assert (reason_view.cpu().numpy() == th.reason).all()
    h = out.host()
    compare_sim({k: (v[:tr.n] if v is not None and v.shape[0] >= tr.n and k not in ("counter",) else v)
                 for k, v in h.items()}, sim)
    for k in ("jain", "max_gap_tokens", "svc_req_pct", "svc_int_pct", "served_users_pct",
              "delayed_users_pct"):
        np.testing.assert_allclose(m[k], getattr(met, k), rtol=1e-9, atol=0, err_msg=k)
    for k in ("throttled", "aborted_midway", "wasted_tokens"):
        assert (m[k] == getattr(met, k)).all(), k


def test_long_fifos_spill_to_hbm_segments_and_refill():
    """A few users with thousands of queued first calls: the pool fills, later first
    calls go to the users' HBM segments and come back in refills."""
    rng = np.random.default_rng(61)
    n, U = 12000, 5
    ts = np.sort(rng.integers(0, 3000, n)).astype(np.int64)
    user = rng.integers(0, U, n).astype(np.int32)
    tr = tg.Trace(1, U, 1, np.array([0, n], np.int64), ts, user, np.zeros(n, np.int32), None,
                  None, None, rng.integers(1, 9, n).astype(np.int32), None, np.zeros(n, np.int32))
    cost = rng.integers(1, 1000, n).astype(np.int64)
    o = oracle.simulate(tr, cost, None, 100, 30, 10 ** 9)
    g = gpu_schedule(tr, cost, None, 100, 30, 10 ** 9)
    compare_sim(g, o)


def test_long_queues_with_pending_chains():
    """Chained calls of users with long queues: later calls arrive while their previous
    call waits (pending), some staged in the pool, some read at refill."""
    rng = np.random.default_rng(62)
    reps = []
    for _ in range(4):
        reps.append(random_trace(rng, 6000, 6, 2, 20000, multi=True, max_tok=9))
    tr = tg.concat(reps)
    cost = rng.integers(1, 5000, tr.n).astype(np.int64)
    reason = rng.integers(0, 3, tr.n).astype(np.uint8)
    for theta in (10 ** 9, 40):
        o = oracle.simulate(tr, cost, reason, 50, 20, theta)
        g = gpu_schedule(tr, cost, reason, 50, 20, theta)
        compare_sim(g, o)
        g2 = gpu_schedule(tr, cost, reason, 50, 20, theta, chunks=37)
        compare_sim(g2, o)


def test_full_replica_workload_c2():
    """All 64 replicas of the 64 x 256 x 8 workload (6.4M requests), bit-exact."""
    wl, tr = workload_trace("c2_replicas")
    say("sched full c2", tr.n)
    g, o, _, _ = _run_workload(wl, tr)
    compare_sim(g, o)


@pytest.mark.parametrize("multi", [False, True])
def test_empty_trace_every_entry_point(multi):
    """Replicas without requests (empty device tensors have no storage, so every
    per-request pointer is NULL): cost, throttle, state init, steps, the whole path and
    the metrics succeed and give the oracle's per-replica results."""
    rng = np.random.default_rng(64 + multi)
    tr = tg.concat([random_trace(rng, 0, 5, 2, 10, multi=multi) for _ in range(3)])
    assert tr.n == 0
    cost = np.zeros(0, np.int64)
    reason = np.zeros(0, np.uint8)
    for literal in (False, True):
        o = oracle.simulate(tr, cost, reason, 10, 50, 5,
                            flags=oracle.FSO_LITERAL if literal else 0)
        g = gpu_schedule(tr, cost, reason, 10, 50, 5, literal=literal)
        compare_sim(g, o)
    dt = fs.DeviceTrace(tr)
    coef = np.full((1, 2, 1, 3), 1 << 16, np.int64)
    w, keep = fs.make_weights(dt, coef, None, False)
    lim = fs.make_limits(100, 3, [2, 2])
    eng = fs.make_engine(10, 50, 5)
    empty_cost = torch.zeros(0, dtype=torch.int64, device=dt.device)
    fs.fs_cost(dt, w, cost=empty_cost)
    out = fs.Outputs(dt)
    ws, cost_view, reason_view = fs.run_trace_buffers(dt)
    fs.fs_run_trace(dt, w, lim, eng, out, ws)
    h = out.host()
    assert (h["steps"] == 0).all() and (h["decisions"] == 0).all() and (h["counter"] == 0).all()
    m = fs.fs_fairness_metrics(dt, empty_cost, out, eng).host()
    mo = oracle.fairness_metrics(tr, cost, np.zeros(0, np.int8), np.zeros(0, np.int32),
                                 h["max_gap"], 10)
    for k in ("jain", "svc_req_pct", "svc_int_pct", "served_users_pct", "delayed_users_pct"):
        np.testing.assert_allclose(m[k], getattr(mo, k), rtol=1e-9, atol=0, err_msg=k)
    for k in ("throttled", "aborted_midway", "wasted_tokens"):
        assert (m[k] == getattr(mo, k)).all(), k
    for raw in (True, False):
        gt = gpu_throttle(tr, 100, 3, [2, 2], raw=raw, counts=True)
        assert gt["reason"].size == 0


def test_state_of_another_trace_is_rejected():
    """fs_schedule_step on a state buffer initialised for another trace (another request
    count), with a corrupted version word, or never initialised: FS_E_STATE, and nothing
    else is written."""
    rng = np.random.default_rng(71)
    tr = random_trace(rng, 40, 4, 2, 200, multi=True)
    other = random_trace(rng, 30, 4, 2, 200, multi=True)
    cost = np.ones(tr.n, np.int64)
    dt, do = fs.DeviceTrace(tr), fs.DeviceTrace(other)
    c = torch.as_tensor(cost).cuda()
    eng = fs.make_engine(10, 50, 5)
    cases = []
    st = fs.fs_state_init(do)                       # initialised for `other`
    big = torch.zeros(max(st.numel(), fs.fs_state_bytes(dt)), dtype=torch.uint8, device="cuda")
    big[:st.numel()].copy_(st)
    cases.append(("other trace", big))
    bad = fs.fs_state_init(dt)
    bad[8:12].copy_(torch.tensor([99, 0, 0, 0], dtype=torch.uint8))  # the version word
    cases.append(("version", bad))
    cases.append(("never initialised", torch.zeros(fs.fs_state_bytes(dt), dtype=torch.uint8,
                                                   device="cuda")))
    for what, state in cases:
        say("state case", what)
        out = fs.Outputs(dt)
        out.steps.fill_(-7)
        with pytest.raises(fs.FairServeError) as ge:
            fs.fs_schedule_step(dt, state, c, None, eng, out, -1)
        assert ge.value.code == fs.FS_E_STATE, what
        assert (out.steps.cpu().numpy() == -7).all(), what
    # the right state still runs
    o = oracle.simulate(tr, cost, None, 10, 50, 5)
    compare_sim(gpu_schedule(tr, cost, None, 10, 50, 5), o)


def test_empty_trace_null_pointers_through_the_abi():
    """A trace without requests whose per-request arrays are all NULL (only the replica
    offsets set), passed to every entry point through the C-ABI: each call succeeds and
    the per-replica outputs are the oracle's."""
    import ctypes as C
    L = fs._lib()
    R, U, A = 3, 5, 2
    rep_h = np.zeros(R + 1, np.int64)
    rep_d = torch.zeros(R + 1, dtype=torch.int64, device="cuda")
    t = fs.fs_trace(R, U, A, rep_h.ctypes.data, rep_d.data_ptr(), None, None, None, None, None,
                    None, None, None, None)
    err = fs.err_word()
    S = fs._stream()
    coef = torch.full((1, A, 1, 3), 1 << 16, dtype=torch.int64, device="cuda")
    w = fs.fs_weights(1, 0, coef.data_ptr(), 0, None)
    assert L.fs_cost(C.byref(t), C.byref(w), None, err.data_ptr(), S) == fs.FS_OK
    t_app = np.array([2, 2], np.int32)
    lim = fs.fs_limits(100, 3, t_app.ctypes.data, 0)
    wsb = int(L.fs_throttle_workspace(C.byref(t)))
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device="cuda")
    for flags in (0, fs.FS_THROTTLE_RAW):
        assert L.fs_throttle(C.byref(t), C.byref(lim), None, flags, None, None, None, None,
                             ws.data_ptr(), wsb, err.data_ptr(), S) == fs.FS_OK
    assert fs.fs_sync_status(err) == fs.FS_OK
    sb = int(L.fs_state_bytes(C.byref(t)))
    state = torch.empty(sb, dtype=torch.uint8, device="cuda")
    assert L.fs_state_init(state.data_ptr(), sb, C.byref(t), S) == fs.FS_OK
    counter = torch.full((R * U,), -1, dtype=torch.int64, device="cuda")
    steps, dec, gap = (torch.full((R,), -1, dtype=torch.int64, device="cuda") for _ in range(3))
    out = fs.fs_outputs(None, None, None, None, None, counter.data_ptr(), steps.data_ptr(),
                        dec.data_ptr(), gap.data_ptr(), err.data_ptr())
    eng = fs.make_engine(10, 50, 5)
    assert L.fs_schedule_step(state.data_ptr(), C.byref(t), None, None, C.byref(eng),
                              C.byref(out), -1, S) == fs.FS_OK
    assert fs.fs_sync_status(err) == fs.FS_OK
    tr = tg.Trace(R, U, A, rep_h, np.zeros(0, np.int64), np.zeros(0, np.int32),
                  np.zeros(0, np.int32), None, None, None, np.zeros(0, np.int32), None,
                  np.zeros(0, np.int32))
    o = oracle.simulate(tr, np.zeros(0, np.int64), None, 10, 50, 5)
    assert (counter.cpu().numpy() == o.counter).all()
    assert (steps.cpu().numpy() == o.steps).all() and (dec.cpu().numpy() == o.decisions).all()
    assert (gap.cpu().numpy() == o.max_gap).all()
    rb = int(L.fs_run_trace_workspace(C.byref(t)))
    rws = torch.empty(max(rb, 256), dtype=torch.uint8, device="cuda")
    assert L.fs_run_trace(C.byref(t), C.byref(w), C.byref(lim), C.byref(eng), C.byref(out),
                          rws.data_ptr(), rb, S) == fs.FS_OK
    assert fs.fs_sync_status(err) == fs.FS_OK
    m = fs.Metrics(fs.DeviceTrace(tr))
    mb = int(L.fs_metrics_workspace(C.byref(t)))
    mws = torch.empty(max(mb, 256), dtype=torch.uint8, device="cuda")
    assert L.fs_fairness_metrics(C.byref(t), None, C.byref(out), C.byref(eng), 0, C.byref(m.s),
                                 mws.data_ptr(), mb, S) == fs.FS_OK
    assert fs.fs_sync_status(err) == fs.FS_OK
    mo = oracle.fairness_metrics(tr, np.zeros(0, np.int64), np.zeros(0, np.int8),
                                 np.zeros(0, np.int32), gap.cpu().numpy(), 10)
    mh = m.host()
    for k in ("jain", "svc_req_pct", "svc_int_pct", "served_users_pct", "delayed_users_pct"):
        np.testing.assert_allclose(mh[k], getattr(mo, k), rtol=1e-9, atol=0, err_msg=k)
    for k in ("throttled", "aborted_midway", "wasted_tokens"):
        assert (mh[k] == getattr(mo, k)).all(), k
    hb = int(L.fs_history_workspace(C.byref(t), 1))
    hws = torch.empty(max(hb, 256), dtype=torch.uint8, device="cuda")
    stats = torch.full((A, 1, 5), -1, dtype=torch.int64, device="cuda")
    assert L.fs_weights_from_history(C.byref(t), 1, 1024, 30, stats.data_ptr(), None, None,
                                     hws.data_ptr(), hb, err.data_ptr(), S) == fs.FS_OK
    assert fs.fs_sync_status(err) == fs.FS_OK
    assert (stats.cpu().numpy() == 0).all()


@pytest.mark.parametrize("users,multi,fcfs", [(3000, False, False), (5000, True, False),
                                              (20000, True, False), (3000, True, True)])
def test_global_memory_path_large_backlog(users, multi, fcfs):
    """Thousands of users backlogged at once on the global-memory path (capacity far
    below the offered load): the argmin reads the minima of blocks of 64 slots and one
    block; run in one call and in chunks of steps, bit-exact against the oracle."""
    rng = np.random.default_rng(users + 7 * multi + 3 * fcfs)
    n = 4 * users
    tr = random_trace(rng, n, users, 3, 20 * users, multi=multi, max_tok=30)
    cost = rng.integers(1, 1 << 20, n).astype(np.int64)
    say("large backlog", users, n, multi, fcfs)
    o = oracle.simulate(tr, cost, None, 40, 200, 10 ** 9, flags=oracle.FSO_FCFS if fcfs else 0)
    compare_sim(gpu_schedule(tr, cost, None, 40, 200, 10 ** 9, global_only=True, fcfs=fcfs), o)
    compare_sim(gpu_schedule(tr, cost, None, 40, 200, 10 ** 9, chunks=97, fcfs=fcfs), o)

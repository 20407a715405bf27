"""Shared helpers for the GPU parity tests (inputs from the seeded generator only)."""
import functools
import sys

import numpy as np

import tracegen as tg


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@functools.lru_cache(maxsize=8)
def workload_trace(name, replicas=None, records=None, users=None):
    base = tg.WORKLOADS[name]
    wl = base if (replicas is None and records is None and users is None) else tg.scaled(
        base, replicas=replicas, records=records, users=users)
    return wl, tg.generate(wl)


def bits_of(bitmap, n):
    b = np.asarray(bitmap, np.uint32)
    idx = np.arange(n)
    return ((b[idx // 32] >> (idx % 32).astype(np.uint32)) & 1).astype(np.uint8)


def gpu_throttle(tr, W, t_user, t_app, overloaded=None, raw=True, counts=True, app_scope=0):
    import paper_2411_15997_amd as fs
    dt = fs.DeviceTrace(tr)
    out = fs.fs_throttle(dt, fs.make_limits(W, t_user, t_app, app_scope), overloaded=overloaded,
                         raw=raw, want_reason=True, want_counts=counts)
    n = tr.n
    res = dict(reason=out.reason.cpu().numpy()[:n], bitmap=out.bitmap.cpu().numpy().view(np.uint32))
    if counts:
        res["cnt_user"] = out.cnt_user.cpu().numpy()[:n]
        res["cnt_app"] = out.cnt_app.cpu().numpy()[:n]
    return res


def gpu_schedule(tr, cost, reason, step_us, cap, theta, n_steps=-1, chunks=None,
                 global_only=False, parity=True, fcfs=False, blind=False, literal=False):
    """fs_state_init + fs_schedule_step (once, or in chunks of `chunks` steps)."""
    import torch
    import paper_2411_15997_amd as fs
    dt = fs.DeviceTrace(tr)
    c = torch.as_tensor(np.ascontiguousarray(cost, np.int64)).cuda()
    rz = None if reason is None else torch.as_tensor(np.ascontiguousarray(reason, np.uint8)).cuda()
    eng = fs.make_engine(step_us, cap, theta, global_only, fcfs=fcfs, blind=blind, literal=literal)
    out = fs.Outputs(dt, parity=parity)
    st = fs.fs_state_init(dt)
    if chunks is None:
        fs.fs_schedule_step(dt, st, c, rz, eng, out, n_steps)
    else:
        done = 0
        while True:
            fs.fs_schedule_step(dt, st, c, rz, eng, out, chunks)
            done += chunks
            steps = out.steps.cpu().numpy()
            # a replica stops advancing once drained; stop when no replica moved
            if n_steps >= 0 and done >= n_steps:
                break
            if done > 10 ** 7 or (steps < done).all():
                break
    h = out.host()
    return {k: (None if v is None else v[:tr.n] if k in ("status", "admit_step", "admit_seq",
                                                        "counter_after", "counter_on_arrival")
                else v) for k, v in h.items()}


def compare_sim(g, o, decided_only=False):
    """Bit-exact comparison of GPU scheduler outputs with the oracle's SimResult."""
    mask = slice(None)
    if decided_only:
        mask = o.status >= 0
    for k in ("status", "admit_step", "admit_seq", "counter_after"):
        if g.get(k) is None:
            continue
        a, b = g[k][mask], getattr(o, k)[mask]
        bad = np.nonzero(a != b)[0]
        assert bad.size == 0, f"{k}: {bad.size} mismatches, first at {bad[:5]}: gpu {a[bad[:5]]} oracle {b[bad[:5]]}"
    if g.get("counter_on_arrival") is not None:
        seen = o.counter_on_arrival >= 0
        a, b = g["counter_on_arrival"][seen], o.counter_on_arrival[seen]
        bad = np.nonzero(a != b)[0]
        assert bad.size == 0, f"counter_on_arrival: {bad.size} mismatches, first {bad[:5]}"
    for k in ("counter", "steps", "decisions", "max_gap"):
        a, b = g[k], getattr(o, k)
        bad = np.nonzero(a != b)[0]
        assert bad.size == 0, f"{k}: {bad.size} mismatches at {bad[:5]}: gpu {a[bad[:5]]} oracle {b[bad[:5]]}"

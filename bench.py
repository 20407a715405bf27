"""Benchmark of the FairServe policy hot path on one MI355X.

One step = the whole path over one synthetic workload resident in HBM:
fs_cost -> fs_throttle (raw) -> fs_state_init -> fs_schedule_step (until drained)
-> fs_fairness_metrics, i.e. the sequence fs_run_trace runs plus the metrics.
The default workload is the 1,024-replica weight sweep (the largest scheduler
workload).  A second leg times fs_throttle (gated, always overloaded) on the
50M-request throttle stream (the largest throttle workload) in its own timed
region.  Prints one JSON line: metric, value = scheduler decisions per second of
the whole step, per-stage medians from HIP events, the roofline of the dominant
kernel and of the throttle leg, and the CPU oracle timed on this host.

`--cpu-protocol` instead runs only the CPU oracle over every workload (one thread on
each, replicas split over the host's threads for the replica workloads, users hashed
over the threads for the throttle stream) and prints a table.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "scheduler decisions/sec + throttle evals/sec on 1 MI355X; % of HBM roofline"
HBM_PEAK_GBS = 8000.0
MALL_BYTES = 256 << 20          # MI355X Infinity Cache
CSRC = os.path.join(ROOT, "paper_2411_15997_amd", "csrc")
STAGE_SRC = {
    "cost": ["fs_cost.hip"],
    "throttle": ["fs_throttle.hip"],
    # the dominant kernel of the stage, k_schedule_onchip, and the header it shares
    "schedule": ["fs_sched_onchip.hip", "fs_sched_common.h"],
    "metrics": ["fs_metrics.hip"],
    "history": ["fs_history.hip"],
    "workload": ["fs_workload.hip"],
}

# HBM traffic of a stage's kernels from rocprofv3 --pmc runs: FETCH_SIZE and
# WRITE_SIZE (KiB per dispatch, summed over the stage's kernels), each scaled by
# bytes / counter of a plain 1 GiB device copy measured in the same run
# (bench.py --calib-copy).  Keyed by workload and stage; an entry counts only while
# the stage's sources hash to `src`.
MEASURED_TRAFFIC = {
    # k_schedule_onchip on the 1,024-replica weight sweep (20.48M requests)
    ("c4_sweep", "schedule"): {"src": "df9073c9ab2d1903", "fetch_kib": 313379.0,
                               "write_kib": 137709.46875, "fetch_factor": 1.99991,
                               "write_factor": 1.0},
    # every kernel of one fs_throttle call on the 50M-request throttle stream
    ("c3_throttle", "throttle"): {"src": "f12662f2bb0b6f6c", "fetch_kib": 1287878.3125,
                                  "write_kib": 1618727.9375, "fetch_factor": 1.99991,
                                  "write_factor": 1.0},
    # the same stream with the app limit counted per (app, replica) over all users
    ("c3_throttle+app_scope", "throttle"): {"src": "f12662f2bb0b6f6c", "fetch_kib": 2582543.5625,
                                            "write_kib": 3290211.28125, "fetch_factor": 1.99992,
                                            "write_factor": 1.0},
}

NO_LIMIT = 2 ** 31 - 1


def src_hash(stage):
    h = hashlib.sha256()
    for name in STAGE_SRC.get(stage, []):
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload, stage):
    m = MEASURED_TRAFFIC.get((workload, stage))
    if not m or m["src"] != src_hash(stage):
        return None
    return int(m["fetch_kib"] * 1024 * m["fetch_factor"] + m["write_kib"] * 1024 * m["write_factor"])


def algo_bytes(stage, tr, raw=True, parity=False, prio=False):
    """Algorithmic bytes per request of a stage: the minimum the method moves for this
    trace (the arrays it has) and these outputs."""
    has_call = tr.call is not None
    has_sys = tr.len_sys is not None
    lens = 8 + (4 if has_sys else 0)                  # len_in, len_out (+ len_sys)
    if stage == "cost":                               # app, (call), lengths, (user) -> cost
        return 4 + (4 if has_call else 0) + lens + (4 if prio else 0) + 8
    if stage == "throttle":
        if raw:                                       # ts, user, app -> reason byte, bitmap bit
            return 8 + 4 + 4 + 1 + 0.125
        # gated: ts, user, app and the interaction's first call -> bitmap bit
        return 8 + 4 + 4 + (4 if has_call else 0) + 0.125
    if stage == "schedule":
        # ts, user, lengths, cost, raw reason, (call, head, prev) -> status, admit_step
        b = 8 + 4 + lens + 8 + 1 + (12 if has_call else 0) + 1 + 4
        return b + (20 if parity else 0)              # admit_seq, counter_after, _on_arrival
    if stage == "metrics":                            # status, admit_step, ts, user, cost
        return 1 + 4 + 8 + 4 + 8 + (8 if has_call else 0)
    if stage == "history":                            # app, (call), lengths, read once
        return 4 + (4 if has_call else 0) + lens
    if stage == "workload":                           # ts, user, app, lengths, (call, head)
        return 8 + 4 + 4 + lens + (8 if has_call else 0)
    return 0.0


def workload_out_bytes(tr):
    """Bytes the workload analysis writes: per (replica, user, app) requests and tokens,
    per (replica, user) the same, and the per-replica histograms."""
    R, U, A = tr.n_replicas, tr.n_users, tr.n_apps
    return 8 * (2 * R * U * A + 2 * R * U + R * ((A + 1) * 2 * 128 + A * 3 * 32 + A * 3 + A * 64
                                                 + 7 * 5 + 1))


def policy_settings(wl, n_apps, policy):
    """Limits, engine flags and coefficient choice of a policy (the paper's own, or one
    it compares with) on a workload: (t_user, t_app, overload_tokens, fcfs, blind,
    equal_coefficients)."""
    if policy == "fs":            # FairServe: WSC plus interaction-aware OIT
        return wl.t_user, list(wl.t_app), wl.overload_tokens, False, False, False
    if policy == "wsc_only":      # the paper's WSC-only ablation: no limits
        return NO_LIMIT, [NO_LIMIT] * n_apps, wl.overload_tokens, False, False, False
    if policy == "vtc":           # virtual token counter: equal token weights, no limits
        return NO_LIMIT, [NO_LIMIT] * n_apps, wl.overload_tokens, False, False, True
    if policy == "rpm":           # per-user request limit, always on, interaction-blind, FCFS
        return wl.t_user, [NO_LIMIT] * n_apps, -1, True, True, False
    raise ValueError(policy)


def host_cpu():
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count() or 1
    return {"model": model, "nproc": os.cpu_count() or 1, "available": avail}


def median(xs):
    import numpy as np
    return float(np.median(np.asarray(xs, np.float64)))


def roofline(stage, algo, ms, workload, limiter=None):
    achieved = algo / (ms / 1000.0) / 1e9
    r = {"bound": "hbm", "kernel": stage, "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
         "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 6), "traffic": measured_traffic(
             workload, stage), "algorithmic_bytes": int(algo), "src": src_hash(stage),
         "mall_resident": bool(algo < MALL_BYTES)}
    if limiter:
        r["limiter"] = limiter
    return r


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c4_sweep")
    ap.add_argument("--throttle-workload", default="c3_throttle",
                    help="workload of the throttle leg ('none' to skip it)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-threads", type=int, default=0)
    ap.add_argument("--cpu-protocol", action="store_true",
                    help="time only the CPU oracle on every workload and print a table")
    ap.add_argument("--stage-only", default="", help="time only this stage (profiling runs): "
                    "cost, throttle, schedule, metrics, history or workload")
    ap.add_argument("--policy", default="fs", choices=["fs", "wsc_only", "vtc", "rpm"],
                    help="the paper's policy (default) or one it compares with")
    ap.add_argument("--engine", default="step", choices=["step", "literal"],
                    help="step: token budget per step, charge at admission; literal: prefill at "
                         "admission, one output token per decode step, KV-cache capacity, "
                         "charge at finish")
    ap.add_argument("--decode-step-us", type=int, default=20_000,
                    help="literal engine: duration of one decode step")
    ap.add_argument("--kv-tokens", type=int, default=1 << 22,
                    help="literal engine: KV-cache capacity per replica, in tokens")
    ap.add_argument("--app-scope", action="store_true",
                    help="count the app limit per (app, replica) over all users (the other "
                         "reading of the paper's app key) instead of per (user, app)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="copy 1 GiB on the device first (calibrates rocprofv3 byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the policy's replicas are independent and this "
              f"build measures one GPU's share (asked for --gpus {args.gpus})", file=sys.stderr)
        sys.exit(2)
    if args.cpu_protocol:
        cpu_protocol(args.cpu_threads)
        return

    import numpy as np
    import torch

    import paper_2411_15997_amd as fs
    import tracegen as tg

    wl = tg.WORKLOADS[args.workload]
    t0 = time.time()
    tr = tg.generate(wl)
    print(f"[bench] generated {wl.name}: {tr.n} requests in {time.time() - t0:.1f}s",
          file=sys.stderr, flush=True)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    dt = fs.DeviceTrace(tr, device=dev)
    throttle_only = wl.throttle_only
    t_user, t_app, theta, fcfs, blind, equal = policy_settings(wl, tr.n_apps, args.policy)
    lim = fs.make_limits(wl.window_us, t_user, t_app, app_scope=1 if args.app_scope else 0)
    N = tr.n
    err = fs.err_word(dev)
    tws = torch.empty(max(fs.fs_throttle_workspace(dt), 1), dtype=torch.uint8, device=dev)
    literal = args.engine == "literal"
    if not throttle_only:
        coef, per_rep = fs.workload_weights(wl, tr)
        if equal:
            coef, per_rep = np.full((1, tr.n_apps, coef.shape[-2], 3), 1 << 16, np.int64), False
        w, keep = fs.make_weights(dt, coef, None, per_rep)
        eng = fs.make_engine(args.decode_step_us if literal else wl.step_us,
                             args.kv_tokens if literal else wl.cap_tokens, theta, fcfs=fcfs,
                             blind=blind, literal=literal)
        out = fs.Outputs(dt, parity=False)
        cost = torch.empty(max(N, 1), dtype=torch.int64, device=dev)
        state = torch.empty(fs.fs_state_bytes(dt), dtype=torch.uint8, device=dev)
        mws = torch.empty(max(fs.fs_metrics_workspace(dt), 1), dtype=torch.uint8, device=dev)
        metrics = fs.Metrics(dt)

    if args.calib_copy:
        src = torch.ones(1 << 28, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    stages = ["throttle"] if throttle_only else ["cost", "throttle", "init", "schedule", "metrics"]
    if args.stage_only:
        stages = [args.stage_only]
    J = wl.n_stages

    # the throttle's raw reasons feed the scheduler (same buffers every step)
    bitmap = torch.empty((N + 31) // 32 + 1, dtype=torch.int32, device=dev)
    reason_buf = None if throttle_only else torch.empty(max(N, 1), dtype=torch.uint8, device=dev)

    def step(evs):
        i = 0
        if "cost" in stages:
            evs[i].record(); i += 1
            fs.fs_cost(dt, w, cost, err, check=False)
        if "throttle" in stages:
            evs[i].record(); i += 1
            fs.fs_throttle(dt, lim, raw=not throttle_only, ws=tws, err=err, check=False,
                           bitmap=bitmap, reason=reason_buf)
        if "init" in stages:
            evs[i].record(); i += 1
            fs.fs_state_init(dt, state)
        if "schedule" in stages:
            evs[i].record(); i += 1
            fs.fs_schedule_step(dt, state, cost, reason_buf, eng, out, -1, check=False)
        if "metrics" in stages:
            evs[i].record(); i += 1
            fs.fs_fairness_metrics(dt, cost, out, eng, 0, metrics, mws, check=False)
        if "history" in stages:
            evs[i].record(); i += 1
            fs.fs_weights_from_history(dt, J, K=wl.weight_K, base_limit=30, err=err, check=False)
        if "workload" in stages:
            evs[i].record(); i += 1
            fs.fs_workload_stats(dt, 60_000_000, out=wstat, ws=wstat_ws, err=err, check=False)
        evs[i].record()

    wstat = wstat_ws = None
    if args.stage_only == "workload":
        wstat = fs.WorkloadStats(dt)
        wstat_ws = torch.empty(max(fs.fs_workload_workspace(dt), 1), dtype=torch.uint8, device=dev)
    if args.stage_only == "schedule":
        stages = ["init", "schedule"]
    if args.stage_only in ("schedule", "metrics"):
        fs.fs_cost(dt, w, cost, err)
        fs.fs_throttle(dt, lim, raw=True, ws=tws, err=err, bitmap=bitmap, reason=reason_buf)
        if args.stage_only == "metrics":
            fs.fs_state_init(dt, state)
            fs.fs_schedule_step(dt, state, cost, reason_buf, eng, out, -1)

    ne = len(stages) + 1
    for _ in range(args.warmup):
        step([torch.cuda.Event(enable_timing=True) for _ in range(ne)])
    torch.cuda.synchronize()
    fs.sync_check(out.err if ("schedule" in stages or "metrics" in stages) else err, "warmup")
    runs = []
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for _ in range(args.steps):
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(ne)]
        step(evs)
        runs.append(evs)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    fs.sync_check(out.err if ("schedule" in stages or "metrics" in stages) else err,
                  "timed steps")
    # per-stage medians over the timed steps (HIP events on the launch stream)
    stage_ms = {s: median([r[i].elapsed_time(r[i + 1]) for r in runs])
                for i, s in enumerate(stages)}
    step_ms_med = median([r[0].elapsed_time(r[-1]) for r in runs])
    ms_per_step = wall * 1000.0 / args.steps

    R = tr.n_replicas
    decisions = int(out.decisions.cpu().numpy().sum()) if "schedule" in stages else 0
    result = {
        "metric": METRIC,
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int64", "data": "synthetic",
        "config": {"workload": wl.name, "policy": args.policy, "engine": args.engine,
                   "replicas": R, "users": tr.n_users, "apps": tr.n_apps,
                   "requests": N, "trace_sha256": tr.sha256()[:16],
                   "step_us": int(eng.step_us) if not throttle_only else wl.step_us,
                   "cap_tokens": int(eng.cap_tokens) if not throttle_only else wl.cap_tokens,
                   "window_us": wl.window_us},
        "ms_per_step_median_events": round(step_ms_med, 4),
        "stages_ms": {k: round(v, 4) for k, v in stage_ms.items()},
    }
    if args.app_scope:
        result["config"]["app_scope"] = "per (app, replica)"
    if "schedule" in stages:
        result["value"] = decisions / (ms_per_step / 1000.0)
        result["unit"] = "decisions/s"
        result["decisions"] = decisions
        result["decisions_per_s_median"] = decisions / (stage_ms["schedule"] / 1000.0)
    elif "throttle" in stage_ms:
        result["value"] = N / (stage_ms["throttle"] / 1000.0)
        result["unit"] = "throttle evals/s"
    else:  # a profiling run of one other stage
        only = next(iter(stage_ms))
        result["value"] = N / (stage_ms[only] / 1000.0)
        result["unit"] = f"records/s through {only}"
    if "throttle" in stage_ms:
        result["throttle_evals_per_s"] = N / (stage_ms["throttle"] / 1000.0)
    result["requests_per_s"] = N / (ms_per_step / 1000.0)

    # algorithmic bytes per request of each stage for this trace and these outputs
    bpr = {s: algo_bytes(s, tr, raw=not throttle_only) for s in stage_ms}
    result["bytes_per_request"] = {s: v for s, v in bpr.items() if v > 0}
    # dominant stage and its roofline (algorithmic bytes / median duration)
    dom = max(stage_ms, key=stage_ms.get)
    limiter = None
    if dom == "schedule":
        limiter = ("latency of each replica's dependent decision chain: one wave per replica, "
                   f"{R} waves on 1,024 SIMDs")
    # the stored traffic was measured on the default policy and engine; the app-level
    # limit has its own entry, any other variant reports none
    tkey = None
    if args.policy == "fs" and args.engine == "step":
        tkey = wl.name + ("+app_scope" if args.app_scope else "")
    result["roofline"] = roofline(dom, bpr[dom] * N, stage_ms[dom], tkey, limiter)
    result["stage_gbs"] = {s: round(bpr[s] * N / (stage_ms[s] / 1000.0) / 1e9, 2)
                           for s in stage_ms if bpr[s] > 0}
    # stages whose algorithmic bytes fit the 256 MB Infinity Cache may be served from it
    result["mall_resident_stages"] = [s for s in stage_ms if 0 < bpr[s] * N < MALL_BYTES]

    if "metrics" in stages:  # the served-experience outcome of the policy (last step's metrics)
        mh = metrics.host()
        result["outcome"] = {"throttled": int(mh["throttled"].sum()),
                             "aborted_midway": int(mh["aborted_midway"].sum()),
                             "wasted_tokens": int(mh["wasted_tokens"].sum()),
                             "svc_int_pct": round(float(np.mean(mh["svc_int_pct"])), 3),
                             "served_users_pct": round(float(np.mean(mh["served_users_pct"])), 3),
                             "delayed_users_pct": round(float(np.mean(mh["delayed_users_pct"])), 3),
                             "jain": round(float(np.mean(mh["jain"])), 5)}
    if not throttle_only and not args.stage_only:
        # weights and app limits derived from this trace as a history (timed on its own)
        hist = []
        for it in range(args.warmup + args.steps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fs.fs_weights_from_history(dt, J, K=wl.weight_K, base_limit=30, err=err, check=False)
            e1.record()
            if it >= args.warmup:
                hist.append((e0, e1))
        torch.cuda.synchronize()
        fs.sync_check(err, "history")
        hms = median([a.elapsed_time(b) for a, b in hist])
        hb = algo_bytes("history", tr)
        hgbs = hb * N / (hms / 1000.0) / 1e9
        result["extra_stages"] = {"history": {"ms": round(hms, 4), "achieved_gbs": round(hgbs, 2),
                                              "frac": round(hgbs / HBM_PEAK_GBS, 4),
                                              "bytes_per_record": hb}}
        # the workload analysis of Sec. 3 on this trace (timed on its own)
        wout = fs.WorkloadStats(dt)
        wws = torch.empty(max(fs.fs_workload_workspace(dt), 1), dtype=torch.uint8, device=dev)
        wl_ev = []
        for it in range(args.warmup + args.steps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fs.fs_workload_stats(dt, 60_000_000, out=wout, ws=wws, err=err, check=False)
            e1.record()
            if it >= args.warmup:
                wl_ev.append((e0, e1))
        torch.cuda.synchronize()
        fs.sync_check(err, "workload stats")
        wms = median([a.elapsed_time(b) for a, b in wl_ev])
        wbytes = algo_bytes("workload", tr) * N + workload_out_bytes(tr)
        wgbs = wbytes / (wms / 1000.0) / 1e9
        result["extra_stages"]["workload"] = {"ms": round(wms, 4), "achieved_gbs": round(wgbs, 2),
                                              "frac": round(wgbs / HBM_PEAK_GBS, 4),
                                              "algorithmic_bytes": int(wbytes)}
        del wout, wws
    cpu = None
    if not args.no_cpu_baseline and not args.stage_only:
        cpu = cpu_baseline(wl, tr, args.cpu_threads, throttle_only, args.policy,
                           (args.decode_step_us, args.kv_tokens) if literal else None,
                           app_scope=1 if args.app_scope else 0)
        result["cpu_baseline"] = cpu

    # the throttle leg: fs_throttle on the largest throttle workload, own timed region
    if (args.throttle_workload != "none" and not throttle_only and not args.stage_only):
        del tws
        result["throttle_leg"] = throttle_leg(args, tg.WORKLOADS[args.throttle_workload], fs,
                                              torch, dev, not args.no_cpu_baseline)
    print(json.dumps(result), flush=True)


def throttle_leg(args, twl, fs, torch, dev, with_cpu):
    import numpy as np
    import tracegen as tg

    t0 = time.time()
    ttr = tg.generate(twl)
    print(f"[bench] generated {twl.name}: {ttr.n} requests in {time.time() - t0:.1f}s",
          file=sys.stderr, flush=True)
    tdt = fs.DeviceTrace(ttr, device=dev)
    tlim = fs.make_limits(twl.window_us, twl.t_user, twl.t_app)
    N = ttr.n
    tws = torch.empty(max(fs.fs_throttle_workspace(tdt), 1), dtype=torch.uint8, device=dev)
    bm = torch.empty((N + 31) // 32 + 1, dtype=torch.int32, device=dev)
    err = fs.err_word(dev)
    evs = []
    for it in range(args.warmup + args.steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        # gated mode with every request arriving while overloaded (NULL overload flags)
        fs.fs_throttle(tdt, tlim, raw=False, want_reason=False, ws=tws, err=err, check=False,
                       bitmap=bm)
        e1.record()
        if it >= args.warmup:
            evs.append((e0, e1))
    torch.cuda.synchronize()
    fs.sync_check(err, "throttle leg")
    ms = median([a.elapsed_time(b) for a, b in evs])
    b = algo_bytes("throttle", ttr, raw=False)
    leg = {"workload": twl.name, "requests": N, "users": ttr.n_users, "apps": ttr.n_apps,
           "trace_sha256": ttr.sha256()[:16], "mode": "gated, always overloaded",
           "runs": len(evs), "ms_median": round(ms, 4),
           "ms_min": round(min(a.elapsed_time(b_) for a, b_ in evs), 4),
           "value": N / (ms / 1000.0), "unit": "throttle evals/s", "bytes_per_request": b,
           "roofline": roofline("throttle", b * N, ms, twl.name)}
    throttled = int(np.unpackbits(bm.cpu().numpy().view(np.uint8), bitorder="little")[:N].sum())
    leg["throttled"] = throttled
    del tws, bm, tdt
    torch.cuda.empty_cache()
    if with_cpu:
        leg["cpu_baseline"] = cpu_throttle_baseline(twl, ttr)
    return leg


# ------------------------------------------------------------------ CPU oracle baselines

def _key_hashed_parts(tr, parts):
    """Splits a single-replica trace by user into `parts` traces (every key of the
    throttle is a user or a (user, app) pair, so each part's window counts are those
    of the whole stream); interaction links are renumbered within the part."""
    import numpy as np
    from tracegen import Trace

    sel = (tr.user.astype(np.int64) * 2654435761 % (1 << 32)) % parts
    out = []
    for p in range(parts):
        idx = np.nonzero(sel == p)[0]
        n = idx.shape[0]
        remap = None
        if tr.call is not None:
            remap = np.full(tr.n, -1, np.int64)
            remap[idx] = np.arange(n)
        cut = lambda a: None if a is None else np.ascontiguousarray(a[idx])
        head = None if tr.head is None else remap[tr.head[idx]].astype(np.int32)
        prev = None
        if tr.prev is not None:
            pv = tr.prev[idx]
            prev = np.where(pv >= 0, remap[np.maximum(pv, 0)], -1).astype(np.int32)
        out.append(Trace(1, tr.n_users, tr.n_apps, np.array([0, n], np.int64), cut(tr.ts_us),
                         cut(tr.user), cut(tr.app), cut(tr.call), head, prev, None, None, None))
    return out


def cpu_throttle_baseline(wl, tr, threads=0, app_scope=0):
    """The oracle's throttle (gated, always overloaded) on the whole stream: one thread,
    then users hashed over the host's threads (part construction not timed).  With the
    app limit counted over all users of an app, a request's two keys (its user, its app)
    cannot both stay within one part, so the stream runs on one thread only."""
    from concurrent.futures import ThreadPoolExecutor

    import oracle

    hc = host_cpu()
    th = threads or min(16, hc["available"])
    t0 = time.perf_counter()
    oracle.throttle(tr, wl.window_us, wl.t_user, wl.t_app, raw=False, counts=False,
                    app_scope=app_scope)
    one = time.perf_counter() - t0
    if app_scope:
        return {"value": tr.n / one, "unit": "throttle evals/s", "cores": 1, "kind": "oracle",
                "sample": f"whole {wl.name} stream ({tr.n} requests), app limit per (app, "
                          f"replica), one thread", "seconds": round(one, 3), "host": hc}
    parts = _key_hashed_parts(tr, th)
    t0 = time.perf_counter()
    with ThreadPoolExecutor(th) as ex:
        list(ex.map(lambda p: oracle.throttle(p, wl.window_us, wl.t_user, wl.t_app, raw=False,
                                              counts=False), parts))
    par = time.perf_counter() - t0
    return {"value": tr.n / par, "unit": "throttle evals/s", "cores": th, "kind": "oracle",
            "sample": f"whole {wl.name} stream ({tr.n} requests), users hashed over {th} threads",
            "seconds": round(par, 3),
            "single_thread": {"value": tr.n / one, "seconds": round(one, 3)},
            "host": hc}


def _oracle_path(wl, tr, th, policy, literal):
    import numpy as np

    import oracle

    if policy == "fs" and literal is None:
        c, thr, sim, met = oracle.run_workload(wl, tr, n_threads=th)
        return sim
    t_user, t_app, theta, fcfs, blind, equal = policy_settings(wl, tr.n_apps, policy)
    coef, per_rep = oracle.weights_for(wl, tr)
    if equal:
        coef, per_rep = np.full((1, tr.n_apps, coef.shape[-2], 3), 1 << 16, np.int64), False
    c = oracle.cost(tr, coef, coef_per_replica=per_rep)
    thr = oracle.throttle(tr, wl.window_us, t_user, t_app, raw=True, counts=False)
    flags = (oracle.FSO_FCFS if fcfs else 0) | (oracle.FSO_BLIND if blind else 0)
    step_us, cap = wl.step_us, wl.cap_tokens
    if literal is not None:
        flags |= oracle.FSO_LITERAL
        step_us, cap = literal
    sim = oracle.simulate(tr, c, thr.reason, step_us, cap, theta, n_threads=th, flags=flags)
    oracle.fairness_metrics(tr, c, sim.status, sim.admit_step, sim.max_gap, step_us)
    return sim


def cpu_baseline(wl, tr, threads, throttle_only, policy="fs", literal=None, app_scope=0):
    """The CPU oracle (as it stands) on this host, same workload, policy and engine
    (literal: (decode step, KV tokens) of the literal engine), whole path
    (cost + throttle + schedule + metrics): replicas split over the host's threads on
    the whole workload, and one thread on a bounded sample of replicas."""
    import tracegen as tg

    if throttle_only:
        return cpu_throttle_baseline(wl, tr, threads, app_scope)
    hc = host_cpu()
    th = threads or min(16, hc["available"], tr.n_replicas)
    t0 = time.perf_counter()
    sim = _oracle_path(wl, tr, th, policy, literal)
    dt = time.perf_counter() - t0
    dec = int(sim.decisions.sum())
    res = {"value": dec / dt, "unit": "decisions/s", "cores": th, "kind": "oracle",
           "sample": f"whole {wl.name} workload ({tr.n} requests, {tr.n_replicas} replicas), "
                     f"cost+throttle+schedule+metrics, replicas split over {th} threads",
           "seconds": round(dt, 3), "host": hc}
    # one thread on the first replicas (about 1.3M requests)
    k = max(1, min(tr.n_replicas, (1_300_000 + tr.n // tr.n_replicas - 1)
                   // max(1, tr.n // tr.n_replicas)))
    sub = tg.concat([tr.replica(r) for r in range(k)]) if k < tr.n_replicas else tr
    t0 = time.perf_counter()
    s1 = _oracle_path(wl, sub, 1, policy, literal)
    d1 = time.perf_counter() - t0
    res["single_thread"] = {"value": int(s1.decisions.sum()) / d1, "seconds": round(d1, 3),
                            "sample": f"first {k} of {tr.n_replicas} replicas ({sub.n} requests)"}
    return res


def cpu_protocol(threads=0):
    """The oracle on every workload: one thread each; replicas split over the host's
    threads (replica workloads); users hashed over the threads (throttle stream)."""
    import tracegen as tg

    hc = host_cpu()
    th = threads or min(16, hc["available"])
    rows = []
    for name, wl in tg.WORKLOADS.items():
        t0 = time.time()
        tr = tg.generate(wl)
        print(f"[cpu] generated {name}: {tr.n} requests in {time.time() - t0:.1f}s",
              file=sys.stderr, flush=True)
        if wl.throttle_only:
            r = cpu_throttle_baseline(wl, tr, th)
            rows.append({"workload": name, "requests": tr.n, "unit": "throttle evals/s",
                         "one_thread": r["single_thread"]["value"],
                         "one_thread_s": r["single_thread"]["seconds"],
                         "threads": th, "parallel": r["value"], "parallel_s": r["seconds"],
                         "split": "users hashed"})
        else:
            t0 = time.perf_counter()
            sim = _oracle_path(wl, tr, 1, "fs", None)
            one = time.perf_counter() - t0
            dec = int(sim.decisions.sum())
            row = {"workload": name, "requests": tr.n, "unit": "decisions/s",
                   "decisions": dec, "one_thread": dec / one, "one_thread_s": round(one, 3)}
            if tr.n_replicas > 1:
                t = min(th, tr.n_replicas)
                t0 = time.perf_counter()
                _oracle_path(wl, tr, t, "fs", None)
                par = time.perf_counter() - t0
                row.update(threads=t, parallel=dec / par, parallel_s=round(par, 3),
                           split="replicas")
            rows.append(row)
        print(json.dumps(rows[-1]), file=sys.stderr, flush=True)
    print(json.dumps({"cpu_protocol": rows, "host": hc}), flush=True)


if __name__ == "__main__":
    main()

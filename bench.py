"""Benchmark of the FairServe policy hot path on one MI355X.

One step = the whole path over one synthetic workload resident in HBM:
fs_cost -> fs_throttle (raw) -> fs_state_init -> fs_schedule_step (until drained)
-> fs_fairness_metrics, i.e. the sequence fs_run_trace runs plus the metrics.
Prints one JSON line (metric, value = scheduler decisions per second of the whole
step, per-stage times from HIP events, the roofline of the dominant kernel, and the
CPU oracle timed on this host on the same workload).
"""
import argparse
import hashlib
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "scheduler decisions/sec + throttle evals/sec on 1 MI355X; % of HBM roofline"
HBM_PEAK_GBS = 8000.0
# Algorithmic bytes per record of each stage (the minimum the method must move):
#   cost      app 4 + lengths 8 (+ sys 4) + cost write 8                       = 20 (24)
#   throttle  ts 8 + user 4 + app 4 + interaction link 4 + 1/8 bitmap bit       = 20.125
#   scheduler ts 8 + user 4 + link 4 + tokens 4 + cost 8 + reason 1/8 + status 1
#             + admit_step 4 + admit_seq 4                                      = 37.125
#   metrics   status 1 + admit_step 4 + ts 8 + user 4 + cost 8                  = 25
#   history   app 4 + call 4 + lengths 8 (+ sys 4) read once (weights from a history;
#             not part of the step, timed on its own)                         = 16 (20)
ALGO_BYTES = {"cost": 20.0, "throttle": 20.125, "init": 0.0, "schedule": 37.125, "metrics": 25.0,
              "history": 16.0}
CSRC = os.path.join(ROOT, "paper_2411_15997_amd", "csrc")
STAGE_SRC = {
    "cost": ["fs_cost.hip"],
    "throttle": ["fs_throttle.hip"],
    # the dominant kernel of the stage, k_schedule_onchip, and the header it shares
    "schedule": ["fs_sched_onchip.hip", "fs_sched_common.h"],
    "metrics": ["fs_metrics.hip"],
    "history": ["fs_history.hip"],
}

# HBM traffic of a stage's main kernel from rocprofv3 --pmc runs: FETCH_SIZE and
# WRITE_SIZE (KiB per dispatch), each scaled by bytes / counter of a plain 1 GiB
# device copy measured in the same run (bench.py --calib-copy).  Keyed by workload
# and stage; an entry counts only while the stage's sources hash to `src`.
MEASURED_TRAFFIC = {
    # k_schedule_onchip on the 64 x 256 x 8 replica workload (6.4M requests)
    ("c2_replicas", "schedule"): {"src": "e54b779cc0911a8b", "fetch_kib": 147786.3125,
                                  "write_kib": 38781.78125, "fetch_factor": 1.99993,
                                  "write_factor": 1.0},
    # k_schedule_onchip on the 1,024-replica weight sweep (20.48M requests)
    ("c4_sweep", "schedule"): {"src": "e54b779cc0911a8b", "fetch_kib": 353983.4375,
                               "write_kib": 137776.03125, "fetch_factor": 1.99988,
                               "write_factor": 1.0},
    # every kernel of one fs_throttle call on the 50M-request throttle stream
    ("c3_throttle", "throttle"): {"src": "e7d650dbb7b01d78", "fetch_kib": 2711800.6875,
                                  "write_kib": 2219110.96875, "fetch_factor": 1.99993,
                                  "write_factor": 1.0},
}



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


NO_LIMIT = 2 ** 31 - 1


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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c2_replicas")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-threads", type=int, default=0)
    ap.add_argument("--stage-only", default="", help="time only this stage (profiling runs): "
                    "cost, throttle, schedule, metrics or history")
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
    ap.add_argument("--calib-copy", action="store_true",
                    help="copy 1 GiB on the device first (calibrates rocprofv3 byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the policy's replicas are independent and this "
              f"build measures one GPU's share (asked for --gpus {args.gpus})", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2411_15997_amd as fs
    from paper_2411_15997_amd import tracegen as tg

    wl = tg.WORKLOADS[args.workload]
    t0 = time.time()
    tr = tg.generate(wl)
    gen_s = time.time() - t0
    print(f"[bench] generated {wl.name}: {tr.n} requests in {gen_s:.1f}s", file=sys.stderr, flush=True)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    dt = fs.DeviceTrace(tr, device=dev)
    throttle_only = wl.throttle_only
    t_user, t_app, theta, fcfs, blind, equal = policy_settings(wl, tr.n_apps, args.policy)
    lim = fs.make_limits(wl.window_us, t_user, t_app)
    N = tr.n
    err = fs.err_word(dev)
    tws = torch.empty(max(fs.fs_throttle_workspace(dt), 1), dtype=torch.uint8, device=dev)
    if not throttle_only:
        coef, per_rep = fs.workload_weights(wl, tr)
        if equal:
            coef, per_rep = np.full((1, tr.n_apps, coef.shape[-2], 3), 1 << 16, np.int64), False
        w, keep = fs.make_weights(dt, coef, None, per_rep)
        literal = args.engine == "literal"
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
    # bytes per record the history pass reads: app, lengths, call and system tokens if present
    ALGO_BYTES["history"] = 12.0 + (4.0 if tr.call is not None else 0.0) + (
        4.0 if tr.len_sys is not None else 0.0)

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
        evs[i].record()

    # the throttle's raw reasons feed the scheduler (same buffers every step)
    bitmap = torch.empty((N + 31) // 32 + 1, dtype=torch.int32, device=dev)
    reason_buf = None if throttle_only else torch.empty(max(N, 1), dtype=torch.uint8, device=dev)
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
    if "schedule" in stages or "metrics" in stages:
        fs.sync_check(out.err, "warmup")
    runs = []
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for _ in range(args.steps):
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(ne)]
        step(evs)
        runs.append(evs)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    if "schedule" in stages or "metrics" in stages:
        fs.sync_check(out.err, "timed steps")
    stage_ms = {s: float(np.mean([r[i].elapsed_time(r[i + 1]) for r in runs]))
                for i, s in enumerate(stages)}
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
        "stages_ms": {k: round(v, 4) for k, v in stage_ms.items()},
    }
    if "schedule" in stages:
        result["value"] = decisions / (ms_per_step / 1000.0)
        result["unit"] = "decisions/s"
        result["decisions"] = decisions
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

    # dominant stage and its roofline (algorithmic bytes / measured duration)
    dom = max(stage_ms, key=stage_ms.get)
    algo = ALGO_BYTES[dom] * N
    achieved = algo / (stage_ms[dom] / 1000.0) / 1e9
    traffic = measured_traffic(wl.name, dom)
    result["roofline"] = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 2),
                          "peak": HBM_PEAK_GBS, "unit": "GB/s",
                          "frac": round(achieved / HBM_PEAK_GBS, 6),
                          "algorithmic_bytes": int(algo), "traffic": traffic,
                          "src": src_hash(dom)}
    if dom == "schedule":
        # what limits it instead of bytes (measured with rocprofv3's SQ counters)
        result["roofline"]["limiter"] = (
            "latency of each replica's dependent decision chain: one wave per replica, "
            f"{wl.n_replicas} waves on 1,024 SIMDs")
    all_stage_gbs = {s: round(ALGO_BYTES[s] * N / (stage_ms[s] / 1000.0) / 1e9, 2)
                     for s in stage_ms if ALGO_BYTES[s] > 0}
    result["stage_gbs"] = all_stage_gbs

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
        hms = float(np.mean([a.elapsed_time(b) for a, b in hist]))
        hgbs = ALGO_BYTES["history"] * N / (hms / 1000.0) / 1e9
        result["extra_stages"] = {"history": {"ms": round(hms, 4), "achieved_gbs": round(hgbs, 2),
                                              "frac": round(hgbs / HBM_PEAK_GBS, 4),
                                              "bytes_per_record": ALGO_BYTES["history"]}}
    if not args.no_cpu_baseline and not args.stage_only:
        result["cpu_baseline"] = cpu_baseline(
            wl, tr, args.cpu_threads, throttle_only, args.policy,
            (args.decode_step_us, args.kv_tokens) if args.engine == "literal" else None)
    print(json.dumps(result), flush=True)


def cpu_baseline(wl, tr, threads, throttle_only, policy="fs", literal=None):
    """The CPU oracle (as it stands) on this host, same workload, policy and engine
    (literal: (decode step, KV tokens) of the literal engine), whole path."""
    import numpy as np

    import oracle

    ncpu = os.cpu_count() or 1
    th = threads or min(16, ncpu, tr.n_replicas) if not throttle_only else 1
    t0 = time.perf_counter()
    if throttle_only:
        # bounded sample: the first 5M requests of the stream
        from paper_2411_15997_amd.tracegen import Trace
        n = min(tr.n, 5_000_000)
        sub = Trace(1, tr.n_users, tr.n_apps, np.array([0, n], np.int64), tr.ts_us[:n],
                    tr.user[:n], tr.app[:n], tr.call[:n], tr.head[:n], tr.prev[:n],
                    None, None, None)
        oracle.throttle(sub, wl.window_us, wl.t_user, wl.t_app, raw=False, counts=False)
        dt = time.perf_counter() - t0
        return {"value": n / dt, "unit": "throttle evals/s", "cores": 1, "kind": "oracle",
                "sample": f"first {n} requests of {wl.name}", "seconds": round(dt, 3),
                "host": platform.processor() or platform.machine()}
    if policy == "fs" and literal is None:
        c, thr, sim, met = oracle.run_workload(wl, tr, n_threads=th)
    else:
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
    dt = time.perf_counter() - t0
    dec = int(sim.decisions.sum())
    return {"value": dec / dt, "unit": "decisions/s", "cores": th, "kind": "oracle",
            "sample": f"whole {wl.name} workload ({tr.n} requests, {tr.n_replicas} replicas), "
                      f"cost+throttle+schedule+metrics",
            "seconds": round(dt, 3), "host_cpus": ncpu}


if __name__ == "__main__":
    main()

"""Brute-force restatement of the policy for tiny traces (pins the oracle).

Every quantity is recomputed from scratch at every use: window counts scan
all earlier requests, the backlogged set X and the set of users with a ready
later call are rebuilt before every decision, and the argmin scans every user.
Python integers make the fixed-point cost exact.  Sources: Alg. 1 (both
streams), Eq. 2, Sec. 4 (OIT and WSC prose).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

VALUE_LIMIT = 1 << 62


def _first(tr, g):
    return tr.call is None or int(tr.call[g]) == 0


def cost(tr, coef, prio=None, coef_per_replica=False):
    """Eq. 2 for one call: floor(E * (c_in L_I + c_sys L_S + c_out L_O) / 256)."""
    out = []
    J = coef.shape[-2]
    for r in range(tr.n_replicas):
        for g in range(int(tr.rep_off[r]), int(tr.rep_off[r + 1])):
            a = int(tr.app[g])
            j = 0 if tr.call is None else min(int(tr.call[g]), J - 1)
            c = coef[r if coef_per_replica else 0][a][j]
            E = 256 if prio is None else int(prio[int(tr.user[g])])
            L_I = int(tr.len_in[g])
            L_S = 0 if tr.len_sys is None else int(tr.len_sys[g])
            L_O = int(tr.len_out[g])
            v = (E * (int(c[0]) * L_I + int(c[1]) * L_S + int(c[2]) * L_O)) // 256
            out.append(v)
    return out


def window_counts(tr, window_us, app_scope=0):
    """c_user(i), c_app(i): requests j <= i of the same key with ts_j > ts_i - W (the app
    key is (user, app), or the app alone when app_scope is 1)."""
    cu, ca = [], []
    for r in range(tr.n_replicas):
        a0, a1 = int(tr.rep_off[r]), int(tr.rep_off[r + 1])
        for i in range(a0, a1):
            lo = int(tr.ts_us[i]) - window_us
            nu = na = 0
            for j in range(a0, i + 1):
                if int(tr.ts_us[j]) > lo:
                    same_user = tr.user[j] == tr.user[i]
                    nu += 1 if same_user else 0
                    if tr.app[j] == tr.app[i] and (same_user or app_scope):
                        na += 1
            cu.append(nu)
            ca.append(na)
    return cu, ca


def throttle_raw(tr, window_us, t_user, t_app, app_scope=0):
    cu, ca = window_counts(tr, window_us, app_scope)
    return [1 if cu[g] > t_user else (2 if ca[g] > t_app[int(tr.app[g])] else 0)
            for g in range(len(cu))]


def throttle_gated(tr, window_us, t_user, t_app, overloaded=None):
    raw = throttle_raw(tr, window_us, t_user, t_app)
    out = [0] * len(raw)
    for r in range(tr.n_replicas):
        base = int(tr.rep_off[r])
        for g in range(base, int(tr.rep_off[r + 1])):
            if _first(tr, g):
                over = True if overloaded is None else bool(overloaded[g])
                out[g] = raw[g] if over else 0
            else:
                out[g] = 3 if out[base + int(tr.head[g])] else 0
    return out


@dataclass
class Result:
    status: List[int]
    admit_step: List[int]
    admit_seq: List[int]
    counter_after: List[int]
    counter_on_arrival: List[int]
    counter: List[int]
    steps: List[int]
    decisions: List[int]
    max_gap: List[int]
    trace_of_counters: list = field(default_factory=list)  # (step, seq, {user: u}) per decision


FCFS, BLIND, LITERAL = 1, 2, 4  # engine flags: first come first served; interaction-blind
# limits; the literal engine (prefill at admission, one output token per step, charge at finish)


def simulate(tr, cost_arr, reason, step_us, cap, theta, max_steps=-1, record_states=False,
             flags=0):
    n_all = tr.n
    res = Result([-1] * n_all, [-1] * n_all, [-1] * n_all, [-1] * n_all, [-1] * n_all,
                 [0] * (tr.n_replicas * tr.n_users), [], [], [])
    for r in range(tr.n_replicas):
        base, end = int(tr.rep_off[r]), int(tr.rep_off[r + 1])
        n = end - base
        U = tr.n_users
        u = [0] * U
        queued: List[int] = []          # replica-local indices, any order
        served = [False] * n
        aborted = [False] * n
        dropped = [False] * n
        last_exit: Optional[int] = None
        debt = backlog = seq = gap = 0
        running: List[list] = []        # literal engine: [record, last decode step], by admission
        nxt = 0
        s = 0
        G = lambda i: base + i
        tok = lambda i: (int(tr.len_in[G(i)]) + (0 if tr.len_sys is None else int(tr.len_sys[G(i)]))
                         + int(tr.len_out[G(i)]))

        def X():
            return sorted({int(tr.user[G(i)]) for i in queued})

        def ready_calls():
            return [i for i in queued if not _first(tr, G(i)) and served[int(tr.prev[G(i)])]]

        while True:
            if 0 <= max_steps <= s:
                break
            if nxt == n and not queued and not running:
                break
            # arrivals of step s (an idle step changes nothing but the debt)
            while nxt < n and int(tr.ts_us[G(nxt)]) // step_us <= s:
                i = nxt
                nxt += 1
                k = int(tr.user[G(i)])
                xs = X()
                if k not in xs:
                    if not xs:
                        if last_exit is not None:
                            u[k] = max(u[k], u[last_exit])
                    else:
                        u[k] = max(u[k], min(u[x] for x in xs))
                res.counter_on_arrival[G(i)] = u[k]
                if not _first(tr, G(i)) and not flags & BLIND:
                    blocked, code = aborted[int(tr.head[G(i)])], 3
                elif not _first(tr, G(i)) and dropped[int(tr.prev[G(i)])]:
                    blocked, code = True, 3
                else:
                    why = 0 if reason is None else int(reason[G(i)])
                    blocked, code = (backlog > theta and why != 0), why
                if blocked:
                    res.status[G(i)] = code
                    dropped[i] = True
                    if _first(tr, G(i)):
                        aborted[i] = True
                else:
                    queued.append(i)
                    backlog += tok(i)
            budget = cap + debt
            kv = sum(tok(i) for i, _ in running)
            while (flags & LITERAL or budget > 0) and queued:
                ready = ready_calls()
                if flags & FCFS:  # the earliest queued request, whoever it belongs to
                    rcand = min(queued)
                    k = int(tr.user[G(rcand)])
                    assert _first(tr, G(rcand)) or rcand in ready
                elif ready:
                    users = sorted({int(tr.user[G(i)]) for i in ready})
                    k = min(users, key=lambda x: (u[x], x))
                    rcand = min(i for i in ready if int(tr.user[G(i)]) == k)
                else:
                    users = X()
                    k = min(users, key=lambda x: (u[x], x))
                    rcand = min(i for i in queued if int(tr.user[G(i)]) == k)
                if flags & LITERAL and running and kv + tok(rcand) > cap:
                    break                   # the chosen call does not fit in the KV cache
                queued.remove(rcand)
                served[rcand] = True
                res.status[G(rcand)] = 0
                budget -= tok(rcand)
                backlog -= tok(rcand)
                if flags & LITERAL:         # charged when its last output token is decoded
                    running.append([rcand, s + max(int(tr.len_out[G(rcand)]), 1) - 1])
                    kv += tok(rcand)
                else:
                    u[k] += int(cost_arr[G(rcand)])
                    if u[k] >= VALUE_LIMIT:
                        raise OverflowError("counter overflow")
                    res.counter_after[G(rcand)] = u[k]
                res.admit_step[G(rcand)] = s
                res.admit_seq[G(rcand)] = seq
                seq += 1
                if k not in X():
                    last_exit = k
                if record_states:
                    res.trace_of_counters.append((s, seq - 1, {x: u[x] for x in X()}, bool(ready), k))
            if flags & LITERAL:
                for rec, fin in running:
                    if fin == s:
                        kk = int(tr.user[G(rec)])
                        u[kk] += int(cost_arr[G(rec)])
                        if u[kk] >= VALUE_LIMIT:
                            raise OverflowError("counter overflow")
                        res.counter_after[G(rec)] = u[kk]
                running = [x for x in running if x[1] != s]
            else:
                debt = min(budget, 0)
            xs = X()
            if xs:
                gap = max(gap, max(u[x] for x in xs) - min(u[x] for x in xs))
            s += 1
        for k in range(U):
            res.counter[r * U + k] = u[k]
        res.steps.append(s)
        res.decisions.append(seq)
        res.max_gap.append(gap)
    return res

"""Every trace with at most 2 users and 5 requests, tokens 1 to 3 and arrival steps 0
to 2, as one replica-batched launch (each trace one replica, 185,130 of them), at
capacities 2 and 4 tokens per step and user limits 1 and 2 in a two-step window:
throttle reasons, window counts and every scheduler output bit-exact against the
oracle (the survey's exhaustive small layer); also on the global-memory path, under the
literal engine and under the rate-limit policy."""
import itertools

import numpy as np
import pytest

import oracle
import tracegen as tg
from gpu_common import compare_sim, gpu_schedule, gpu_throttle, say

pytestmark = pytest.mark.gpu

STEP = 1000          # one step, in microseconds
WINDOW = 2 * STEP    # the limit's window
THETA = 1            # overloaded while more than one token is queued
NO_LIMIT = 2 ** 31 - 1
_GRID = None


def grid_trace():
    """All (users, tokens, nondecreasing steps) of 1 to 5 requests, one replica each."""
    global _GRID
    if _GRID is not None:
        return _GRID
    users, toks, steps, sizes = [], [], [], []
    for n in range(1, 6):
        S = np.array([s for s in itertools.product(range(3), repeat=n)
                      if all(s[i] <= s[i + 1] for i in range(n - 1))], np.int64)
        Us = np.array(list(itertools.product(range(2), repeat=n)), np.int32)
        Ts = np.array(list(itertools.product((1, 2, 3), repeat=n)), np.int32)
        iu, it, is_ = (a.ravel() for a in np.meshgrid(np.arange(len(Us)), np.arange(len(Ts)),
                                                     np.arange(len(S)), indexing="ij"))
        users.append(Us[iu].ravel())
        toks.append(Ts[it].ravel())
        steps.append(S[is_].ravel())
        sizes.append(np.full(iu.size, n, np.int64))
    sizes = np.concatenate(sizes)
    rep_off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    n = int(rep_off[-1])
    tok = np.concatenate(toks).astype(np.int32)
    _GRID = tg.Trace(int(sizes.size), 2, 1, rep_off, np.concatenate(steps) * STEP,
                     np.concatenate(users).astype(np.int32), np.zeros(n, np.int32), None, None,
                     None, tok, None, np.zeros(n, np.int32))
    return _GRID


def test_grid_shape():
    tr = grid_trace()
    assert tr.n_replicas == 185_130 and tr.n == 901_170


@pytest.mark.parametrize("cap,t_user,global_only", [(2, 1, False), (2, 2, False), (4, 1, False),
                                                    (4, 2, False), (2, 1, True)])
def test_exhaustive_grid_one_launch(cap, t_user, global_only):
    tr = grid_trace()
    say("exhaustive grid", tr.n_replicas, tr.n, cap, t_user, global_only)
    ot = oracle.throttle(tr, WINDOW, t_user, [NO_LIMIT], raw=True, counts=True)
    gt = gpu_throttle(tr, WINDOW, t_user, [NO_LIMIT], raw=True, counts=True)
    for k, w in (("reason", ot.reason), ("cnt_user", ot.cnt_user), ("cnt_app", ot.cnt_app)):
        bad = np.nonzero(gt[k] != w)[0]
        assert bad.size == 0, f"{k}: {bad.size} mismatches, first {bad[:5]}"
    cost = tr.len_in.astype(np.int64)
    o = oracle.simulate(tr, cost, ot.reason, STEP, cap, THETA)
    compare_sim(gpu_schedule(tr, cost, ot.reason, STEP, cap, THETA, global_only=global_only), o)


@pytest.mark.parametrize("mode", ["literal", "rate_limit"])
def test_exhaustive_grid_other_engines(mode):
    """The same grid under the literal engine (KV capacity 4 tokens, charge at finish)
    and under the rate-limit policy (first come first served, interaction-blind, always
    overloaded)."""
    tr = grid_trace()
    cost = tr.len_in.astype(np.int64)
    say("exhaustive grid", mode)
    if mode == "literal":
        ot = oracle.throttle(tr, WINDOW, 2, [NO_LIMIT], raw=True, counts=False)
        o = oracle.simulate(tr, cost, ot.reason, STEP, 4, THETA, flags=oracle.FSO_LITERAL)
        g = gpu_schedule(tr, cost, ot.reason, STEP, 4, THETA, literal=True)
    else:
        ot = oracle.throttle(tr, WINDOW, 1, [NO_LIMIT], raw=True, counts=False)
        o = oracle.simulate(tr, cost, ot.reason, STEP, 2, -1,
                            flags=oracle.FSO_FCFS | oracle.FSO_BLIND)
        g = gpu_schedule(tr, cost, ot.reason, STEP, 2, -1, fcfs=True, blind=True)
    compare_sim(g, o)

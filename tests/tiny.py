"""Small hand-written and random traces for the pin and parity tests."""
from __future__ import annotations

import json
import os

import numpy as np

from tracegen import Trace, concat

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load_golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def trace_from_case(c, n_apps=1):
    n = len(c["ts"])
    arr = lambda k, dt=np.int32: None if c.get(k) is None else np.asarray(c[k], dt)
    tok = np.asarray(c["tok"], np.int32) if "tok" in c else np.ones(n, np.int32)
    return Trace(1, c["U"], n_apps, np.array([0, n], np.int64), np.asarray(c["ts"], np.int64),
                 np.asarray(c["user"], np.int32),
                 arr("app") if c.get("app") is not None else np.zeros(n, np.int32),
                 arr("call"), arr("head"), arr("prev"), tok, None, np.zeros(n, np.int32))


def random_trace(rng, n, U, A, ts_span, multi=True, max_tok=5, n_replicas=1):
    """Random valid trace; interactions are chains of calls of one user and app."""
    reps = []
    for _ in range(n_replicas):
        ts = np.sort(rng.integers(0, max(1, ts_span), size=n)).astype(np.int64)
        user = rng.integers(0, U, size=n).astype(np.int32)
        app = rng.integers(0, A, size=n).astype(np.int32)
        call = np.zeros(n, np.int32)
        head = np.arange(n, dtype=np.int32)
        prev = np.full(n, -1, np.int32)
        if multi:
            # link some requests to an earlier open interaction of the same user
            last_of_user = {}
            for i in range(n):
                k = int(user[i])
                if k in last_of_user and rng.random() < 0.5:
                    p = last_of_user[k]
                    call[i] = call[p] + 1
                    head[i] = head[p]
                    prev[i] = p
                    app[i] = app[p]
                last_of_user[k] = i
        lin = rng.integers(0, max_tok + 1, size=n).astype(np.int32)
        lsys = rng.integers(0, max_tok + 1, size=n).astype(np.int32)
        lout = rng.integers(0, max_tok + 1, size=n).astype(np.int32)
        reps.append(Trace(1, U, A, np.array([0, n], np.int64), ts, user, app,
                          call if multi else None, head if multi else None,
                          prev if multi else None, lin, lsys, lout))
    return concat(reps)

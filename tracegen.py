"""Seeded synthetic multi-tenant LLM request traces.

The paper evaluates on a proprietary one-day production trace that is not
available.  This module builds synthetic stand-ins with the shapes the paper
states in prose: per-application token diversity (Sec. 3, input- vs
output-heavy apps), 1 to 20 chained LLM calls per interaction (Sec. 3,
Fig. 4 discussion and Table 2), calls spread out in time, system prompts
(Sec. 3, Fig. 5 discussion) and heavy-tailed per-user activity (Sec. 3,
Fig. 2 discussion).

This module is shared by the CPU oracle's tests and the HIP path's tests and
benchmark; it lives outside both (the oracle and the library import nothing from
each other, and neither imports it for arithmetic).  It holds
none of the method's arithmetic: no cost, no window counting, no weights.
It only draws random requests and records the workload constants (limits,
engine capacity, expected token counts) that the method takes as inputs.

Layout produced (structure of arrays, replicas concatenated):
  ts_us  int64  arrival time in microseconds, non-decreasing per replica
  user   int32  [0, U)
  app    int32  [0, A)
  call   int32  stage j of the interaction, 0 for its first call
  head   int32  replica-local index of the interaction's first call (itself for a first call)
  prev   int32  replica-local index of call j-1, -1 for a first call
  len_in, len_sys, len_out int32 token counts (len_sys may be absent)
"""
from __future__ import annotations

import dataclasses
import hashlib
import math
from typing import List, Optional, Sequence

import numpy as np

US_PER_S = 1_000_000
INT32_MAX = 2**31 - 1
Q16 = 1 << 16


# ----------------------------------------------------------------------------
# workload descriptions
# ----------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class TokenDist:
    """Lognormal token count, rounded half-even to an int and clipped.

    Either ``mu`` is given directly, or ``mean`` is and mu = ln(mean) - sigma^2/2.
    ``mean`` may be a per-app list; ``stage_slope`` multiplies the mean by
    (1 + j * stage_slope) at stage j.
    """
    sigma: float
    lo: int
    hi: int
    mu: Optional[float] = None
    mean: Optional[Sequence[float]] = None
    stage_slope: float = 0.0

    def mean_of(self, app: int, stage: int) -> float:
        """Nominal (unclipped) expectation for app ``app`` at stage ``stage``."""
        if self.mu is not None:
            return math.exp(self.mu + 0.5 * self.sigma ** 2)
        return float(self.mean[app]) * (1.0 + stage * self.stage_slope)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    config_id: int
    n_replicas: int
    n_users: int
    n_apps: int
    records_per_replica: int
    horizon_s: float
    # per-user activity
    zipf_s: Optional[float]           # None => explicit rates
    user_rates: Optional[Sequence[float]]
    n_abusive: int
    abuse_mult: float
    diurnal: bool
    # calls per interaction
    calls_kind: str                   # "one" | "geom" | "table2"
    geom_p: Optional[Sequence[float]] = None   # per app
    # tokens
    tok_in: Optional[TokenDist] = None
    tok_out: Optional[TokenDist] = None
    tok_sys: Optional[TokenDist] = None
    # weights: either direct Q16 table or expectations for Eq. 1
    n_stages: int = 1
    coef_direct: Optional[Sequence[Sequence[int]]] = None  # [A][3] Q16 {in,sys,out}
    coef_grid_per_replica: bool = False                    # weight sweep (one (w_in,w_out) per replica)
    weight_K: int = 1024
    # limits
    window_s: float = 60.0
    t_user: int = INT32_MAX
    t_app: Sequence[int] = ()
    # engine
    step_ms: float = 250.0
    cap_tokens: int = 16384
    overload_tokens: Optional[int] = None   # None => all overloaded (throttle-only workload)
    throttle_only: bool = False
    seed: int = 0

    @property
    def n_records(self) -> int:
        return self.n_replicas * self.records_per_replica

    @property
    def window_us(self) -> int:
        return int(round(self.window_s * US_PER_S))

    @property
    def step_us(self) -> int:
        return int(round(self.step_ms * 1000))

    def direct_coef_table(self, trace) -> Optional[np.ndarray]:
        """The Q16 table this workload fixes directly (None: derive it with Eq. 1)."""
        return coef_direct_table(self, trace)

    def expectations(self):
        """Nominal expected token counts per (app, stage): arrays [A][J] for in, sys, out."""
        A, J = self.n_apps, self.n_stages
        e_in = np.zeros((A, J))
        e_sys = np.zeros((A, J))
        e_out = np.zeros((A, J))
        for a in range(A):
            for j in range(J):
                e_in[a, j] = self.tok_in.mean_of(a, j) if self.tok_in else 0.0
                e_sys[a, j] = self.tok_sys.mean_of(a, j) if self.tok_sys else 0.0
                e_out[a, j] = self.tok_out.mean_of(a, j) if self.tok_out else 0.0
        return e_in, e_sys, e_out


def _c2_means():
    mi = [200.0 * 20.0 ** (a / 7.0) for a in range(8)]
    mo = [200.0 * 20.0 ** ((7 - a) / 7.0) for a in range(8)]
    return mi, mo


def _c5_means():
    mi = [200.0 * 32.0 ** (a / 31.0) for a in range(32)]
    mo = [30.0 * 20.0 ** (((13 * a) % 32) / 31.0) for a in range(32)]
    ms = [50.0 * 40.0 ** (a / 31.0) for a in range(32)]
    return mi, mo, ms


_MI2, _MO2 = _c2_means()
_MI5, _MO5, _MS5 = _c5_means()

# Table 2 of the paper gives the share of REQUESTS by interaction size; only the
# first three bins carry mass that matters at these sizes.  Renormalised over
# those bins.
TABLE2_BINS = ((1, 1, 73.22), (2, 10, 26.09), (11, 20, 0.50))

WORKLOADS = {
    # 1 replica x 8 users x 2 apps, 2,000 single-call requests over 60 s.
    "c1_small": Workload(
        name="c1_small", config_id=0, n_replicas=1, n_users=8, n_apps=2,
        records_per_replica=2000, horizon_s=60.0,
        zipf_s=None, user_rates=[0.5] * 7 + [20.0], n_abusive=0, abuse_mult=1.0, diurnal=False,
        calls_kind="one",
        tok_in=TokenDist(mu=6.0, sigma=1.0, lo=1, hi=8192),
        tok_out=TokenDist(mu=5.0, sigma=1.0, lo=1, hi=4096),
        coef_direct=[[1 * Q16, 2 * Q16, 2 * Q16], [1 * Q16, 2 * Q16, 4 * Q16]],
        window_s=10.0, t_user=INT32_MAX, t_app=[30, 30],
        step_ms=250.0, cap_tokens=4096, overload_tokens=4096, seed=0),
    # 64 replicas x 256 users x 8 apps, 100k requests per replica over 1 h.
    "c2_replicas": Workload(
        name="c2_replicas", config_id=1, n_replicas=64, n_users=256, n_apps=8,
        records_per_replica=100_000, horizon_s=3600.0,
        zipf_s=1.1, user_rates=None, n_abusive=13, abuse_mult=10.0, diurnal=False,
        calls_kind="geom", geom_p=[1.0, 1.0, 0.7, 0.5, 0.5, 0.3, 0.3, 0.2],
        tok_in=TokenDist(mean=_MI2, sigma=1.0, lo=1, hi=32768),
        tok_out=TokenDist(mean=_MO2, sigma=1.0, lo=1, hi=32768),
        window_s=60.0, t_user=240, t_app=[30, 30, 43, 60, 60, 100, 100, 149],
        step_ms=250.0, cap_tokens=16384, overload_tokens=16384, seed=0),
    # throttle-only stream: 50M requests, 10,000 users, 16 apps.
    "c3_throttle": Workload(
        name="c3_throttle", config_id=2, n_replicas=1, n_users=10_000, n_apps=16,
        records_per_replica=50_000_000, horizon_s=3600.0,
        zipf_s=1.1, user_rates=None, n_abusive=500, abuse_mult=10.0, diurnal=False,
        calls_kind="geom", geom_p=[0.3] * 16,
        window_s=60.0, t_user=300, t_app=[100] * 16,
        overload_tokens=None, throttle_only=True, seed=0),
    # weight sweep: 1,024 replicas x 1,024 users x 8 apps, 20k requests each.
    "c4_sweep": Workload(
        name="c4_sweep", config_id=3, n_replicas=1024, n_users=1024, n_apps=8,
        records_per_replica=20_000, horizon_s=600.0,
        zipf_s=1.1, user_rates=None, n_abusive=51, abuse_mult=10.0, diurnal=False,
        calls_kind="one",
        tok_in=TokenDist(mean=_MI2, sigma=1.0, lo=1, hi=32768),
        tok_out=TokenDist(mean=_MO2, sigma=1.0, lo=1, hi=32768),
        coef_grid_per_replica=True,
        window_s=60.0, t_user=120, t_app=[30] * 8,
        step_ms=200.0, cap_tokens=16384, overload_tokens=16384, seed=0),
    # large tenant: 1 replica, 100,000 users, 32 apps, 10M requests over 24 h.
    "c5_tenant": Workload(
        name="c5_tenant", config_id=4, n_replicas=1, n_users=100_000, n_apps=32,
        records_per_replica=10_000_000, horizon_s=86_400.0,
        zipf_s=1.2, user_rates=None, n_abusive=1000, abuse_mult=50.0, diurnal=True,
        calls_kind="table2",
        tok_in=TokenDist(mean=_MI5, sigma=0.5, lo=1, hi=65536, stage_slope=0.25),
        tok_sys=TokenDist(mean=_MS5, sigma=0.5, lo=1, hi=65536),
        tok_out=TokenDist(mean=_MO5, sigma=0.5, lo=1, hi=16384),
        n_stages=20,
        window_s=60.0, t_user=300, t_app=[38] * 32,
        step_ms=160.0, cap_tokens=65536, overload_tokens=65536, seed=0),
}

# Weight-sweep grid: (w_in, w_out) each on {1, 1+1/16, ..., 8} (113 points), Q16.
SWEEP_GRID_Q16 = [Q16 + k * (Q16 // 16) for k in range(113)]


def scaled(wl: Workload, replicas: Optional[int] = None, records: Optional[int] = None,
           users: Optional[int] = None, name: Optional[str] = None) -> Workload:
    """The same workload recipe at a smaller size (for parity tests the oracle finishes quickly).

    Shrinking the record count keeps the per-user request rates by shrinking
    the horizon in proportion.
    """
    kw = {}
    if replicas is not None:
        kw["n_replicas"] = replicas
    if records is not None:
        kw["records_per_replica"] = records
        kw["horizon_s"] = wl.horizon_s * records / wl.records_per_replica
    if users is not None:
        kw["n_users"] = users
        if wl.n_abusive:
            kw["n_abusive"] = max(1, int(round(wl.n_abusive * users / wl.n_users)))
    kw["name"] = name or (wl.name + "_scaled")
    return dataclasses.replace(wl, **kw)


# ----------------------------------------------------------------------------
# trace container
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class Trace:
    n_replicas: int
    n_users: int
    n_apps: int
    rep_off: np.ndarray           # int64 [R+1]
    ts_us: np.ndarray             # int64 [N]
    user: np.ndarray              # int32 [N]
    app: np.ndarray               # int32 [N]
    call: Optional[np.ndarray]    # int32 [N] or None (all first calls)
    head: Optional[np.ndarray]
    prev: Optional[np.ndarray]
    len_in: Optional[np.ndarray]
    len_sys: Optional[np.ndarray]
    len_out: Optional[np.ndarray]
    # per-replica sweep weights (Q16 w_in, w_out), weight-sweep workloads only
    sweep_w: Optional[np.ndarray] = None

    @property
    def n(self) -> int:
        return int(self.ts_us.shape[0])

    def arrays(self):
        return {k: v for k, v in dataclasses.asdict(self).items() if isinstance(v, np.ndarray)}

    def sha256(self) -> str:
        h = hashlib.sha256()
        for k in ("rep_off", "ts_us", "user", "app", "call", "head", "prev",
                  "len_in", "len_sys", "len_out", "sweep_w"):
            v = getattr(self, k)
            h.update(k.encode())
            if v is not None:
                h.update(np.ascontiguousarray(v).tobytes())
        return h.hexdigest()

    def replica(self, r: int) -> "Trace":
        a, b = int(self.rep_off[r]), int(self.rep_off[r + 1])
        sl = lambda x: None if x is None else x[a:b].copy()
        return Trace(1, self.n_users, self.n_apps, np.array([0, b - a], np.int64),
                     sl(self.ts_us), sl(self.user), sl(self.app), sl(self.call), sl(self.head),
                     sl(self.prev), sl(self.len_in), sl(self.len_sys), sl(self.len_out),
                     None if self.sweep_w is None else self.sweep_w[r:r + 1].copy())


def concat(traces: List[Trace]) -> Trace:
    """Concatenate single- or multi-replica traces into one multi-replica trace."""
    t0 = traces[0]
    offs = [0]
    for t in traces:
        for r in range(t.n_replicas):
            offs.append(offs[-1] + int(t.rep_off[r + 1] - t.rep_off[r]))

    def cat(name):
        xs = [getattr(t, name) for t in traces]
        if all(x is None for x in xs):
            return None
        if any(x is None for x in xs):
            raise ValueError(f"cannot concat: {name} missing in some traces")
        return np.concatenate(xs)

    return Trace(sum(t.n_replicas for t in traces), max(t.n_users for t in traces),
                 max(t.n_apps for t in traces), np.array(offs, np.int64),
                 cat("ts_us"), cat("user"), cat("app"), cat("call"), cat("head"), cat("prev"),
                 cat("len_in"), cat("len_sys"), cat("len_out"), cat("sweep_w"))


# ----------------------------------------------------------------------------
# generation
# ----------------------------------------------------------------------------

def _rng(wl: Workload, rep: int) -> np.random.Generator:
    ss = np.random.SeedSequence(entropy=wl.seed, spawn_key=(wl.config_id, rep))
    return np.random.Generator(np.random.PCG64(ss))


def _table2_sizes():
    """Interaction-size distribution whose REQUEST shares follow Table 2's bins."""
    sizes, probs = [], []
    for lo, hi, share in TABLE2_BINS:
        nb = hi - lo + 1
        for s in range(lo, hi + 1):
            sizes.append(s)
            probs.append(share / (nb * s))   # request share of size s = share / nb
    p = np.array(probs)
    return np.array(sizes, np.int64), p / p.sum()


def _calls(wl: Workload, rng: np.random.Generator, apps: np.ndarray) -> np.ndarray:
    n = apps.shape[0]
    if wl.calls_kind == "one":
        return np.ones(n, np.int64)
    if wl.calls_kind == "geom":
        p = np.asarray(wl.geom_p, np.float64)[apps]
        return np.minimum(20, rng.geometric(p)).astype(np.int64)
    if wl.calls_kind == "table2":
        sizes, probs = _table2_sizes()
        return sizes[rng.choice(sizes.shape[0], size=n, p=probs)]
    raise ValueError(wl.calls_kind)


def _lognormal(rng, dist: TokenDist, apps: np.ndarray, stages: np.ndarray) -> np.ndarray:
    if dist.mu is not None:
        mu = np.full(apps.shape[0], dist.mu)
    else:
        mean = np.asarray(dist.mean, np.float64)[apps] * (1.0 + stages * dist.stage_slope)
        mu = np.log(mean) - 0.5 * dist.sigma ** 2
    x = rng.lognormal(mean=mu, sigma=dist.sigma)
    return np.clip(np.rint(x), dist.lo, dist.hi).astype(np.int32)


def _diurnal_times(rng, n: int, horizon_s: float) -> np.ndarray:
    """Inverse-CDF sampling of rate lambda(t) ~ 1 + 0.5 sin(2 pi t / P - pi/2)."""
    P = horizon_s
    grid = np.linspace(0.0, P, 1 << 20)
    cum = grid - (P / (4.0 * math.pi)) * np.sin(2.0 * math.pi * grid / P)
    cum /= cum[-1]
    u = rng.random(n)
    return np.interp(u, cum, grid)


def generate_replica(wl: Workload, rep: int) -> Trace:
    rng = _rng(wl, rep)
    U, A, N = wl.n_users, wl.n_apps, wl.records_per_replica
    # per-user activity weights
    if wl.user_rates is not None:
        w = np.asarray(wl.user_rates, np.float64)
        rng.permutation(U)  # keep the draw sequence uniform across workloads
        abusive = np.zeros(0, np.int64)
    else:
        rank = rng.permutation(U) + 1
        w = rank.astype(np.float64) ** (-wl.zipf_s)
        abusive = rng.choice(U, size=wl.n_abusive, replace=False) if wl.n_abusive else np.zeros(0, np.int64)
        w[abusive] *= wl.abuse_mult
    w = w / w.sum()
    home = rng.integers(0, A, size=U)
    sweep_w = None
    if wl.coef_grid_per_replica:
        g = np.asarray(SWEEP_GRID_Q16, np.int64)
        sweep_w = g[rng.integers(0, g.shape[0], size=2)].reshape(1, 2)

    # interactions until the record count is reached; the last one is truncated
    users_l, apps_l, m_l = [], [], []
    total = 0
    while total < N:
        chunk = max(64, int(1.25 * (N - total)) + 64)
        us = rng.choice(U, size=chunk, p=w)
        own = rng.random(chunk) < 0.8
        other = rng.integers(0, A, size=chunk)
        ap = np.where(own, home[us], other)
        m = _calls(wl, rng, ap)
        users_l.append(us); apps_l.append(ap); m_l.append(m)
        total += int(m.sum())
    us = np.concatenate(users_l); ap = np.concatenate(apps_l); m = np.concatenate(m_l)
    cm = np.cumsum(m)
    k_last = int(np.searchsorted(cm, N))          # first interaction reaching N
    us, ap, m = us[:k_last + 1], ap[:k_last + 1], m[:k_last + 1].copy()
    m[-1] -= int(cm[k_last] - N)
    n_int = us.shape[0]

    # interaction start times (integer microseconds)
    if wl.diurnal:
        t0 = np.sort(_diurnal_times(rng, n_int, wl.horizon_s))
    else:
        t0 = np.sort(rng.random(n_int) * wl.horizon_s)
    t0 = np.floor(t0 * US_PER_S).astype(np.int64)

    # records in (interaction, stage) order
    inter = np.repeat(np.arange(n_int, dtype=np.int64), m)
    first = np.concatenate([[0], np.cumsum(m)[:-1]])
    stage = np.arange(N, dtype=np.int64) - np.repeat(first, m)
    ts = t0[inter] + stage * US_PER_S
    r_user = us[inter].astype(np.int32)
    r_app = ap[inter].astype(np.int32)

    tin = _lognormal(rng, wl.tok_in, r_app, stage) if wl.tok_in else None
    tsys = _lognormal(rng, wl.tok_sys, r_app, stage) if wl.tok_sys else None
    tout = _lognormal(rng, wl.tok_out, r_app, stage) if wl.tok_out else None

    # stream order: (ts, interaction, stage); records are generated in (interaction, stage) order
    order = np.argsort(ts, kind="stable")
    pos = np.empty(N, np.int64)
    pos[order] = np.arange(N, dtype=np.int64)
    head_gen = first[inter]                                   # generation index of call 0
    prev_gen = np.where(stage > 0, np.arange(N) - 1, -1)
    head = pos[head_gen][order].astype(np.int32)
    prev_o = prev_gen[order]
    prev = np.where(prev_o >= 0, pos[np.maximum(prev_o, 0)], -1).astype(np.int32)
    call = stage[order].astype(np.int32)
    multi = wl.calls_kind != "one"
    take = lambda x: None if x is None else np.ascontiguousarray(x[order])
    return Trace(1, U, A, np.array([0, N], np.int64), ts[order].astype(np.int64),
                 r_user[order], r_app[order],
                 call if multi else None, head if multi else None, prev if multi else None,
                 take(tin), take(tsys), take(tout), sweep_w)


def generate(wl: Workload, replicas: Optional[Sequence[int]] = None) -> Trace:
    """Generate the workload (all replicas, or the listed replica ids)."""
    reps = range(wl.n_replicas) if replicas is None else replicas
    return concat([generate_replica(wl, r) for r in reps])


def coef_direct_table(wl: Workload, trace: Trace) -> Optional[np.ndarray]:
    """Q16 coefficient table [R or 1][A][J][3] for workloads that fix it directly
    (the workload's constants, or the weight pair each replica drew).

    Returns None when the table must be derived from expectations via Eq. 1.
    """
    if wl.coef_direct is not None:
        t = np.asarray(wl.coef_direct, np.int64).reshape(1, wl.n_apps, 1, 3)
        return np.ascontiguousarray(t)
    if wl.coef_grid_per_replica:
        R = trace.n_replicas
        t = np.zeros((R, wl.n_apps, 1, 3), np.int64)
        t[:, :, 0, 0] = trace.sweep_w[:, 0:1]
        t[:, :, 0, 1] = 2 * Q16
        t[:, :, 0, 2] = trace.sweep_w[:, 1:2]
        return t
    return None

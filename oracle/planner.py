"""Plain exhaustive search of the system-planning phase (Section 4.3 "System Planning Phase",
Algorithm 2).  Test infrastructure only (see ``oracle/__init__.py``).

A party's per-iteration computation delay is the sum of power laws in the
batch size B of Eqs. 7-9, each scaled by its worker count w over its cores
C; the exchange adds (E + G) / B_b with E and G the per-row embedding and
gradient sizes times B; B_max comes from the memory model
M(B) = M0 + rho * B**chi per worker (the bound below Eq. 14).  Algorithm 2
evaluates every feasible (w_a, w_p, B) and keeps the minimum of
max(T_A, T_P) + T_comm.  Profiles are dicts with the keys of
``vfl_plan_party`` (``lam`` for lambda); party B's top terms are zero.
"""
from __future__ import annotations

import math


def delay(q: dict, B: float, w: int) -> float:
    """Eqs. 7-9 with equal cores per worker: sum of coef * B**exp, times w / C."""
    t = (q["lam"] * B ** q["gamma"] + q["phi"] * B ** q["beta"]
         + q.get("lam_top", 0.0) * B ** q.get("gamma_top", 0.0)
         + q.get("phi_top", 0.0) * B ** q.get("beta_top", 0.0))
    return t * w / q["cores"]


def batch_cap(q: dict, chi: float) -> float:
    """The memory bound on B: ((M_bar - M0) / rho) ** (1 / chi)."""
    if q.get("mem_coef", 0.0) <= 0.0:
        return math.inf
    room = q["mem_cap"] - q["mem_base"]
    return 0.0 if room <= 0.0 else (room / q["mem_coef"]) ** (1.0 / chi)


def plan(a: dict, p: dict, link: dict, batches):
    """Algorithm 2: the first minimum over batches (in order), w_a, w_p of
    max(T_A, T_P) + (E + G) / B_b; returns ((w_a, w_p, B), cost) or None."""
    bmax = min(batch_cap(a, link["chi"]), batch_cap(p, link["chi"]))
    best, arg = math.inf, None
    for B in batches:
        if B < 1 or B > bmax:
            continue
        comm = B * (link["emb"] + link["grad"]) / link["bandwidth"]
        for wa in range(a["w_min"], a["w_max"] + 1):
            for wp in range(p["w_min"], p["w_max"] + 1):
                o = max(delay(a, B, wa), delay(p, B, wp)) + comm
                if o < best:
                    best, arg = o, (wa, wp, B)
    return None if arg is None else (arg, best)


def fit_power_law(batches, seconds):
    """One delay term of Eqs. 7-9, T = coef * B**exp, fitted to measured
    (B, T) pairs of a batch-size sweep by least squares on log T against
    log B (normal equations of the straight line); returns (coef, exp)."""
    xs = [math.log(b) for b in batches]
    ys = [math.log(t) for t in seconds]
    n = len(xs)
    sx, sy = sum(xs), sum(ys)
    sxx = sum(x * x for x in xs)
    sxy = sum(x * y for x, y in zip(xs, ys))
    expo = (n * sxy - sx * sy) / (n * sxx - sx * sx)
    coef = math.exp((sy - expo * sx) / n)
    return coef, expo

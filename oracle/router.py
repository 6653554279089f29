"""Latency-constrained routing of one layer (oracle; test infrastructure only).

Sec. 3.4: one candidate per unit, minimise the summed risk subject to
t_probe + sum t_ker <= T_layer (Eqs. 6-8), solved greedily from the all-dense choice by
risk-per-microsecond substitutions; then candidates whose lower mass is below tau get
the next larger budget of their family that passes, else the cheapest other sparse
candidate that passes, else dense; finally units are grouped by (pattern, budget).  The greedy, expand/fallback and grouping follow the
inference-procedure table (steps 3-6).

Reading of the greedy (the paper gives one sentence): start with every unit on the
dense candidate.  While the total exceeds the budget, over every (unit, candidate) whose
time is below the unit's current time take the minimum of
rho = (R(c) - R(cur)) / (t(cur) - t(c)), ties to the lowest (unit, candidate) in
row-major order, and switch that unit.  If none remains the route is flagged over
budget.  The tau step runs after the solve, as in the table's order, and may exceed the
budget, which is flagged too.  The total is always recomputed as t_probe plus the unit
times summed in unit order.

All arithmetic is IEEE fp64 in a fixed order, so a second implementation that performs
the same operations agrees bit for bit.
"""
from __future__ import annotations

import numpy as np

from .coverage import disagreement, lower_mass, risk

DENSE, ASHAPE, VSLASH, BSPARSE = 0, 1, 2, 3


def unit_tables(mhat, msub, nsub, e, fam, alpha, beta, delta_q):
    """Risk and lower mass per (unit, candidate) from the probe's coverage arrays."""
    U, C = mhat.shape
    R = np.zeros((U, C))
    ML = np.ones((U, C))
    for u in range(U):
        for c in range(C):
            if fam[c] == DENSE:
                continue
            mh = float(mhat[u, c])
            uu = disagreement([float(x) for x in msub[u, c]], [int(x) for x in nsub[u]])
            R[u, c] = risk(mh, uu, float(e[u, c]), alpha, beta)
            ML[u, c] = lower_mass(mh, delta_q)
    return R, ML


def total_time(t, choice, t_probe):
    tot = float(t_probe)
    for u, c in enumerate(choice):
        tot = tot + float(t[u, c])
    return tot


def greedy(R, t, choice, t_probe, T_layer):
    """Risk-per-microsecond substitutions until the budget holds (Sec. 3.4)."""
    U, C = R.shape
    choice = list(choice)
    over = False
    while total_time(t, choice, t_probe) > T_layer:
        cur = np.array(choice)
        t_cur = t[np.arange(U), cur][:, None]
        r_cur = R[np.arange(U), cur][:, None]
        ok = t < t_cur
        if not ok.any():
            over = True
            break
        with np.errstate(divide="ignore", invalid="ignore"):
            rho = (R - r_cur) / (t_cur - t)
        rho = np.where(ok, rho, np.inf)
        flat = int(np.argmin(rho))           # first minimum in (unit, candidate) order
        u, c = divmod(flat, C)
        if not ok[u, c]:
            over = True
            break
        choice[u] = c
    return choice, over


def expand_or_fallback(choice, fam, brank, ML, tau, dense_c, t):
    """A sparse choice whose lower mass is below tau first expands its budget: the smallest
    larger budget of the same family with m_lower >= tau.  If none passes, dense is taken
    only when no sparse candidate at all reaches tau (Sec. 3.4): first the cheapest sparse
    candidate of any family with m_lower >= tau (lowest time, then lowest candidate index),
    else the dense candidate."""
    out = list(choice)
    C = len(fam)
    nfb = 0
    for u, c in enumerate(choice):
        if fam[c] == DENSE or ML[u, c] >= tau:
            continue
        larger = sorted((brank[c2], c2) for c2 in range(C)
                        if fam[c2] == fam[c] and brank[c2] > brank[c])
        pick = None
        for _, c2 in larger:
            if ML[u, c2] >= tau:
                pick = c2
                break
        if pick is None:
            best_t = None
            for c2 in range(C):
                if fam[c2] == DENSE or not ML[u, c2] >= tau:
                    continue
                if best_t is None or t[u, c2] < best_t:
                    best_t = t[u, c2]
                    pick = c2
        if pick is None:
            pick = dense_c
            nfb += 1
        out[u] = pick
    return out, nfb


def group(choice, C):
    """Units grouped by candidate (one (pattern, budget) per group), grid order."""
    groups = []
    for c in range(C):
        us = [u for u, cc in enumerate(choice) if cc == c]
        if us:
            groups.append((c, us))
    return groups


def route_layer(mhat, msub, nsub, e, t, fam, brank, t_probe, T_layer, tau, alpha, beta,
                delta_q):
    """Full routing of one layer.  Arrays are [units, candidates] (``msub`` has a third
    axis for the R/U/Bd subset means, ``nsub`` is [units, 3]).  Returns a dict with the
    choice per unit, groups, total time, summed risk, fallback count and flags."""
    mhat = np.asarray(mhat, dtype=np.float64)
    U, C = mhat.shape
    fam = [int(f) for f in fam]
    dense = [c for c in range(C) if fam[c] == DENSE]
    if not dense:
        raise ValueError("the candidate grid must contain the dense candidate")
    dense_c = dense[0]
    R, ML = unit_tables(mhat, np.asarray(msub, dtype=np.float64), np.asarray(nsub),
                        np.asarray(e, dtype=np.float64), fam, alpha, beta, delta_q)
    t = np.asarray(t, dtype=np.float64)
    choice, over_solve = greedy(R, t, [dense_c] * U, t_probe, T_layer)
    choice, nfb = expand_or_fallback(choice, fam, list(brank), ML, tau, dense_c, t)
    tot = total_time(t, choice, t_probe)
    rsum = 0.0
    for u, c in enumerate(choice):
        rsum = rsum + float(R[u, c])
    return dict(choice=choice, groups=group(choice, C), total=tot, risk=rsum,
                n_fallback=nfb, over_budget=bool(over_solve or tot > T_layer),
                infeasible=bool(over_solve), R=R, ML=ML)

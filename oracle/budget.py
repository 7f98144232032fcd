"""Response-budget rule (Sec. 3.2 and the Sec. 4.1 protocol).

Test infrastructure only (see oracle/__init__.py).

The budget tau is the smallest table-cost threshold at which the median
calibration schedule reaches ceil(rho_tar (K-1)) reuses.  Reading: the
candidate thresholds are the values min_h J_K(n, h) over all calibration plans
and counts n (B* can only change at those values); the median of an even
number of counts is the mean of the two middle ones; if no candidate reaches
the target, the largest candidate is taken.
"""
from __future__ import annotations

import math

from .dp import forward, min_cost_by_count
from .planner import scene_tables


def target_reuses(rho: float, K: int) -> int:
    return int(math.ceil(rho * (K - 1)))


def bstar_at(m, tau):
    b = 0
    for n, v in enumerate(m):
        if v is not None and v <= tau:
            b = n
    return b


def select_tau(problems, rho: float) -> int:
    """problems: calibration scheduling problems (initial plans, no spent budget)."""
    curves = []
    for p in problems:
        t = scene_tables(p)
        if not t.supported:
            curves.append([0])          # full inference: zero reuses at any budget
            continue
        J = forward(p, t)
        curves.append(min_cost_by_count(J, p.K))
    cands = sorted({v for m in curves for v in m if v is not None})
    target = target_reuses(rho, problems[0].K)
    for tau in cands:
        b = sorted(bstar_at(m, tau) for m in curves)
        n = len(b)
        if n % 2 == 1:
            ok = b[n // 2] >= target
        else:
            ok = b[n // 2 - 1] + b[n // 2] >= 2 * target
        if ok:
            return tau
    return cands[-1]

"""Anchor selection from a calibration set (Sec. 3.1).

Test infrastructure only (see oracle/__init__.py).

The paper standardises the motion statistics L and Theta (Eq. 2) of the
calibration clips with their calibration means and standard deviations.  The
low-motion anchor is the clip whose standardised values have the smallest sum.
The moving-turn anchor is chosen among the clips whose raw Theta is above the
calibration median and whose raw L and Theta are both above the low-motion
anchor's: it is the one whose standardised values have the largest product.
The clip index breaks ties; with no candidate, DriveCache falls back to full
inference.

Readings where the paper is silent:
  * the standard deviation is the population one (divide by n); a zero
    deviation is replaced by eps, as the other denominators of Sec. 3.1 are;
  * the median of an even count is the mean of the two middle values;
  * "the clip index breaks ties" keeps the lowest index;
  * sums run in clip order, one IEEE double operation at a time.
"""
from __future__ import annotations

import math


def standardise(x, eps):
    """z_i = (x_i - mean) / max(std, eps), population mean and standard deviation."""
    n = len(x)
    s = 0.0
    for v in x:
        s = s + float(v)
    mean = s / n
    ss = 0.0
    for v in x:
        dv = float(v) - mean
        ss = ss + dv * dv
    sd = math.sqrt(ss / n)
    den = max(sd, eps)
    return [(float(v) - mean) / den for v in x]


def median(x):
    """Median; for an even count the mean of the two middle values."""
    s = sorted(float(v) for v in x)
    n = len(s)
    if n % 2 == 1:
        return s[n // 2]
    return (s[n // 2 - 1] + s[n // 2]) / 2.0


def select_anchors(L, Th, eps):
    """Calibration clips' (L_i, Theta_i) -> (i0, i1): the low-motion and moving-turn
    anchor indices; i1 is None when no clip qualifies (full-inference fallback)."""
    n = len(L)
    if n < 1 or len(Th) != n:
        raise ValueError("need one (L, Theta) pair per clip")
    zL = standardise(L, eps)
    zT = standardise(Th, eps)
    i0 = 0
    best = zL[0] + zT[0]
    for i in range(1, n):
        v = zL[i] + zT[i]
        if v < best:
            i0, best = i, v
    med = median(Th)
    i1 = None
    best1 = 0.0
    for i in range(n):
        if not (float(Th[i]) > med and float(L[i]) > float(L[i0]) and float(Th[i]) > float(Th[i0])):
            continue
        v = zL[i] * zT[i]
        if i1 is None or v > best1:
            i1, best1 = i, v
    return i0, i1

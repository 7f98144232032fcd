"""Scene-level planner: planned ego motion -> scene run costs and drift thresholds.

Test infrastructure only (see oracle/__init__.py).

Follows Sec. 3.1 of the paper:
  Eq. 2  total translation L and accumulated wrapped rotation Theta,
  Eq. 3  normalisation against the two anchors, with the coordinatewise
         support gate [0,1]^2 (outside it: full inference),
  Eq. 4  motion intensity D,
  Eq. 8  one-sided interpolation of the anchor responses (and, with the same
         rule, of the anchor drift tables, giving the thresholds d-bar),
  Eq. 9  monotone envelope Q and incremental run cost c-hat.

Readings where the paper is silent: costs are carried as exact integers in
units of 2^-40 (Q rounded half-to-even after the scaling, which is exact);
every scalar operation is a single IEEE double operation in the order written.
"""
from __future__ import annotations

import math

COST_SCALE = 2.0 ** 40


def wrap(a: float) -> float:
    """Wrap an angle difference into [-pi, pi)."""
    two_pi = 2.0 * math.pi
    return a - two_pi * math.floor((a + math.pi) / two_pi)


def motion_statistics(xy, yaw):
    """Eq. 2: L = sum_t ||p_t - p_{t-1}||_2, Theta = sum_t |wrap(psi_t - psi_{t-1})|."""
    L = 0.0
    Th = 0.0
    for t in range(1, len(yaw)):
        dx = float(xy[t][0]) - float(xy[t - 1][0])
        dy = float(xy[t][1]) - float(xy[t - 1][1])
        L = L + math.sqrt(dx * dx + dy * dy)
        Th = Th + abs(wrap(float(yaw[t]) - float(yaw[t - 1])))
    return L, Th


def normalise(L, Th, L0, Th0, L1, Th1, eps):
    """Eq. 3: z^L = (L - L0) / max(L1 - L0, eps), and likewise for Theta."""
    zL = (L - L0) / max(L1 - L0, eps)
    zTh = (Th - Th0) / max(Th1 - Th0, eps)
    return zL, zTh


def in_support(zL, zTh) -> bool:
    """The scene is inside the calibration support iff (zL, zTh) lies in [0,1]^2."""
    return 0.0 <= zL <= 1.0 and 0.0 <= zTh <= 1.0


def motion_intensity(zL, zTh):
    """Eq. 4: D = sqrt(zL^2 + zTh^2) / sqrt(2)."""
    return math.sqrt(zL * zL + zTh * zTh) / math.sqrt(2.0)


def interpolate(t0, t1, D):
    """Eq. 8 applied entrywise: t0 + D * max(t1 - t0, 0)."""
    return [[t0[j][h] + D * max(t1[j][h] - t0[j][h], 0.0) for h in range(len(t0[j]))]
            for j in range(len(t0))]


def envelope_costs(qt):
    """Eq. 9: Q_{j,h} = max_{1<=l<=h} q~_{j,l}; c_{j,h} = Q_{j,h} - Q_{j,h-1}, Q_{j,0} = 0.

    Returns (Q_q, c_q): integer tables in units of 2^-40 (Q rounded half-to-even)."""
    Qq, cq = [], []
    for row in qt:
        Qrow = []
        for h in range(len(row)):
            Qrow.append(max(row[: h + 1]))
        Qint = [round(v * COST_SCALE) for v in Qrow]     # Python round(): ties to even
        Qq.append(Qint)
        cq.append([Qint[h] - (Qint[h - 1] if h > 0 else 0) for h in range(len(Qint))])
    return Qq, cq


class SceneTables:
    """Everything the DP and the runtime need for one scene."""

    def __init__(self, L, Th, zL, zTh, supported, D, chat_q, dbar):
        self.L, self.Th, self.zL, self.zTh = L, Th, zL, zTh
        self.supported, self.D = supported, D
        self.chat_q = chat_q      # chat_q[j-1][h-1], integer units of 2^-40
        self.dbar = dbar          # dbar[j-1][h-1], float

    def cost(self, j: int, h: int) -> int:
        """c-hat for refresh step j (1-based) and age h (1-based)."""
        return self.chat_q[j - 1][h - 1]

    def threshold(self, j: int, h: int) -> float:
        return self.dbar[j - 1][h - 1]


def scene_tables(prob) -> SceneTables:
    """Planned poses + anchor tables -> scene costs and thresholds (Eq. 2, 3, 4, 8, 9)."""
    L, Th = motion_statistics(prob.pose_xy, prob.pose_yaw)
    zL, zTh = normalise(L, Th, prob.L0, prob.Th0, prob.L1, prob.Th1, prob.eps)
    sup = in_support(zL, zTh)
    D = motion_intensity(zL, zTh)
    q0 = [[float(v) for v in r] for r in prob.q0]
    q1 = [[float(v) for v in r] for r in prob.q1]
    d0 = [[float(v) for v in r] for r in prob.d0]
    d1 = [[float(v) for v in r] for r in prob.d1]
    qt = interpolate(q0, q1, D)
    _, cq = envelope_costs(qt)
    dbar = interpolate(d0, d1, D)
    return SceneTables(L, Th, zL, zTh, sup, D, cq, dbar)

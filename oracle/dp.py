"""Exact reuse schedule (Sec. 3.2, Eq. 10-11) and a brute-force check of it.

Test infrastructure only (see oracle/__init__.py).

State after step k: (n reuses so far, cache age h).  J_s(0,0) = 0 at the first
decided step s (s = 1 for the initial plan; after a forced refresh at step s,
the replan starts there from age zero).  For the next step k+1:
  full   J_{k+1}(n, 0)     = min_h J_k(n, h)
  reuse  J_{k+1}(n+1, h+1) = J_k(n, h) + c_{k-h, h+1}
         allowed only when h+1 <= H_max, the step is legal, the run does not
         cross a segment boundary, and n+1 stays within the reuse cap.
Eq. 11: B* = max{ n : min_h J_K(n, h) <= tau }.  Backtracking returns the
minimum-cost schedule at B*; ties are broken deterministically by taking the
smallest cache age at every backtracking step, which is the schedule whose
refresh/reuse mask is smallest when read from step K downward with full < reuse.

Readings: legality L(k, h+1) is the legality of reusing at step k+1 (1-based)
with age h+1; a run started by the refresh at step j may only reuse at steps in
j's segment; costs are exact integers (units of 2^-40); on a replan the budget
is tau - spent_q and the cap n_cap - spent_n.
"""
from __future__ import annotations

from .planner import scene_tables

INF = None   # unreachable state


def _better(a, b):
    """a < b where None is +infinity."""
    if a is None:
        return False
    return b is None or a < b


def _allowed(prob, k_next: int, j: int) -> bool:
    """May step k_next (1-based) reuse the cache refreshed at step j?"""
    if not prob.legal[k_next - 1]:
        return False
    if prob.segment is not None and prob.segment[k_next - 1] != prob.segment[j - 1]:
        return False
    return True


def forward(prob, tables):
    """Tables J[k][n][h] for k = s..K (dict keyed by 1-based step)."""
    K, H, s = prob.K, prob.h_max, prob.start_step
    nmax = max(0, prob.n_cap - prob.spent_n)
    J = {s: [[INF] * (H + 1) for _ in range(nmax + 1)]}
    J[s][0][0] = 0
    for k in range(s, K):
        cur = J[k]
        nxt = [[INF] * (H + 1) for _ in range(nmax + 1)]
        for n in range(nmax + 1):
            # full evaluation at k+1: pays nothing and resets the age
            best = INF
            for h in range(H + 1):
                if _better(cur[n][h], best):
                    best = cur[n][h]
            nxt[n][0] = best
        for n in range(nmax):
            for h in range(H):
                if cur[n][h] is None:
                    continue
                j = k - h                       # last full evaluation of this run
                if not _allowed(prob, k + 1, j):
                    continue
                cand = cur[n][h] + tables.cost(j, h + 1)
                if _better(cand, nxt[n + 1][h + 1]):
                    nxt[n + 1][h + 1] = cand
        J[k + 1] = nxt
    return J


def min_cost_by_count(J, K):
    """m(n) = min_h J_K(n, h) (None if unreachable)."""
    out = []
    for row in J[K]:
        best = INF
        for v in row:
            if _better(v, best):
                best = v
        out.append(best)
    return out


class Schedule:
    def __init__(self, reuse, n_reuse, cost_q, tables):
        self.reuse = reuse            # list of 0/1 per step (index k-1); steps <= start_step are 0
        self.n_reuse = n_reuse
        self.cost_q = cost_q
        self.tables = tables

    def __repr__(self):
        return f"Schedule(n={self.n_reuse}, cost={self.cost_q}, mask={''.join(map(str, self.reuse))})"


def schedule(prob, tables=None) -> Schedule:
    """Eq. 10-11 plus backtracking for one scene (initial plan or suffix replan)."""
    if tables is None:
        tables = scene_tables(prob)
    K, s = prob.K, prob.start_step
    reuse = [0] * K
    if not tables.supported:
        return Schedule(reuse, 0, 0, tables)        # outside the support: full inference
    J = forward(prob, tables)
    m = min_cost_by_count(J, K)
    budget = prob.tau_q - prob.spent_q
    bstar = 0
    for n, v in enumerate(m):
        if v is not None and v <= budget:
            bstar = n
    # backtrack: smallest age at the end, smallest predecessor age at each full state
    n = bstar
    h = min(hh for hh in range(prob.h_max + 1) if J[K][n][hh] == m[n])
    cost = m[n]
    for k in range(K, s, -1):
        if h > 0:
            reuse[k - 1] = 1
            n, h = n - 1, h - 1
        else:
            target = J[k][n][0]
            h = min(hh for hh in range(prob.h_max + 1) if J[k - 1][n][hh] == target)
    return Schedule(reuse, bstar, cost, tables)


# ----------------------------------------------------------------------------
# independent check: enumerate every placement of reuses after step s
# ----------------------------------------------------------------------------
def mask_cost(prob, tables, mask):
    """Cost of a full/reuse mask over steps 1..K, or None if illegal.
    Steps <= start_step must be full."""
    K, s = prob.K, prob.start_step
    cost = 0
    n = 0
    j = None
    age = 0
    for k in range(1, K + 1):
        r = mask[k - 1]
        if k <= s:
            if r:
                return None
            j, age = k, 0
            continue
        if not r:
            j, age = k, 0
            continue
        age += 1
        if age > prob.h_max or not _allowed(prob, k, j):
            return None
        cost += tables.cost(j, age)
        n += 1
    if n > prob.n_cap - prob.spent_n:
        return None
    return n, cost


def brute_force(prob, tables=None) -> Schedule:
    """The feasible mask with the most reuses, then least cost, then the
    smallest mask read from step K downward (full < reuse)."""
    if tables is None:
        tables = scene_tables(prob)
    K, s = prob.K, prob.start_step
    if not tables.supported:
        return Schedule([0] * K, 0, 0, tables)
    free = K - s
    budget = prob.tau_q - prob.spent_q
    best = None
    for bits in range(1 << free):
        mask = [0] * s + [(bits >> i) & 1 for i in range(free)]
        r = mask_cost(prob, tables, mask)
        if r is None:
            continue
        n, c = r
        if c > budget:
            continue
        key = (-n, c, tuple(reversed(mask)))
        if best is None or key < best[0]:
            best = (key, mask, n, c)
    _, mask, n, c = best
    return Schedule(mask, n, c, tables)

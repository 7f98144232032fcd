"""Causal cache controller and the cached / uncached samplers (Sec. 3, Eq. 1, Eq. 12).

Test infrastructure only (see oracle/__init__.py).

Per scene and step k (Sec. 3.2):
  * step 1 is always a full evaluation (Eq. 1 discussion);
  * a planned full step evaluates the backbone, refreshes the cache r = h_out - h_in
    and the reference input u_j, and resets the age;
  * before a planned reuse (the h-th of a run started at j) the observed drift
    d_obs = dist(u_{j+h}, u_j) / (norm(u_{j+h}) + eps) is measured before any
    backbone call; reuse is accepted iff d_obs <= dbar_{j,h} + eps and
    C + c_{j,h} <= tau, and then C grows by c_{j,h};
  * otherwise the step evaluates the backbone and refreshes (C unchanged), and
    the unexecuted suffix is replanned from age zero with budget tau - C; the
    executed prefix is never changed.
Reading (Eq. 12 vs the workload's stated metric): the distance is selectable:
"l1" uses sums of absolute values, "l2" the Euclidean norms of Eq. 12; both use
the whole per-scene video-row tensor.

Model-specific legality (Sec. 3.2, last paragraph; Table 4):
  * two experts (a high-noise backbone for steps k < k_switch, a low-noise one from
    k_switch on): each step runs the active expert's whole network (patch embedding,
    conditioning, blocks, head); no cached entry crosses the switch, which the
    scene's segment[] expresses (a segment change at k_switch), so step k_switch
    always evaluates the backbone;
  * guidance branches: a conditional branch (txt) and an unconditional one
    (txt_null) with separate residual caches, combined as
    v = v_u + w (v_c - v_u) before the Euler update.  Both branches share the
    step's decision; u (block 0's modulated input of the video rows) does not
    depend on the text, so the one drift check serves both.
"""
from __future__ import annotations

import math

import numpy as np

from . import dit
from .dp import schedule


class StepRecord:
    __slots__ = ("k", "planned", "realized", "drift", "drift_l2", "threshold", "vetoed", "j", "age")

    def __init__(self, **kw):
        for s in self.__slots__:
            setattr(self, s, kw.get(s))


class SampleResult:
    def __init__(self, x, records, plans, charge, plan):
        self.x = x                  # final latent x_{K+1}
        self.plan = plan            # the plan as it stood at the end (prefix executed, suffixes replanned)
        self.records = records      # StepRecord per step
        self.plans = plans          # every schedule used (initial + replans)
        self.charge = charge        # final accumulated charge C (2^-40 units)

    @property
    def realized(self):
        return [r.realized for r in self.records]

    def margins(self):
        """|d_obs - threshold| at every drift check."""
        return [abs(r.drift - r.threshold) for r in self.records if r.drift is not None]


def drift_sums(u, u_ref):
    """(sum|u-u_ref|, sum|u|, sum (u-u_ref)^2, sum u^2) over the whole tensor."""
    dlt = u - u_ref
    return (float(np.abs(dlt).sum()), float(np.abs(u).sum()),
            float((dlt * dlt).sum()), float((u * u).sum()))


def drift_value(sums, eps, metric="l1"):
    s1, s2, s3, s4 = sums
    if metric == "l1":
        return s1 / (s2 + eps)
    return math.sqrt(s3) / (math.sqrt(s4) + eps)


def sample(W, x1, txt, sigmas, prob, metric="l1", uncached=False, force_veto=(),
           W_low=None, k_switch=None, guidance=None, txt_null=None, steps=None, on_step=None,
           resume=None, block_memo=None):
    """One cached K-step sample of one scene.

    W: `Weights`; x1 [C,T,H,W]; txt [n_txt, d]; sigmas [K+1]; prob: `SchedProblem`.
    uncached=True runs every step in full with no drift checks (the plain sampler).
    force_veto: steps whose planned reuse is rejected regardless of the drift
    (exercises the veto path).
    W_low, k_switch: the low-noise expert and the first step it runs (prob.segment
    must change at k_switch).  guidance, txt_null: the guidance scale w and the
    unconditional text; the branches keep separate caches.
    steps: stop after this many steps (default K); the result then holds x_{steps+1}.
    on_step(k, x, records, plan, state): called after each step with the latent x_{k+1},
    the records so far, the current plan and the whole controller state (a dict), for
    writing intermediate results.
    resume: such a state dict; the sample continues after its step (a long run can be
    stopped and picked up again without recomputing the executed steps).
    block_memo: passed to dit.backbone for the conditional branch (see there)."""
    experts = [dit.Params(W)]
    if W_low is not None:
        if prob.segment is None or prob.segment[k_switch - 1] == prob.segment[k_switch - 2]:
            raise ValueError("a two-expert scene needs a segment change at k_switch")
        experts.append(dit.Params(W_low))
    cfg = guidance is not None
    m = W.m
    K = prob.K
    x = x1.astype(np.float64)
    plan = schedule(prob)
    plans = [plan]
    tables = plan.tables
    mask = list(plan.reuse)
    C = 0
    n_done = 0
    j = 1
    age = 0
    r = None
    r_u = None
    u_ref = None
    records = []
    k0 = 1
    if resume is not None:
        x, mask, C, n_done, j, age = resume["x"], list(resume["mask"]), resume["C"], resume["n_done"], \
            resume["j"], resume["age"]
        r, r_u, u_ref = resume["r"], resume["r_u"], resume["u_ref"]
        records, plans = list(resume["records"]), list(resume["plans"])
        k0 = resume["k"] + 1
    for k in range(k0, (K if steps is None else min(steps, K)) + 1):
        P = experts[1] if (W_low is not None and k >= k_switch) else experts[0]
        mods, head_mod = dit.step_modulation(P, sigmas[k - 1])
        h_in = dit.embed(P, x, txt)
        h_in_u = dit.embed(P, x, txt_null) if cfg else None
        u = dit.backbone_input(P, h_in, mods[0])
        planned = 0 if (uncached or k == 1) else mask[k - 1]
        rec = StepRecord(k=k, planned=planned, drift=None, drift_l2=None, threshold=None,
                         vetoed=False)
        reuse = False
        if planned:
            sums = drift_sums(u, u_ref)
            d_obs = drift_value(sums, prob.eps, metric)
            thr = tables.threshold(j, age + 1)
            c = tables.cost(j, age + 1)
            rec.drift, rec.drift_l2, rec.threshold = d_obs, drift_value(sums, prob.eps, "l2"), thr
            if k not in force_veto and d_obs <= thr + prob.eps and C + c <= prob.tau_q:
                reuse = True
                C += c
                age += 1
                n_done += 1
            else:
                rec.vetoed = True
        if reuse:
            g = h_in[: m.n_v] + r
            g_u = h_in_u[: m.n_v] + r_u if cfg else None
        else:
            h_out = dit.backbone(P, mods, h_in, memo=block_memo)
            r = h_out[: m.n_v] - h_in[: m.n_v]
            g = h_out[: m.n_v]
            if cfg:
                h_out_u = dit.backbone(P, mods, h_in_u)
                r_u = h_out_u[: m.n_v] - h_in_u[: m.n_v]
                g_u = h_out_u[: m.n_v]
            u_ref = u
            j, age = k, 0
            if rec.vetoed:
                newp = schedule(prob.replace(start_step=k, spent_q=C, spent_n=n_done))
                plans.append(newp)
                mask = mask[:k] + list(newp.reuse[k:])
        rec.realized = 1 if reuse else 0
        rec.j, rec.age = j, age
        records.append(rec)
        v = dit.head(P, head_mod, g)
        if cfg:
            v_u = dit.head(P, head_mod, g_u)
            v = v_u + guidance * (v - v_u)
        x = dit.euler(x, v, sigmas[k - 1], sigmas[k])
        if on_step is not None:
            on_step(k, x, records, mask, {"k": k, "x": x, "mask": list(mask), "C": C, "n_done": n_done,
                                          "j": j, "age": age, "r": r, "r_u": r_u, "u_ref": u_ref,
                                          "records": list(records), "plans": list(plans)})
    return SampleResult(x, records, plans, C, mask)

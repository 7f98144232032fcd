"""Seeded synthetic workloads for the cache-aware denoising step.

This module is shared by the HIP path's tests/bench and by the CPU oracle, so it
holds none of the method's arithmetic: only random draws, round-to-nearest-even
conversion to bf16, the closed-form synthetic response tables, and the pose
integration that turns a (speed, yaw-rate) profile into planned ego poses.

Every array is a pure function of its key, so any single tensor (say one
block's weights) can be regenerated without drawing the others, and the result
does not depend on how many threads draw it.
"""
from __future__ import annotations

import hashlib
import json
import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

CHUNK = 1 << 22            # elements per independently seeded chunk
WEIGHT_STD = 0.02          # every generator parameter is N(0, 0.02)
NO_VETO = 1e30             # a drift threshold no observed drift reaches (finite, so the
                           # one-sided interpolation of the threshold tables stays finite)


# ----------------------------------------------------------------------------
# random draws
# ----------------------------------------------------------------------------
def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def normal(shape, std: float, key) -> np.ndarray:
    """float32 N(0, std^2) array; chunk c is drawn from PCG64(SeedSequence(key + [c]))."""
    shape = tuple(int(s) for s in shape)
    n = int(np.prod(shape)) if shape else 1
    out = np.empty(n, np.float32)
    bounds = [(a, min(n, a + CHUNK)) for a in range(0, n, CHUNK)]

    def fill(ci):
        a, b = bounds[ci]
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key) + [ci])))
        g.standard_normal(out=out[a:b], dtype=np.float32)

    if len(bounds) > 1:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, range(len(bounds))))
    elif bounds:
        fill(0)
    if std != 1.0:
        out *= np.float32(std)
    return out.reshape(shape)


def uniform(n: int, lo: float, hi: float, key) -> np.ndarray:
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key))))
    return g.uniform(lo, hi, size=n)


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 value (ties to even); returns float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = a.view(np.uint32).astype(np.uint64)
    bias = np.uint64(0x7FFF) + ((bits >> np.uint64(16)) & np.uint64(1))
    bits = ((bits + bias) & np.uint64(0xFFFF0000)).astype(np.uint32)
    return bits.view(np.float32).reshape(a.shape)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """uint16 bit patterns of float32 values that are already bf16-representable."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    if not np.array_equal(round_bf16(a), a):
        raise ValueError("array is not bf16-representable")
    return (a.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


# ----------------------------------------------------------------------------
# model shape and workloads
# ----------------------------------------------------------------------------
@dataclass(frozen=True)
class ModelShape:
    n_blocks: int
    hidden: int
    heads: int
    head_dim: int
    mlp_hidden: int
    lat_c: int
    lat_t: int
    lat_h: int          # latent height (pixels of the latent grid, before patching)
    lat_w: int
    patch: int
    n_txt: int
    dtype: str          # "f32" or "bf16": GEMM/attention operand and cache dtype
    ln_eps: float = 1e-6
    t_freq: int = 256   # sinusoidal timestep features

    @property
    def hp(self) -> int:
        return self.lat_h // self.patch

    @property
    def wp(self) -> int:
        return self.lat_w // self.patch

    @property
    def n_v(self) -> int:
        return self.lat_t * self.hp * self.wp

    @property
    def n_tok(self) -> int:
        return self.n_v + self.n_txt

    @property
    def patch_dim(self) -> int:
        return self.lat_c * self.patch * self.patch

    @property
    def latent_shape(self):
        return (self.lat_c, self.lat_t, self.lat_h, self.lat_w)


@dataclass(frozen=True)
class Motion:
    """Planned ego motion: constant speed v (m/s); yaw rate omega (rad/s) that
    starts after `straight_s` seconds of straight driving."""
    v: float
    omega: float
    straight_s: float = 0.0


@dataclass(frozen=True)
class Workload:
    cfg_id: int
    name: str
    model: ModelShape
    batch: int
    K: int
    h_max: int
    n_cap: int | None           # None -> K-1
    tau: str                    # "inf" or "rule"
    rho: float                  # target reuse fraction for the budget rule
    thr: float                  # constant drift threshold (d0 = d1 = thr)
    motions: tuple = field(default_factory=tuple)   # one Motion per scene, or () = random
    eps: float = 1e-6
    dt: float = 0.1             # pose sampling period (10 Hz)

    @property
    def n_pose(self) -> int:
        return 4 * (self.model.lat_t - 1) + 1

    @property
    def horizon_s(self) -> float:
        return (self.n_pose - 1) * self.dt

    @property
    def cap(self) -> int:
        return self.K - 1 if self.n_cap is None else self.n_cap


TINY = ModelShape(2, 256, 4, 64, 1024, 16, 4, 16, 16, 2, 16, "f32")
MID = ModelShape(12, 1152, 16, 72, 4608, 16, 8, 32, 56, 2, 120, "bf16")
TARGET = ModelShape(30, 1920, 30, 64, 7680, 16, 13, 60, 90, 2, 226, "bf16")
WIDE = ModelShape(42, 3072, 48, 64, 12288, 16, 13, 60, 90, 2, 226, "bf16")

WORKLOADS = {
    "dit-tiny-f32": Workload(1, "dit-tiny-f32", TINY, 1, 10, 2, 3, "inf", 0.5, NO_VETO,
                             (Motion(8.0, 0.0),)),
    "dit-12x1152-bf16": Workload(2, "dit-12x1152-bf16", MID, 1, 30, 3, None, "rule", 0.5, 0.15,
                                 (Motion(0.0, 0.0),)),
    "dit-30x1920-bf16": Workload(3, "dit-30x1920-bf16", TARGET, 1, 50, 3, None, "rule", 0.5, 0.15,
                                 (Motion(6.0, 0.25),)),
    "dit-42x3072-bf16": Workload(4, "dit-42x3072-bf16", WIDE, 1, 50, 3, None, "rule", 0.5, 0.15,
                                 (Motion(15.0, 0.15, straight_s=2.0),)),
    "dit-30x1920-bf16-b4": Workload(5, "dit-30x1920-bf16-b4", TARGET, 4, 50, 3, None, "rule", 0.5,
                                    0.15, ()),
}


def scene_motions(w: Workload):
    """One Motion per scene; random scenes draw speed U[0,20] and yaw rate U[-0.3,0.3]."""
    if w.motions:
        assert len(w.motions) == w.batch
        return list(w.motions)
    out = []
    for s in range(w.batch):
        v, om = uniform(2, 0.0, 1.0, (4000 + s,))
        out.append(Motion(20.0 * float(v), -0.3 + 0.6 * float(om)))
    return out


def calibration_motions(n: int = 32):
    """The budget rule's calibration plans (speed U[0,20] m/s, yaw rate U[-0.3,0.3])."""
    out = []
    for i in range(n):
        v, om = uniform(2, 0.0, 1.0, (5000 + i,))
        out.append(Motion(20.0 * float(v), -0.3 + 0.6 * float(om)))
    return out


# ----------------------------------------------------------------------------
# planned poses and synthetic response/drift tables
# ----------------------------------------------------------------------------
def poses(m: Motion, n_pose: int, dt: float):
    """Integrate (v, omega) at dt: psi_i = psi_{i-1} + omega_i dt and
    p_i = p_{i-1} + v dt (cos psi_{i-1}, sin psi_{i-1}).  Returns (xy [n,2], yaw [n]) f64."""
    xy = np.zeros((n_pose, 2), np.float64)
    yaw = np.zeros(n_pose, np.float64)
    for i in range(1, n_pose):
        om = m.omega if (i * dt) > m.straight_s + 1e-12 else 0.0
        step = m.v * dt
        xy[i, 0] = xy[i - 1, 0] + step * math.cos(yaw[i - 1])
        xy[i, 1] = xy[i - 1, 1] + step * math.sin(yaw[i - 1])
        yaw[i] = yaw[i - 1] + om * dt
    return xy, yaw


def anchors(w: Workload):
    """Low-motion anchor (0, 0) and moving-turn anchor (20 m/s, 0.3 rad/s) over the horizon."""
    th = w.horizon_s
    return 0.0, 0.0, 20.0 * th, 0.3 * th


def response_tables(K: int, h_max: int):
    """Synthetic anchor response tables q0, q1 [(K-1), h_max] (f64).

    Non-monotone in the age h (so an envelope matters) and q1 < q0 at early
    refresh steps (so the one-sided interpolation matters)."""
    S = []
    acc = 0.0
    for l in range(1, h_max + 1):
        acc += (1.0 + l / 2.0) * (1.0 if l % 2 == 1 else -0.5)
        S.append(acc)
    q0 = np.zeros((K - 1, h_max))
    q1 = np.zeros((K - 1, h_max))
    for j in range(1, K):
        x = (j - 1) / (K - 1) if K > 1 else 0.0
        for h in range(1, h_max + 1):
            q0[j - 1, h - 1] = 1e-3 * (1.0 + 3.0 * (1.0 - x) ** 2) * S[h - 1]
            q1[j - 1, h - 1] = 2e-3 * (1.0 + 3.0 * x * x) * S[h - 1]
    return q0, q1


def drift_tables(K: int, h_max: int, thr: float):
    d = np.full((K - 1, h_max), thr, np.float64)
    return d.copy(), d.copy()


# ----------------------------------------------------------------------------
# model weights, latents, text
# ----------------------------------------------------------------------------
GLOBAL_TENSORS = ("w_pe", "b_pe", "pos", "w_t1", "b_t1", "w_t2", "b_t2", "w_m", "b_m",
                  "head_mod", "w_head", "b_head")
BLOCK_TENSORS = ("w_qkv", "b_qkv", "w_o", "b_o", "w_1", "b_1", "w_2", "b_2", "mod_offset")


def tensor_shapes(m: ModelShape):
    d, F, P = m.hidden, m.mlp_hidden, m.patch_dim
    g = {"w_pe": (d, P), "b_pe": (d,), "pos": (m.n_v, d),
         "w_t1": (d, m.t_freq), "b_t1": (d,), "w_t2": (d, d), "b_t2": (d,),
         "w_m": (6 * d, d), "b_m": (6 * d,), "head_mod": (2, d),
         "w_head": (P, d), "b_head": (P,)}
    b = {"w_qkv": (3 * d, d), "b_qkv": (3 * d,), "w_o": (d, d), "b_o": (d,),
         "w_1": (F, d), "b_1": (F,), "w_2": (d, F), "b_2": (d,), "mod_offset": (6, d)}
    return g, b


class Weights:
    """Lazily drawn generator weights (row-major [out, in] matrices, "y = x W^T + b").

    Parameter seed is 1000 + cfg_id; tensor t of block l is keyed (seed, 100 + 16 l + t).
    bf16 models round every parameter to bf16 (RNE); values are float32 arrays.
    `zero_out` zeroes the listed block tensors (used for invariance tests)."""

    def __init__(self, m: ModelShape, cfg_id: int, zero_out=()):
        self.m = m
        self.seed = 1000 + cfg_id
        self.zero_out = frozenset(zero_out)
        self._g, self._b = tensor_shapes(m)
        self._cache = {}

    def _draw(self, shape, key):
        a = normal(shape, WEIGHT_STD, key)
        return round_bf16(a) if self.m.dtype == "bf16" else a

    def get(self, name: str) -> np.ndarray:
        if name not in self._cache:
            i = GLOBAL_TENSORS.index(name)
            self._cache[name] = self._draw(self._g[name], (self.seed, i))
        return self._cache[name]

    def block(self, l: int, name: str) -> np.ndarray:
        if name in self.zero_out:
            return np.zeros(self._b[name], np.float32)
        key = (l, name)
        if key not in self._cache:
            t = BLOCK_TENSORS.index(name)
            self._cache[key] = self._draw(self._b[name], (self.seed, 100 + 16 * l + t))
        return self._cache[key]

    def drop(self):
        self._cache.clear()


def latent(m: ModelShape, cfg_id: int, scene: int = 0) -> np.ndarray:
    """Initial noise x_1 ~ N(0,1), [C, T, H, W] float32."""
    return normal(m.latent_shape, 1.0, (2000 + cfg_id, scene))


def text(m: ModelShape, cfg_id: int, scene: int = 0) -> np.ndarray:
    """Text-token embeddings ~ N(0,1), [n_txt, d] float32 (bf16-rounded for bf16 models)."""
    a = normal((m.n_txt, m.hidden), 1.0, (3000 + cfg_id, scene))
    return round_bf16(a) if m.dtype == "bf16" else a


def hidden_state(m: ModelShape, key, scale_video: float = 0.16) -> np.ndarray:
    """A residual-stream-like [n_tok, d] float32 input for single-block tests:
    video rows ~ N(0, 0.16^2) (the scale of a patch-embedded latent), text rows ~ N(0,1)."""
    h = normal((m.n_tok, m.hidden), 1.0, (6000,) + tuple(key))
    h[: m.n_v] *= np.float32(scale_video)
    return h


def sigmas(K: int) -> np.ndarray:
    """Flow-matching noise levels sigma_k = 1 - (k-1)/K, k = 1..K+1 (shift 1), f64."""
    return np.array([1.0 - (k - 1) / K for k in range(1, K + 2)], np.float64)


# ----------------------------------------------------------------------------
# one scene's scheduling problem (plain data, mirrors the C struct)
# ----------------------------------------------------------------------------
TAU_INF = (1 << 63) - 1     # "no budget": the largest int64


@dataclass
class SchedProblem:
    K: int
    h_max: int
    n_cap: int
    legal: np.ndarray            # uint8 [K]; entry 0 (step 1) is ignored
    segment: np.ndarray | None   # int32 [K] or None
    pose_xy: np.ndarray          # f64 [n_pose, 2]
    pose_yaw: np.ndarray         # f64 [n_pose]
    L0: float
    Th0: float
    L1: float
    Th1: float
    eps: float
    q0: np.ndarray               # f64 [(K-1), h_max]; row j-1 = refresh step j, column h-1 = age h
    q1: np.ndarray
    d0: np.ndarray
    d1: np.ndarray
    tau_q: int = TAU_INF         # budget in units of 2^-40
    start_step: int = 1          # 1 = initial plan; k = replan after a forced refresh at step k
    spent_q: int = 0
    spent_n: int = 0

    def replace(self, **kw) -> "SchedProblem":
        d = dict(self.__dict__)
        d.update(kw)
        return SchedProblem(**d)


def scene_problem(w: Workload, m: Motion, tau_q: int = TAU_INF, thr: float | None = None) -> SchedProblem:
    xy, yaw = poses(m, w.n_pose, w.dt)
    L0, Th0, L1, Th1 = anchors(w)
    q0, q1 = response_tables(w.K, w.h_max)
    d0, d1 = drift_tables(w.K, w.h_max, w.thr if thr is None else thr)
    legal = np.ones(w.K, np.uint8)
    return SchedProblem(w.K, w.h_max, w.cap, legal, None, xy, yaw, L0, Th0, L1, Th1, w.eps,
                        q0, q1, d0, d1, tau_q)


# ----------------------------------------------------------------------------
# fingerprints (run records and stored oracle samples)
# ----------------------------------------------------------------------------
def input_fingerprint(w: Workload) -> str:
    """sha256 over a few generated tensors (scene 0's latent and text, the patch
    embedding, the head, slices of the first and last block): a changed generator
    changes it."""
    W = Weights(w.model, w.cfg_id)
    h = hashlib.sha256()
    for a in (latent(w.model, w.cfg_id, 0), text(w.model, w.cfg_id, 0), W.get("w_pe"),
              W.get("w_head"), W.block(0, "w_qkv")[:64], W.block(w.model.n_blocks - 1, "w_2")[:64]):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def config_hash(w: Workload, tau_q: int, input_fp: str) -> str:
    """sha256 of the workload definition (shape, schedule parameters, scene motions),
    the budget and the input fingerprint: one value per run configuration."""
    rec = {"workload": repr(w), "motions": [repr(m) for m in scene_motions(w)],
           "tau_q": int(tau_q), "inputs": input_fp}
    return hashlib.sha256(json.dumps(rec, sort_keys=True).encode()).hexdigest()

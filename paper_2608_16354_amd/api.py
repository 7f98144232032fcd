"""Python binding of the DriveCache C ABI (include/dc.h).

Functions keep the C names; they marshal torch tensors (device memory, owned by
the caller) and numpy arrays (host) into the C calls.  Every computation runs in
libdrivecache.so; nothing here computes.
"""
from __future__ import annotations

import ctypes as C

import numpy as np

from . import _lib as L
from .inputs import ModelShape, SchedProblem as PySchedProblem

__all__ = ["model_cfg", "DeviceModel", "Workspace", "SamplerBuffers", "profile", "dc_workspace_bytes", "dc_time_modulation",
           "dc_patch_embed", "dc_block_forward", "dc_cache_store", "dc_cache_apply",
           "dc_drift_l1", "dc_head_euler", "dc_schedule_dp", "dc_select_tau", "dc_motion_statistics",
           "dc_select_anchors", "Sampler"]


def _torch():
    import torch
    return torch


def _ptr(t):
    return C.c_void_p(0 if t is None else int(t.data_ptr()))


def _stream(stream=None):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return C.c_void_p(int(s.cuda_stream))


def _idx(idx):
    arr = np.ascontiguousarray(np.asarray(idx, dtype=np.int32))
    return arr, arr.ctypes.data_as(L.i32p), int(arr.size)


def model_cfg(m: ModelShape) -> L.ModelCfg:
    return L.ModelCfg(m.n_blocks, m.hidden, m.heads, m.head_dim, m.mlp_hidden, m.lat_c, m.lat_t,
                      m.lat_h, m.lat_w, m.patch, m.n_txt, L.DC_BF16 if m.dtype == "bf16" else L.DC_F32,
                      m.ln_eps)


class DeviceModel:
    """Generator weights uploaded to the GPU in the library's layout."""

    MATRICES = ("w_qkv", "w_o", "w_1", "w_2")

    def __init__(self, W, device="cuda:0"):
        torch = _torch()
        self.m = W.m
        self.cfg = model_cfg(W.m)
        self.device = device
        mdt = torch.bfloat16 if W.m.dtype == "bf16" else torch.float32

        def up(a, dt=torch.float32):
            return torch.from_numpy(np.ascontiguousarray(a)).to(device=device, dtype=dt)

        self.g = {}
        for name in ("w_pe", "b_pe", "w_t1", "b_t1", "w_t2", "b_t2", "w_m", "b_m", "head_mod", "b_head"):
            self.g[name] = up(W.get(name))
        self.g["pos"] = up(W.get("pos"), mdt)
        self.g["w_head"] = up(W.get("w_head"), mdt)
        self.blocks = []
        for l in range(W.m.n_blocks):
            b = {}
            for name in ("w_qkv", "b_qkv", "w_o", "b_o", "w_1", "b_1", "w_2", "b_2", "mod_offset"):
                b[name] = up(W.block(l, name), mdt if name in self.MATRICES else torch.float32)
            self.blocks.append(b)
        self._cblocks = (L.BlockWeights * W.m.n_blocks)()
        for l, b in enumerate(self.blocks):
            self._cblocks[l] = L.BlockWeights(*[_ptr(b[n]) for n in (
                "w_qkv", "b_qkv", "w_o", "b_o", "w_1", "b_1", "w_2", "b_2", "mod_offset")])
        gw = self.g
        self.cweights = L.ModelWeights(
            _ptr(gw["w_pe"]), _ptr(gw["b_pe"]), _ptr(gw["pos"]), _ptr(gw["w_t1"]), _ptr(gw["b_t1"]),
            _ptr(gw["w_t2"]), _ptr(gw["b_t2"]), _ptr(gw["w_m"]), _ptr(gw["b_m"]), _ptr(gw["head_mod"]),
            _ptr(gw["w_head"]), _ptr(gw["b_head"]), self._cblocks)

    def block(self, l):
        return C.pointer(self._cblocks[l])


def dc_workspace_bytes(m: ModelShape, batch: int = 1) -> int:
    cfg = model_cfg(m)
    n = L.load().dc_workspace_bytes(C.byref(cfg), batch)
    if n == 0:
        raise L.DriveCacheError("dc_workspace_bytes", L.DC_ERR_SHAPE, "unsupported shape")
    return int(n)


class Workspace:
    """Device scratch of dc_workspace_bytes() bytes (256-byte aligned)."""

    def __init__(self, m: ModelShape, batch=1, device="cuda:0"):
        torch = _torch()
        self.nbytes = dc_workspace_bytes(m, batch)
        self.buf = torch.empty(self.nbytes + 256, dtype=torch.uint8, device=device)
        off = (-int(self.buf.data_ptr())) % 256
        self.ptr = C.c_void_p(int(self.buf.data_ptr()) + off)


def dc_time_modulation(dm: DeviceModel, sigmas, mod, ws: Workspace, stream=None):
    sig = np.ascontiguousarray(np.asarray(sigmas, np.float64))
    L.check("dc_time_modulation", L.load().dc_time_modulation(
        C.byref(dm.cfg), C.byref(dm.cweights), sig.ctypes.data_as(C.POINTER(C.c_double)), int(sig.size),
        _ptr(mod), ws.ptr, ws.nbytes, _stream(stream)))


def dc_patch_embed(dm: DeviceModel, x, txt, h_in, idx, ws: Workspace, stream=None):
    arr, p, n = _idx(idx)
    L.check("dc_patch_embed", L.load().dc_patch_embed(
        C.byref(dm.cfg), C.byref(dm.cweights), _ptr(x), _ptr(txt), _ptr(h_in), p, n, ws.ptr, ws.nbytes,
        _stream(stream)))


def dc_block_forward(dm: DeviceModel, l: int, mod, h, idx, ws: Workspace, stream=None):
    arr, p, n = _idx(idx)
    L.check("dc_block_forward", L.load().dc_block_forward(
        C.byref(dm.cfg), dm.block(l), _ptr(mod), _ptr(h), p, n, ws.ptr, ws.nbytes, _stream(stream)))


def dc_cache_store(cfg, h_out, h_in, resid, idx, stream=None):
    arr, p, n = _idx(idx)
    L.check("dc_cache_store", L.load().dc_cache_store(
        C.byref(cfg), _ptr(h_out), _ptr(h_in), _ptr(resid), p, n, _stream(stream)))


def dc_cache_apply(cfg, h_in, resid, g, idx, stream=None):
    arr, p, n = _idx(idx)
    L.check("dc_cache_apply", L.load().dc_cache_apply(
        C.byref(cfg), _ptr(h_in), _ptr(resid), _ptr(g), p, n, _stream(stream)))


def dc_drift_l1(cfg, h_in, mod0, u_ref, snapshot, sums, idx, ws: Workspace, stream=None):
    arr, p, n = _idx(idx)
    L.check("dc_drift_l1", L.load().dc_drift_l1(
        C.byref(cfg), _ptr(h_in), _ptr(mod0), _ptr(u_ref), int(bool(snapshot)), _ptr(sums), p, n,
        ws.ptr, ws.nbytes, _stream(stream)))


def dc_drift_l1_noalloc(cfg, h_in, mod0, u_ref, snapshot, sums, idx, stream=None):
    """dc_drift_l1 without a workspace (the library's fixed per-GPU scratch)."""
    arr, p, n = _idx(idx)
    L.check("dc_drift_l1_noalloc", L.load().dc_drift_l1_noalloc(
        C.byref(cfg), _ptr(h_in), _ptr(mod0), _ptr(u_ref), int(bool(snapshot)), _ptr(sums), p, n,
        _stream(stream)))


def dc_head_euler(dm: DeviceModel, head_mod, g, x, dsigma, idx, ws: Workspace, stream=None):
    arr, p, n = _idx(idx)
    L.check("dc_head_euler", L.load().dc_head_euler(
        C.byref(dm.cfg), C.byref(dm.cweights), _ptr(head_mod), _ptr(g), _ptr(x), float(dsigma), p, n,
        ws.ptr, ws.nbytes, _stream(stream)))


def dc_calibrate_tables(dm: DeviceModel, x1, txt, sigmas, h_max: int, eps: float, stream=None):
    """Anchor calibration of one clip (Eq. 5-7) on the GPU: returns (q, d), f64
    [(K-1), h_max] each.  x1 [C, T, H, W], txt [N_t, d]: the clip's inputs (torch
    tensors on the device); sigmas: the K+1 noise levels."""
    torch = _torch()
    sig = np.ascontiguousarray(np.asarray(sigmas, np.float64))
    K = sig.size - 1
    nbytes = L.load().dc_calibrate_workspace_bytes(C.byref(dm.cfg), K)
    if nbytes == 0:
        raise L.DriveCacheError("dc_calibrate_workspace_bytes", L.DC_ERR_ARG, "bad model or K")
    ws = torch.empty(nbytes, dtype=torch.uint8, device=dm.device)
    q = np.zeros((K - 1, h_max), np.float64)
    d = np.zeros((K - 1, h_max), np.float64)
    x1 = x1.to(device=dm.device, dtype=torch.float32).contiguous()
    txt = txt.to(device=dm.device, dtype=torch.float32).contiguous()
    L.check("dc_calibrate_tables", L.load().dc_calibrate_tables(
        C.byref(dm.cfg), C.byref(dm.cweights), _ptr(x1), _ptr(txt),
        sig.ctypes.data_as(C.POINTER(C.c_double)), K, int(h_max), float(eps),
        q.ctypes.data_as(C.POINTER(C.c_double)), d.ctypes.data_as(C.POINTER(C.c_double)),
        int(ws.data_ptr()), nbytes, _stream(stream)))
    return q, d


class _CProblem:
    """A dc_sched_problem whose arrays stay alive with it."""

    def __init__(self, p: PySchedProblem):
        f64 = lambda a: np.ascontiguousarray(np.asarray(a, np.float64))
        self.keep = dict(legal=np.ascontiguousarray(np.asarray(p.legal, np.uint8)),
                         xy=f64(p.pose_xy).reshape(-1), yaw=f64(p.pose_yaw),
                         q0=f64(p.q0).reshape(-1), q1=f64(p.q1).reshape(-1),
                         d0=f64(p.d0).reshape(-1), d1=f64(p.d1).reshape(-1))
        seg = None
        if p.segment is not None:
            self.keep["seg"] = np.ascontiguousarray(np.asarray(p.segment, np.int32))
            seg = self.keep["seg"].ctypes.data_as(C.POINTER(C.c_int32))
        dp = lambda a: a.ctypes.data_as(C.POINTER(C.c_double))
        k = self.keep
        self.c = L.SchedProblem(
            p.K, p.h_max, p.n_cap, k["legal"].ctypes.data_as(C.POINTER(C.c_uint8)), seg,
            len(k["yaw"]), dp(k["xy"]), dp(k["yaw"]), p.L0, p.Th0, p.L1, p.Th1, p.eps,
            dp(k["q0"]), dp(k["q1"]), dp(k["d0"]), dp(k["d1"]), int(p.tau_q), p.start_step,
            int(p.spent_q), p.spent_n)


class ScheduleResult:
    def __init__(self, reuse, chat_q, dbar, s: L.Schedule):
        self.reuse = [int(v) for v in reuse]
        self.chat_q = chat_q
        self.dbar = dbar
        self.n_reuse = int(s.n_reuse)
        self.cost_q = int(s.cost_q)
        self.L, self.Theta, self.zL, self.zTh, self.D = s.L, s.Theta, s.zL, s.zTh, s.D
        self.in_support = bool(s.in_support)


def dc_schedule_dp(p: PySchedProblem) -> ScheduleResult:
    cp = _CProblem(p)
    reuse = np.zeros(p.K, np.uint8)
    nt = max(p.K - 1, 0) * p.h_max
    chat = np.zeros(max(nt, 1), np.int64)
    dbar = np.zeros(max(nt, 1), np.float64)
    out = L.Schedule(reuse.ctypes.data_as(C.POINTER(C.c_uint8)), chat.ctypes.data_as(C.POINTER(C.c_int64)),
                     dbar.ctypes.data_as(C.POINTER(C.c_double)), 0, 0, 0, 0, 0, 0, 0, 0)
    L.check("dc_schedule_dp", L.load().dc_schedule_dp(C.byref(cp.c), C.byref(out)))
    return ScheduleResult(reuse, chat[:nt].reshape(max(p.K - 1, 0), p.h_max),
                          dbar[:nt].reshape(max(p.K - 1, 0), p.h_max), out)


def dc_select_tau(problems, rho: float) -> int:
    cps = [_CProblem(p) for p in problems]
    arr = (L.SchedProblem * len(cps))(*[c.c for c in cps])
    tau = C.c_int64(0)
    L.check("dc_select_tau", L.load().dc_select_tau(arr, len(cps), float(rho), C.byref(tau)))
    return int(tau.value)


def dc_motion_statistics(xy, yaw):
    """Eq. 2 for one pose sequence: (L, Theta)."""
    xy = np.ascontiguousarray(xy, np.float64).reshape(-1, 2)
    yaw = np.ascontiguousarray(yaw, np.float64)
    n = len(yaw)
    Lv, Tv = C.c_double(0.0), C.c_double(0.0)
    dp = C.POINTER(C.c_double)
    L.check("dc_motion_statistics", L.load().dc_motion_statistics(
        xy.ctypes.data_as(dp), yaw.ctypes.data_as(dp), n, C.byref(Lv), C.byref(Tv)))
    return float(Lv.value), float(Tv.value)


def dc_select_anchors(Ls, Ths, eps: float):
    """Sec. 3.1 anchors from calibration clips: ((L0, Th0, L1, Th1), (i0, i1)); i1 = None
    when no clip qualifies (full-inference fallback)."""
    Ls = np.ascontiguousarray(Ls, np.float64)
    Ths = np.ascontiguousarray(Ths, np.float64)
    out = (C.c_double * 4)()
    idx = (C.c_int32 * 2)()
    dp = C.POINTER(C.c_double)
    L.check("dc_select_anchors", L.load().dc_select_anchors(
        Ls.ctypes.data_as(dp), Ths.ctypes.data_as(dp), len(Ls), float(eps), out, idx))
    return tuple(float(v) for v in out), (int(idx[0]), None if idx[1] < 0 else int(idx[1]))


class SamplerBuffers:
    """Caller-owned device buffers for a batch of B scenes (allocated once, reusable).
    branches = 2 (guidance): h_in, h and resid hold 2B entries and the workspace 2B;
    experts = 2: a second modulation table for the low-noise expert."""

    def __init__(self, m: ModelShape, B: int, K: int, device="cuda:0", branches=1, experts=1):
        torch = _torch()
        mdt = torch.bfloat16 if m.dtype == "bf16" else torch.float32
        self.m, self.B, self.K = m, B, K
        E = branches * B
        self.x = torch.empty((B,) + tuple(m.latent_shape), device=device, dtype=torch.float32)
        self.txt = torch.zeros((B, m.n_txt, m.hidden), device=device, dtype=torch.float32)
        self.txt_null = torch.zeros_like(self.txt) if branches == 2 else None
        self.h_in = torch.empty((E, m.n_tok, m.hidden), device=device, dtype=torch.float32)
        self.h = torch.empty_like(self.h_in)
        self.resid = torch.empty((E, m.n_v, m.hidden), device=device, dtype=mdt)
        self.u_ref = torch.empty((B, m.n_v, m.hidden), device=device, dtype=mdt)
        self.mod = torch.empty((K, m.n_blocks + 1, 6, m.hidden), device=device, dtype=torch.float32)
        self.mod_low = torch.empty_like(self.mod) if experts == 2 else None
        self.sums = torch.zeros((B, 4), device=device, dtype=torch.float64)
        self.ws = Workspace(m, E, device)
        self.c = L.Buffers(_ptr(self.x), _ptr(self.txt), _ptr(self.h_in), _ptr(self.h), _ptr(self.resid),
                           _ptr(self.u_ref), _ptr(self.mod), _ptr(self.sums), self.ws.ptr, self.ws.nbytes)


class Sampler:
    """dc_sampler: the causal controller over caller-owned device buffers.

    x1, txt: initial latents [B, C, T, H, W] and text [B, N_t, d] (torch tensors,
    host or device); they are copied into `bufs` (allocated here if not given)."""

    def __init__(self, dm: DeviceModel, problems, sigmas, x1, txt, drift_metric=0, stream=None,
                 bufs: SamplerBuffers = None, low_expert=None, guidance=None):
        """low_expert: (DeviceModel, k_switch), the low-noise expert from step k_switch on
        (every problem's segment must change there); guidance: (w, txt_null [B, N_t, d]),
        guidance branches with separate caches."""
        B = len(problems)
        self.dm, self.B, self.K = dm, B, problems[0].K
        if bufs is None:
            bufs = SamplerBuffers(dm.m, B, self.K, dm.device, branches=2 if guidance else 1,
                                  experts=2 if low_expert else 1)
        self.bufs = bufs
        assert self.bufs.B == B and self.bufs.K == self.K
        self.bufs.x.copy_(x1, non_blocking=True)
        if dm.m.n_txt:
            self.bufs.txt.copy_(txt, non_blocking=True)
        self.x = self.bufs.x
        self._cps = [_CProblem(p) for p in problems]
        arr = (L.SchedProblem * B)(*[c.c for c in self._cps])
        sig = np.ascontiguousarray(np.asarray(sigmas, np.float64))
        self._h = C.c_void_p()
        opts = L.SamplerOpts()
        opts.drift_metric = int(drift_metric)
        self._low = None
        if low_expert is not None:
            self._low, k_switch = low_expert
            assert self.bufs.mod_low is not None
            opts.w_low = C.pointer(self._low.cweights)
            opts.k_switch = int(k_switch)
            opts.mod_low = int(self.bufs.mod_low.data_ptr())
        if guidance is not None:
            w, txt_null = guidance
            assert self.bufs.txt_null is not None
            if dm.m.n_txt:
                self.bufs.txt_null.copy_(txt_null, non_blocking=True)
            opts.cfg = 1
            opts.guidance = float(w)
            opts.txt_null = int(self.bufs.txt_null.data_ptr())
        L.check("dc_sampler_create_ex", L.load().dc_sampler_create_ex(
            C.byref(dm.cfg), C.byref(dm.cweights), B, arr, sig.ctypes.data_as(C.POINTER(C.c_double)),
            C.byref(self.bufs.c), C.byref(opts), _stream(stream), C.byref(self._h)))
        self.k = 0

    def step(self, stream=None):
        """Run the next denoising step; returns (realized [B] uint8, drift [B] f64)."""
        self.k += 1
        realized = np.zeros(self.B, np.uint8)
        drift = np.zeros(self.B, np.float64)
        L.check("dc_denoise_step", L.load().dc_denoise_step(
            self._h, self.k, _stream(stream), realized.ctypes.data_as(C.POINTER(C.c_uint8)),
            drift.ctypes.data_as(C.POINTER(C.c_double))))
        return realized, drift

    def run(self, stream=None):
        """All K steps; returns (realized [K, B], drift [K, B])."""
        rs, ds = [], []
        for _ in range(self.K):
            r, d = self.step(stream)
            rs.append(r)
            ds.append(d)
        return np.stack(rs), np.stack(ds)

    def plan(self, b=0):
        reuse = np.zeros(self.K, np.uint8)
        nv = C.c_int32(0)
        cq = C.c_int64(0)
        L.check("dc_sampler_plan", L.load().dc_sampler_plan(
            self._h, b, reuse.ctypes.data_as(C.POINTER(C.c_uint8)), C.byref(nv), C.byref(cq)))
        return reuse, int(nv.value), int(cq.value)

    def close(self):
        if self._h:
            L.load().dc_sampler_destroy(self._h)
            self._h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class profile:
    """Context manager timing kernel classes with hipEvents (dc_profile_*).

    with api.profile(["attention"]) as p: ...;  p.read() -> {name: (launches, total_ms)}"""

    def __init__(self, classes):
        self.ids = [L.KERNEL_CLASSES.index(c) for c in classes]

    def __enter__(self):
        lib = L.load()
        L.check("dc_profile_reset", lib.dc_profile_reset())
        mask = 0
        for i in self.ids:
            mask |= 1 << i
        L.check("dc_profile_enable", lib.dc_profile_enable(mask))
        return self

    def __exit__(self, *exc):
        L.load().dc_profile_enable(0)
        return False

    def read(self):
        out = {}
        for i in self.ids:
            n = C.c_int64(0)
            ms = C.c_double(0.0)
            L.check("dc_profile_read", L.load().dc_profile_read(i, C.byref(n), C.byref(ms)))
            out[L.KERNEL_CLASSES[i]] = (int(n.value), float(ms.value))
        return out

"""Benchmark: cached K-step sampling of the 30-block video DiT on one MI355X.

One benchmark step = one whole cached sample of the workload: the host schedule
(dc_sampler_create: modulation table + exact DP), then K calls of
dc_denoise_step (patch embedding, drift checks with their readbacks, refresh
blocks or cache reuse, head + Euler).  Inputs (weights, initial latent, text)
are resident in HBM before the timed region.

Prints one JSON line: latent tokens x steps / s = B * N_v * K / (seconds per
sample), the roofline of the dominant kernel (attention, timed live with
hipEvents over the timed region), the combined GEMM + attention MFMA fraction of
the refresh steps, the HBM rate of every reuse-path kernel, a run record (config
hash, realized masks, vetoes, every drift with its margin to the threshold) and
the CPU oracle's rate on a bounded sample.
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MI355X_BF16_DENSE_TFLOPS = 2500.0     # published dense bf16 MFMA peak
MI355X_HBM_GBPS = 8000.0
COPY_BYTES = 1 << 30                  # plain device copy used to scale the HBM byte counters


def traffic_from_profile(kernel_file):
    """HBM bytes per launch of the dominant kernel from the committed counter summary
    (FETCH_SIZE and WRITE_SIZE per dispatch, scaled by a plain copy of known size),
    or None when the kernel source changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "attention_dit-30x1920-bf16_traffic.txt")
    src = os.path.join(ROOT, "paper_2608_16354_amd", "csrc", kernel_file)
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if "=" in line and not line.startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
    if kv.get("source_sha256") != sha:
        return None
    return float(kv["hbm_bytes_per_launch"])


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def gemm_flops(m):
    """Algorithmic FLOPs of one block's four GEMMs (QKV, out-projection, MLP up and down)."""
    N, d, F = m.n_tok, m.hidden, m.mlp_hidden
    return 2.0 * N * d * (3 * d + d + 2 * F)


def hbm_bytes(m):
    """Algorithmic HBM bytes per launch (one scene) of the HBM-bound kernels: every
    operand read once and every result written once."""
    Nv, N, d = m.n_v, m.n_tok, m.hidden
    e = 2 if m.dtype == "bf16" else 4
    lat = 4 * m.lat_c * m.lat_t * m.lat_h * m.lat_w
    return {
        "patch_embed": Nv * d * 4 + Nv * d * e + lat,          # write h_in rows, read pos and x
        "drift": Nv * d * (4 + e),                             # read h_in and u_ref / write u_ref
        "cache_store": Nv * d * (4 + 4 + e),                   # read h_out, h_in; write r
        "cache_apply": Nv * d * (4 + e + 4),                   # read h_in, r; write g
        "head": Nv * d * 4 + 2 * lat,                          # read g; read and write x
        "head_reuse": Nv * d * (4 + e) + 2 * lat,              # read h_in and r; read and write x
        "ln_modulate": N * d * (4 + e),                        # read h; write a
    }


def attention_flops(m):
    """Algorithmic FLOPs of one attention launch (one scene, all heads): QK^T and PV."""
    return 4.0 * m.n_tok * m.n_tok * m.hidden


def refresh_flops(m):
    """Algorithmic FLOPs of one refresh step of one scene (blocks + patch embed + head)."""
    N, d, F = m.n_tok, m.hidden, m.mlp_hidden
    per_block = 2.0 * N * d * (3 * d + d + 2 * F) + attention_flops(m)
    return m.n_blocks * per_block + 2.0 * 2 * m.n_v * 64 * d


def host_info():
    """CPU model name and NumPy's BLAS (the oracle's matrix products)."""
    import numpy as np
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        b = np.show_config(mode="dicts")["Build Dependencies"]["blas"]
        blas = f"{b.get('name')} {b.get('version')}"
    except Exception:
        blas = "unknown"
    return model, blas


def cpu_baseline(w, W, schedule, budget_s=10.0):
    """The fp64 oracle on a bounded sample of the same workload, extrapolated to one
    cached sample: whole blocks at full length (all rows; blocks 0, 1, 2 until budget_s
    of block time is spent) and one full reuse step."""
    import numpy as np
    from oracle import dit
    from paper_2608_16354_amd import inputs as I

    m = w.model
    P = dit.Params(W)
    mods, head_mod = dit.step_modulation(P, 0.5)
    h = I.hidden_state(m, (90,)).astype(np.float64)
    times = []
    for l in range(min(3, m.n_blocks)):
        for name in ("w_qkv", "b_qkv", "w_o", "b_o", "w_1", "b_1", "w_2", "b_2"):
            P.b(l, name)                                 # weights made before the clock starts
        t0 = time.perf_counter()
        dit.block(P, l, mods[l], h)
        times.append(time.perf_counter() - t0)
        if sum(times) >= budget_s:
            break
    t_block = sum(times) / len(times)
    x = I.latent(m, w.cfg_id, 0).astype(np.float64)
    txt = I.text(m, w.cfg_id, 0)
    t0 = time.perf_counter()
    h_in = dit.embed(P, x, txt)
    u = dit.backbone_input(P, h_in, mods[0])
    _ = np.abs(u - u).sum()
    g = h_in[: m.n_v] + h_in[: m.n_v]
    dit.euler(x, dit.head(P, head_mod, g), 0.5, 0.48)
    t_reuse = time.perf_counter() - t0
    n_ref = sum(1 for r in schedule if not r)
    n_reu = len(schedule) - n_ref
    t_sample = n_ref * (m.n_blocks * t_block + t_reuse) + n_reu * t_reuse
    cores = min(16, len(os.sched_getaffinity(0)))     # the oracle's worker and BLAS threads
    spent = sum(times) + t_reuse
    cpu, blas = host_info()
    return {"value": w.batch * m.n_v * w.K / (w.batch * t_sample), "unit": "latent token*steps/s",
            "cores": cores, "kind": "oracle", "dtype": "f64", "cpu_model": cpu, "blas": blas,
            "sample": (f"fp64 oracle: {len(times)} whole block(s) at {m.n_tok} tokens "
                       f"({', '.join(f'{t:.1f}s' for t in times)}) + one full reuse step ({t_reuse:.1f}s), "
                       f"extrapolated to the {n_ref}-refresh/{n_reu}-reuse schedule; {spent:.0f}s of CPU work")}


def run_record(api, w, probs, realized, drift, plans):
    """Per scene: the realized mask (1 = reuse), vetoes, and every drift check with its
    threshold dbar_{j,h} (the scene table of the run's refresh step j at age h) and its
    margin thr - drift (negative: vetoed by the drift)."""
    import numpy as np
    scenes = []
    for b, p in enumerate(probs):
        dbar = api.dc_schedule_dp(p).dbar
        j, age, checks = 1, 0, []
        for k in range(1, w.K + 1):
            d = float(drift[k - 1, b])
            if not np.isnan(d) and age < dbar.shape[1]:
                thr = float(dbar[j - 1, age])
                checks.append({"k": k, "drift": d, "threshold": thr, "margin": thr - d})
            if realized[k - 1, b]:
                age += 1
            else:
                j, age = k, 0
        scenes.append({"mask": "".join(str(int(v)) for v in realized[:, b]),
                       "n_veto": int(plans[b][1]), "charge_q": int(plans[b][2]),
                       "min_abs_margin": min((abs(c["margin"]) for c in checks), default=None),
                       "checks": checks})
    return {"scenes": scenes}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3, help="timed cached samples")
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="dit-30x1920-bf16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="skip the live kernel timing")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run a plain 1 GiB device copy (reference for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path, "
              "so no figure for more than one GPU is measured", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_16354_amd import api
    from paper_2608_16354_amd import inputs as I

    w = I.WORKLOADS[args.workload]
    m = w.model
    dev = "cuda:0"
    if args.copy_calibration:
        src = torch.empty(COPY_BYTES, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log(f"copy calibration: 3 x {COPY_BYTES} B device copies")
    t0 = time.time()
    W = I.Weights(m, w.cfg_id)
    dm = api.DeviceModel(W, dev)
    log(f"weights drawn and uploaded in {time.time() - t0:.1f}s")
    cal = [I.scene_problem(w, mo) for mo in I.calibration_motions(32)]
    tau = I.TAU_INF if w.tau == "inf" else api.dc_select_tau(cal, w.rho)
    motions = I.scene_motions(w)
    probs = [I.scene_problem(w, mo, tau_q=tau) for mo in motions]
    x1 = torch.from_numpy(np.stack([I.latent(m, w.cfg_id, s) for s in range(w.batch)])).to(dev)
    txt = torch.from_numpy(np.stack([I.text(m, w.cfg_id, s) for s in range(w.batch)])).to(dev)
    bufs = api.SamplerBuffers(m, w.batch, w.K, dev)
    sig = I.sigmas(w.K)
    torch.cuda.synchronize()

    last = {}

    def one_sample():
        smp = api.Sampler(dm, probs, sig, x1, txt, bufs=bufs)
        rs, ds = [], []
        for _ in range(w.K):
            r, d = smp.step()
            rs.append(r)
            ds.append(d)
        last["plans"] = [smp.plan(b) for b in range(w.batch)]
        last["drift"] = np.stack(ds)
        smp.close()
        return np.stack(rs)

    for i in range(args.warmup):
        one_sample()
        torch.cuda.synchronize()
        log(f"warmup {i + 1}/{args.warmup} done")
    prof = api.profile(list(api.L.KERNEL_CLASSES)) if not args.no_profile else None
    torch.cuda.synchronize()
    if prof:
        prof.__enter__()
    t0 = time.perf_counter()
    masks = []
    for i in range(args.steps):
        masks.append(one_sample())
        log(f"timed sample {i + 1}/{args.steps}")
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    if prof:
        prof.__exit__(None, None, None)
        kstats = prof.read()
    ms_per = 1000.0 * el / args.steps
    value = w.batch * m.n_v * w.K / (ms_per / 1000.0)
    realized = masks[-1]
    n_refresh = int((realized == 0).sum())
    fp = I.input_fingerprint(w)
    record = run_record(api, w, probs, realized, last["drift"], last["plans"])
    out = {
        "metric": "latent tokens x steps / s, cached 50-step sample",
        "value": value, "unit": "latent token*steps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": m.dtype, "data": "synthetic (seeded latents, random-init weights)",
        "config": {"workload": w.name, "blocks": m.n_blocks, "hidden": m.hidden, "heads": m.heads,
                   "video_tokens": m.n_v, "text_tokens": m.n_txt, "denoise_steps": w.K,
                   "batch": w.batch, "refresh_steps": n_refresh, "reuse_steps": int(realized.sum()),
                   "tau_q": int(tau) if tau != I.TAU_INF else None,
                   "config_hash": I.config_hash(w, tau, fp)},
        "run": record,
    }
    if prof:
        n, tot = kstats["attention"]
        avg_ms = tot / max(n, 1)
        achieved = attention_flops(m) / (avg_ms / 1000.0) / 1e12
        out["roofline"] = {"kernel": "attention", "bound": "mfma", "achieved": achieved,
                           "peak": MI355X_BF16_DENSE_TFLOPS, "unit": "TFLOP/s",
                           "frac": achieved / MI355X_BF16_DENSE_TFLOPS,
                           "traffic": traffic_from_profile("attention.hip"),
                           "launches": n, "avg_ms": avg_ms}
        # refresh steps: the block GEMMs and attention together against the dense bf16 peak
        mm = ["attention", "gemm_qkv", "gemm_out", "gemm_up", "gemm_down"]
        mm_ms = sum(kstats[c][1] for c in mm)
        blocks_run = kstats["attention"][0]
        if blocks_run and mm_ms > 0:
            fl = blocks_run * (attention_flops(m) + gemm_flops(m))
            rate = fl / (mm_ms / 1000.0) / 1e12
            out["refresh_mfma"] = {"kernels": "block GEMMs + attention", "achieved": rate,
                                   "peak": MI355X_BF16_DENSE_TFLOPS, "unit": "TFLOP/s",
                                   "frac": rate / MI355X_BF16_DENSE_TFLOPS,
                                   "ms_per_block": mm_ms / blocks_run,
                                   "per_kernel_avg_us": {c: 1000.0 * kstats[c][1] / max(kstats[c][0], 1)
                                                         for c in mm}}
        hb = hbm_bytes(m)
        # scenes processed per class over the timed samples: one launch per scene, except the
        # drift, cache-store and cache-apply launches, which take every selected scene at once
        n_checks = int(np.sum(~np.isnan(last["drift"])))
        n_reuse = int(realized.sum())
        units = {"drift": n_checks + n_refresh, "cache_store": n_refresh, "cache_apply": n_reuse}
        out["hbm_kernels"] = {}
        for c, nbytes in hb.items():
            n_c, ms_c = kstats[c]
            if n_c:
                n_s = units[c] * args.steps if c in units else n_c
                gbs = nbytes * n_s / (ms_c / 1000.0) / 1e9
                out["hbm_kernels"][c] = {"avg_us_per_scene": 1000.0 * ms_c / n_s, "launches": n_c,
                                         "scenes": n_s, "algorithmic_bytes_per_scene": nbytes,
                                         "GB/s": gbs, "frac": gbs / MI355X_HBM_GBPS}
    # refresh FLOPs of the executed schedule over the whole sample time (reuse steps included)
    out["sample_tflops"] = refresh_flops(m) * n_refresh / (ms_per / 1000.0) / 1e12
    if not args.no_cpu_baseline:
        log("cpu baseline (fp64 oracle, bounded sample)")
        out["cpu_baseline"] = cpu_baseline(w, W, realized[:, 0].tolist())
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

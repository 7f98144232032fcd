"""Write the oracle's cached sample of a workload for the GPU parity tests.
Calls only the oracle and the seeded input generator.

    python tests/golden/make_oracle_artifacts.py dit-12x1152-bf16
    python tests/golden/make_oracle_artifacts.py dit-12x1152-bf16 --thr 0.05 --tag veto
    python tests/golden/make_oracle_artifacts.py dit-30x1920-bf16 --every-step --checkpoint <file>

The file `oracle_<workload>[-<tag>].npz` holds the latent after `steps` steps
(float32), the realized, planned and vetoed flags of every step, every observed
drift (rel-L1 and rel-L2; NaN where no check ran) with the threshold it was
compared with, the plan as it stood after the last step, the veto count, the
charge, the budget tau and a fingerprint of the generated inputs.  With
--every-step the file is rewritten after each step (a long run leaves a valid
truncated artefact at every point); with --checkpoint the whole controller state is
saved after each step to that file (this script's own pickle) and a run started
with an existing checkpoint continues after its step; --block-dir additionally keeps
each block's output of the step in progress (keyed by the sha256 of the block's
input), so an interrupted refresh step picks up after its last finished block.
"""
import argparse
import hashlib
import os
import pickle
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import budget, runtime  # noqa: E402
from paper_2608_16354_amd import inputs as I  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))


fingerprint = I.input_fingerprint      # hash of the generated inputs (a changed generator is detected)


def artefact_path(name, tag=None):
    return os.path.join(HERE, f"oracle_{name}{'' if not tag else '-' + tag}.npz")


def _write(path, name, thr, tau, fp, k, x, records, plan, seconds):
    nan = np.nan
    rec = {
        "x": x.astype(np.float32),
        "steps": np.int32(k),
        "realized": np.array([r.realized for r in records], np.uint8),
        "planned": np.array([r.planned for r in records], np.uint8),
        "vetoed": np.array([bool(r.vetoed) for r in records], np.uint8),
        "drift": np.array([nan if r.drift is None else r.drift for r in records]),
        "drift_l2": np.array([nan if r.drift_l2 is None else r.drift_l2 for r in records]),
        "threshold": np.array([nan if r.threshold is None else r.threshold for r in records]),
        "plan": np.array(plan, np.uint8),
        "n_veto": np.int32(sum(bool(r.vetoed) for r in records)),
        "tau_q": np.int64(tau),
        "thr": np.float64(thr),
        "fingerprint": np.array(fp),
        "workload": np.array(name),
        "oracle_seconds": np.float64(seconds),
    }
    tmp = path + ".tmp.npz"
    np.savez(tmp, **rec)
    os.replace(tmp, path)


class BlockStore:
    """Block outputs of the refresh step in progress, on disk, keyed by the block index
    and the sha256 of the block's input (a stale entry never matches)."""

    def __init__(self, root):
        self.root = root
        os.makedirs(root, exist_ok=True)

    def _key(self, l, h):
        return os.path.join(self.root, f"block{l:03d}-{hashlib.sha256(h.tobytes()).hexdigest()[:32]}.npy")

    def load(self, l, h):
        path = self._key(l, h)
        return np.load(path, allow_pickle=False) if os.path.exists(path) else None

    def save(self, l, h, out):
        path = self._key(l, h)
        np.save(path + ".tmp.npy", out)
        os.replace(path + ".tmp.npy", path)

    def clear(self):
        for f in os.listdir(self.root):
            if f.startswith("block"):
                os.remove(os.path.join(self.root, f))


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("name", nargs="?", default="dit-12x1152-bf16")
    ap.add_argument("--thr", type=float, default=None, help="drift threshold (default: the workload's)")
    ap.add_argument("--tag", default=None, help="suffix of the file name")
    ap.add_argument("--steps", type=int, default=None, help="stop after this many steps")
    ap.add_argument("--every-step", action="store_true", help="rewrite the file after every step")
    ap.add_argument("--checkpoint", default=None, help="state file to save after each step and resume from")
    ap.add_argument("--block-dir", default=None, help="directory for the block outputs of the step in progress")
    a = ap.parse_args(argv)
    w = I.WORKLOADS[a.name]
    thr = w.thr if a.thr is None else a.thr
    cal = [I.scene_problem(w, m) for m in I.calibration_motions(32)]
    tau = budget.select_tau(cal, w.rho)
    p = I.scene_problem(w, w.motions[0], tau_q=tau, thr=thr)
    W = I.Weights(w.model, w.cfg_id)
    fp = fingerprint(w)
    path = artefact_path(a.name, a.tag)
    t0 = time.time()

    resume = None
    if a.checkpoint and os.path.exists(a.checkpoint):
        with open(a.checkpoint, "rb") as f:
            resume = pickle.load(f)
        print(f"{a.name}: resuming after step {resume['k']}", flush=True)

    store = BlockStore(a.block_dir) if a.block_dir else None

    def on_step(k, x, records, plan, state):
        W.drop()          # the oracle keeps its own float64 copies of every tensor it used
        if a.checkpoint:
            tmp = a.checkpoint + ".tmp"
            with open(tmp, "wb") as f:
                pickle.dump(state, f, protocol=pickle.HIGHEST_PROTOCOL)
            os.replace(tmp, a.checkpoint)
        if store is not None:
            store.clear()                 # the step is in the checkpoint
        r = records[-1]
        d = "" if r.drift is None else f" drift {r.drift:.6f} thr {r.threshold:.4f}"
        print(f"{a.name} step {k}: {'reuse' if r.realized else 'full'}{' (vetoed)' if r.vetoed else ''}"
              f"{d}  [{time.time() - t0:.0f} s]", flush=True)
        if a.every_step:
            _write(path, a.name, thr, tau, fp, k, x, records, plan, time.time() - t0)

    res = runtime.sample(W, I.latent(w.model, w.cfg_id, 0), I.text(w.model, w.cfg_id, 0),
                         I.sigmas(w.K), p, steps=a.steps, on_step=on_step, resume=resume,
                         block_memo=store)
    k = len(res.records)
    _write(path, a.name, thr, tau, fp, k, res.x, res.records, res.plan, time.time() - t0)
    print(f"{a.name}: {time.time() - t0:.1f} s, {k} steps, realized "
          f"{''.join(map(str, res.realized))}, vetoes {sum(r.vetoed for r in res.records)}")


if __name__ == "__main__":
    main()

"""Write the oracle's full cached sample of the 12-block bf16 workload
(dit-12x1152-bf16: 3,584 + 120 tokens, 30 steps, stationary plan) for the GPU
parity test.  Calls only the oracle and the seeded input generator.

    python tests/golden/make_oracle_artifacts.py
"""
import hashlib
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import budget, runtime  # noqa: E402
from paper_2608_16354_amd import inputs as I  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))


def fingerprint(w):
    """Hash of the generated inputs, so a changed generator is detected."""
    W = I.Weights(w.model, w.cfg_id)
    h = hashlib.sha256()
    for a in (I.latent(w.model, w.cfg_id, 0), I.text(w.model, w.cfg_id, 0), W.get("w_pe"),
              W.get("w_head"), W.block(0, "w_qkv")[:64], W.block(w.model.n_blocks - 1, "w_2")[:64]):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def main(name="dit-12x1152-bf16"):
    w = I.WORKLOADS[name]
    cal = [I.scene_problem(w, m) for m in I.calibration_motions(32)]
    tau = budget.select_tau(cal, w.rho)
    p = I.scene_problem(w, w.motions[0], tau_q=tau)
    W = I.Weights(w.model, w.cfg_id)
    t0 = time.time()
    res = runtime.sample(W, I.latent(w.model, w.cfg_id, 0), I.text(w.model, w.cfg_id, 0),
                         I.sigmas(w.K), p)
    print(f"{name}: {time.time() - t0:.1f} s, realized {''.join(map(str, res.realized))}")
    drift = np.array([np.nan if r.drift is None else r.drift for r in res.records])
    np.savez(os.path.join(HERE, f"oracle_{name}.npz"), x=res.x.astype(np.float32),
             realized=np.array(res.realized, np.uint8), drift=drift, tau_q=np.int64(tau),
             fingerprint=np.array(fingerprint(w)))


if __name__ == "__main__":
    main(*sys.argv[1:])

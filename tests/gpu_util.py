"""Helpers for the GPU parity tests (shared seeded inputs, error metrics)."""
import sys

import numpy as np

from paper_2608_16354_amd import inputs as I


def say(*a):
    """Name the case before a GPU step, flushed (a faulting kernel can end the process)."""
    print("[gpu]", *a, flush=True)
    sys.stdout.flush()


def rel_l2(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def t(a, dev, dtype=None):
    import torch
    x = torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    return x if dtype is None else x.to(dtype)


def mod_input(m, key, std=0.1):
    """A seeded [6, d] modulation vector set (shift1, scale1, gate1, shift2, scale2, gate2)."""
    return I.normal((6, m.hidden), std, (7000,) + tuple(key))

"""Helpers shared by the GPU parity tests (comparison metrics and device staging)."""
import json
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

# Tolerances.  Weights after one pooled update: max |w_gpu - w_ref| / max |w_ref|
# per layer; per-epoch summed squared error: relative difference.
W_TOL = 1e-5
SSE_TOL = 1e-3


def layer_views(sizes, flat):
    out, o = [], 0
    for l in range(len(sizes) - 1):
        r, c = sizes[l] + 1, sizes[l + 1]
        out.append(np.asarray(flat[o:o + r * c], dtype=np.float64).reshape(r, c))
        o += r * c
    return out


def rel_maxabs(sizes, got, ref):
    """Per-layer max |got - ref| / max |ref|."""
    res = []
    for g, r in zip(layer_views(sizes, got), layer_views(sizes, ref)):
        den = np.max(np.abs(r))
        res.append(float(np.max(np.abs(g - r)) / (den if den > 0 else 1.0)))
    return res


def rel(a, b):
    return abs(a - b) / abs(b) if b != 0 else abs(a)


def load_golden(name):
    p = os.path.join(GOLDEN, f"epoch_{name}.json")
    if not os.path.exists(p):
        return None
    with open(p) as f:
        return json.load(f)


def to_device(w, dev):
    """Inputs (dense or active indices) and targets of a workload as device tensors."""
    import torch
    t = torch.from_numpy(w.targets).to(dev)
    if w.active is not None:
        return None, torch.from_numpy(w.active).to(dev), t
    return torch.from_numpy(w.inputs).to(dev), None, t

"""Shared helpers for the tests: metrics and oracle calls on device tensors."""

import numpy as np
import torch

from oracle import linsimp as O


def rel_l2(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))


# per-row bars of the parity tests: a single wrong row (one anchor tile, one
# feature block or one partial slot lost) moves a whole-tensor relative L2 by
# little, so every row is held to its own bar as well
ROW_TOL = {"f32": 1e-4, "bf16": 5e-2}


def row_max_rel(got, ref, floor=1e-2, scale=None) -> float:
    """Largest per-row relative L2 error (rows = all but the last axis).  A row
    whose reference norm is below ``floor`` times ``scale`` (default: the RMS
    row norm of ``ref``) is measured against that floor instead of its own
    norm, so rows that are nearly zero by construction do not divide by ~0."""
    got = np.asarray(got, np.float64).reshape(-1, np.shape(got)[-1])
    ref = np.asarray(ref, np.float64).reshape(-1, np.shape(ref)[-1])
    num = np.linalg.norm(got - ref, axis=1)
    den = np.linalg.norm(ref, axis=1)
    if scale is None:
        scale = np.linalg.norm(ref) / np.sqrt(ref.shape[0])
    return float(np.max(num / np.maximum(den, max(floor * scale, 1e-300))))


def f64(t: torch.Tensor) -> np.ndarray:
    """Exact upcast of a device tensor's values to float64 on the host."""
    return t.detach().float().cpu().double().numpy()


def oracle_forward(x, w, pairs, eps=O.EPS):
    """float64 oracle outputs for the (b, h) pairs, from the same input values."""
    out = {}
    for b, h in pairs:
        out[(b, h)] = O.forward_recurrent(f64(x["q"][b, h]), f64(x["k"][b, h]), f64(x["v"][b, h]),
                                          f64(x["r"][b, h]), f64(x["u"][b, h]), f64(x["omega"][h]),
                                          w, eps)
    return out


def oracle_backward(x, w, pairs, eps=O.EPS):
    out = {}
    for b, h in pairs:
        out[(b, h)] = O.backward(f64(x["q"][b, h]), f64(x["k"][b, h]), f64(x["v"][b, h]),
                                 f64(x["r"][b, h]), f64(x["u"][b, h]), f64(x["omega"][h]),
                                 w, f64(x["dO"][b, h]), eps)
    return out

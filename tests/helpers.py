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


# unit roundoff of the operand types (round to nearest)
UNIT_ROUNDOFF = {"f32": 2.0 ** -24, "bf16": 2.0 ** -9}


def row_max_rel(got, ref, window=64, where=False, slack=None):
    """Largest per-row relative L2 error over arrays [..., n, width] (the
    second-to-last axis runs along one sequence).  Row i is measured against
    max(|ref_i|, local_i), local_i being the RMS norm of the reference rows
    within `window` positions of i in the same sequence (and at least 1e-3 of
    the tensor's RMS row norm).  A row whose exact value cancels to ~0 (dq of
    a sequence's first row is zero by definition: its output is v_0 (*) u_0
    whatever q_0 is) is thus judged on the scale of the rows around it, which
    is the scale of the terms that cancel in it; a wrong row, whose error is
    of the order of its own norm, is still caught.  ``slack`` (same leading
    shape as the rows) is an absolute allowance per row taken off the error
    first: the rounding bound of a row whose exact value cancels between much
    larger terms (u times the sum of their absolute values)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    n, width = ref.shape[-2], ref.shape[-1]
    got = got.reshape(-1, n, width)
    ref = ref.reshape(-1, n, width)
    err = np.linalg.norm(got - ref, axis=-1)                 # [S, n]
    if slack is not None:
        err = np.maximum(err - np.asarray(slack, np.float64).reshape(err.shape), 0.0)
    nr2 = np.sum(ref * ref, axis=-1)
    # sum of nr2 over rows [i - window, i + window] of each sequence
    c = np.concatenate([np.zeros((nr2.shape[0], 1)), np.cumsum(nr2, axis=-1)], axis=-1)
    lo = np.maximum(np.arange(n) - window, 0)
    hi = np.minimum(np.arange(n) + window + 1, n)
    local = np.sqrt((c[:, hi] - c[:, lo]) / (hi - lo))
    glob = np.sqrt(np.mean(nr2))
    den = np.maximum(np.maximum(np.sqrt(nr2), local), max(1e-3 * glob, 1e-300))
    ratio = err / den
    if where:      # (value, sequence, row, error, own norm, local RMS norm), norms over the RMS
        s_, i_ = np.unravel_index(np.argmax(ratio), ratio.shape)
        return (float(ratio[s_, i_]), int(s_), int(i_), float(err[s_, i_] / glob),
                float(np.sqrt(nr2[s_, i_]) / glob), float(local[s_, i_] / glob))
    return float(np.max(ratio))


def row_report(got, ref, k=3):
    """The k worst rows by error / RMS row norm: (row, |err|/rms, |ref_row|/rms)."""
    got = np.asarray(got, np.float64).reshape(-1, np.shape(got)[-1])
    ref = np.asarray(ref, np.float64).reshape(-1, np.shape(ref)[-1])
    rms = np.linalg.norm(ref) / np.sqrt(ref.shape[0])
    e = np.linalg.norm(got - ref, axis=1) / rms
    nr = np.linalg.norm(ref, axis=1) / rms
    idx = np.argsort(-e)[:k]
    return [(int(i), float(e[i]), float(nr[i])) for i in idx]


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


def oracle_backward(x, w, pairs, eps=O.EPS, scales=None):
    """float64 oracle gradients for the (b, h) pairs; with ``scales`` (a dict)
    also the per-key absolute term scale of dk, scales[(b, h)]."""
    out = {}
    for b, h in pairs:
        ts = {} if scales is not None else None
        out[(b, h)] = O.backward(f64(x["q"][b, h]), f64(x["k"][b, h]), f64(x["v"][b, h]),
                                 f64(x["r"][b, h]), f64(x["u"][b, h]), f64(x["omega"][h]),
                                 w, f64(x["dO"][b, h]), eps, term_scale=ts)
        if scales is not None:
            scales[(b, h)] = ts["dk"]
    return out

"""GPU parity of the full head (L2 normalisation + temperature, core, gated
RMSNorm; per-head and channel-wise gates) against the float64 oracle of
oracle.layer, through the C ABI (include/linsimp_head.h).

Outputs and the gradients of q, k, v, r, u and of the channel-gate logits are
held to relative L2 <= 1e-4 (float32) and <= 2e-2 (bf16), the output and the
five stream gradients also per row (<= 1e-4 float32, <= 5e-2 bf16, each row
against the larger of its own norm and the RMS norm of the rows within w
positions, helpers.row_max_rel); a gradient that is
zero by definition (n = 1; reference norm below 1e-6 of the largest of the
five) is measured against the largest reference gradient norm.  The per-head sums
dtau = <q_hat, dq_core> and dgamma = <dy, o_hat g (1 - g)> are inner products
over all rows of a head; the gradient bar on their factor (relative L2 <= tol)
bounds their error by tol |a| |b| (Cauchy-Schwarz), which is the bar used
for them.
"""

import numpy as np
import pytest
import torch

from oracle import layer as LY
from paper_2608_09307_amd import linsimp as L
from paper_2608_09307_amd.workloads import Workload, make_head_params, make_inputs

from helpers import ROW_TOL, f64, rel_l2, row_max_rel

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
TOL = {"f32": 1e-4, "bf16": 2e-2}
NAMES = ("dq", "dk", "dv", "dr", "du")


def _oracle(x, p, wl, pairs, channel):
    ys, grads, scale = {}, {}, {}
    for b, h in pairs:
        args = [f64(x[nm][b, h]) for nm in ("q", "k", "v", "r", "u")]
        om = f64(x["omega"][h])
        tau = float(p["tau"][h])
        gate = f64(p["gate"][b, h]) if channel else float(p["gate"][h])
        ys[(b, h)], _ = LY.head_forward(*args, om, wl.w, tau, gate)
        parts = {}
        grads[(b, h)] = LY.head_backward(*args, om, wl.w, tau, gate, f64(x["dO"][b, h]), parts=parts)
        scale[(b, h)] = {k: float(np.sum(v * v)) for k, v in parts.items()}
    return ys, grads, scale


def _cs_scale(scale, pairs, H, a, b, big):
    """Cauchy-Schwarz scale |a| |b| of a per-head inner product over its rows
    (|b| taken as `big`, the largest reference gradient norm, where b is zero
    by definition, as the core gradients of q at n = 1)."""
    sa, sb = np.zeros(H), np.zeros(H)
    for (bb, h) in pairs:
        sa[h] += scale[(bb, h)][a]
        sb[h] += scale[(bb, h)][b]
    nb = np.sqrt(sb)
    return np.sqrt(sa) * np.where(nb > 1e-6 * big, nb, big)


def _run(wl: Workload, channel: bool, zero_rows: bool = False, pairs=None):
    print(f"[head] {wl} channel={channel} zero_rows={zero_rows}", flush=True)
    x = make_inputs(wl, device=DEV, with_grad=True)
    p = make_head_params(wl, device=DEV, channel_gate=channel)
    if zero_rows:                       # rows below the norm floor
        x["q"][:, :, 3] = 0
        x["r"][:, :, 5] = 0
        x["k"][:, :, 7] = 0
    y, saved = L.head_fwd(x["q"], x["k"], x["v"], x["r"], x["u"], x["omega"], wl.w, p["tau"], p["gate"])
    g = L.head_bwd(x["q"], x["k"], x["v"], x["r"], x["u"], x["omega"], wl.w, p["tau"], p["gate"],
                   saved, x["dO"])
    torch.cuda.synchronize()
    if pairs is None:
        pairs = [(b, h) for b in range(wl.B) for h in range(wl.H)]
    heads = sorted({h for _, h in pairs})
    ys, ref, scale = _oracle(x, p, wl, pairs, channel)
    tol = TOL[wl.dtype]
    ygot, yref = np.stack([f64(y[b, h]) for b, h in pairs]), np.stack([ys[q] for q in pairs])
    errs = {"y": rel_l2(ygot, yref)}
    rows = {"y": row_max_rel(ygot, yref)}
    exps = [np.stack([ref[q][gi] for q in pairs]) for gi in range(len(NAMES))]
    big = max(np.linalg.norm(e) for e in exps)
    for gi, nm in enumerate(NAMES):
        got = np.stack([f64(g[gi][b, h]) for b, h in pairs])
        assert np.all(np.isfinite(got)), nm
        nr = np.linalg.norm(exps[gi])
        zero = nr <= 1e-6 * big
        errs[nm] = float(np.linalg.norm(got - exps[gi]) / (big if zero else nr))
        if not zero:                                   # (a zero tensor has no row scale)
            rows[nm] = row_max_rel(got, exps[gi])
    dtau_ref = np.zeros(wl.H)
    for (b, h) in pairs:
        dtau_ref[h] += ref[(b, h)][5]
    cs = _cs_scale(scale, pairs, wl.H, "q_hat", "dq_core", big)
    errs["dtau"] = float(np.max((np.abs(g[5].cpu().double().numpy() - dtau_ref) / np.maximum(cs, 1e-300))[heads]))
    if channel:
        got = np.stack([f64(g[6][b, h]) for b, h in pairs])
        errs["dgate"] = rel_l2(got, np.stack([ref[q][6] for q in pairs]))
    else:
        dg_ref = np.zeros(wl.H)
        for (b, h) in pairs:
            dg_ref[h] += ref[(b, h)][6]
        cs = _cs_scale(scale, pairs, wl.H, "dy", "gate_factor", big)
        errs["dgamma"] = float(np.max((np.abs(g[6].cpu().double().numpy() - dg_ref) / np.maximum(cs, 1e-300))[heads]))
    print("      " + " ".join(f"{k}={v:.2e}" for k, v in errs.items()), flush=True)
    print("      rows " + " ".join(f"{k}={v:.2e}" for k, v in rows.items()), flush=True)
    for nm, e in errs.items():
        assert e <= tol, (nm, e)
    for nm, e in rows.items():
        assert e <= ROW_TOL[wl.dtype], (nm, "row", e)
    return x, p, y, saved, g


@pytest.mark.parametrize("channel", [False, True])
@pytest.mark.parametrize("D,m,n,w,B,H,dt", [
    (32, 32, 100, 20, 1, 2, "f32"),
    (64, 64, 77, 64, 2, 1, "f32"),
    (128, 128, 300, 64, 1, 2, "bf16"),
    (64, 64, 257, 48, 2, 2, "bf16"),
    (32, 32, 130, 64, 1, 1, "bf16"),
    (128, 256, 150, 64, 1, 2, "bf16"),   # two feature blocks
])
def test_head_parity(D, m, n, w, B, H, dt, channel):
    _run(Workload("head", B, H, n, D, D, m, w, dt, "fwdbwd", seed=61), channel)


def test_head_layer16k_sampled_head():
    """The 16k layer at full size (the launch configuration of bench.py --head):
    head 9 of both sequences, so dtau[9] and dgamma[9] are complete sums."""
    from paper_2608_09307_amd.workloads import WORKLOADS
    _run(WORKLOADS["layer16k_bf16"], False, pairs=[(0, 9), (1, 9)])


@pytest.mark.parametrize("n,dt", [(1, "bf16"), (31, "f32")])
def test_head_short_sequences(n, dt):
    _run(Workload("head_short", 1, 2, n, 32, 32, 32, 64, dt, "fwdbwd", seed=64), True)


def test_head_rows_below_the_norm_floor():
    _run(Workload("head0", 1, 2, 40, 32, 32, 32, 16, "f32", "fwdbwd", seed=62), False, zero_rows=True)


def test_head_backward_is_bitwise_reproducible():
    wl = Workload("head_det", 2, 2, 500, 128, 128, 128, 64, "bf16", "fwdbwd", seed=63)
    x = make_inputs(wl, device=DEV, with_grad=True)
    p = make_head_params(wl, device=DEV)
    args = (x["q"], x["k"], x["v"], x["r"], x["u"], x["omega"], wl.w, p["tau"], p["gate"])
    y, saved = L.head_fwd(*args)
    g1 = L.head_bwd(*args, saved, x["dO"])
    g2 = L.head_bwd(*args, saved, x["dO"])
    torch.cuda.synchronize()
    for a, b in zip(g1, g2):
        assert torch.equal(a, b)


def test_head_backward_reusing_forward_states_is_bitwise_equal():
    import ctypes
    wl = Workload("head_reuse", 1, 2, 300, 128, 128, 128, 64, "bf16", "fwdbwd", seed=65)
    x = make_inputs(wl, device=DEV, with_grad=True)
    p = make_head_params(wl, device=DEV, channel_gate=True)
    args = (x["q"], x["k"], x["v"], x["r"], x["u"], x["omega"], wl.w, p["tau"], p["gate"])
    d = L.dims_of(x["q"], x["v"], x["omega"], wl.w)
    ws = L._aligned_bytes(int(L.lib().linsimp_head_workspace_size(ctypes.byref(d), 1)), DEV)
    y, saved = L.head_fwd(*args, workspace=ws)
    g_re = tuple(t.clone() for t in L.head_bwd(*args, saved, x["dO"], workspace=ws, reuse_states=True))
    g_rc = L.head_bwd(*args, saved, x["dO"])
    torch.cuda.synchronize()
    for a_, b_ in zip(g_re, g_rc):
        assert torch.equal(a_, b_)

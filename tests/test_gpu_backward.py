"""GPU parity of the backward pass against the float64 oracle (through the C ABI).

Each gradient (dq, dk, dv, dr, du) is held to relative L2 <= 1e-4 for float32
inputs and <= 2e-2 for bf16 inputs, and every gradient row to its own relative
L2 bar (1e-4 for float32, 5e-2 for bf16), measured against the larger of its
own norm and the RMS norm of the rows within w positions (helpers.row_max_rel:
dq of a sequence's first row is zero by definition, and the bf16 output the
backward receives leaves a rounding residue there of the size of its
neighbours' rounding).  dk rows also get the first-order rounding bound of
their terms as slack (two bf16 unit roundoffs times the absolute term sum,
oracle.linsimp.backward's term_scale): a key whose exact gradient cancels
between much larger terms carries their rounding.  A gradient that is
exactly zero in the
definition (n = 1: the output is v_0 (*) u_0 whatever q, k, r are; its
reference norm is below 1e-6 of the largest of the five) has no relative
scale; its error is measured against the largest reference gradient norm,
the size of the terms that cancel in it.  Shapes cover several chunks, ragged tails,
windows that are not multiples of 32, w = 1, single rows and single partial
chunks, both feature-block layouts (m = 256 splits features in two) and
full-size sampled heads of the 16k layer and the 64k stress shape.
"""

import numpy as np
import pytest
import torch

from paper_2608_09307_amd import linsimp as L
from paper_2608_09307_amd.workloads import WORKLOADS, Workload, make_inputs

from helpers import ROW_TOL, UNIT_ROUNDOFF, f64, oracle_backward, rel_l2, row_max_rel

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
TOL = {"f32": 1e-4, "bf16": 2e-2}
NAMES = ("dq", "dk", "dv", "dr", "du")


def _run(wl: Workload, pairs=None):
    print(f"[bwd] {wl}", flush=True)
    x = make_inputs(wl, device=DEV, with_grad=True)
    out, stats = L.fwd(x["q"], x["k"], x["v"], x["r"], x["u"], x["omega"], wl.w)
    grads = L.bwd(x["q"], x["k"], x["v"], x["r"], x["u"], x["omega"], wl.w, out, stats, x["dO"])
    torch.cuda.synchronize()
    if pairs is None:
        pairs = [(b, h) for b in range(wl.B) for h in range(wl.H)]
    tscale = {}
    ref = oracle_backward(x, wl.w, pairs, scales=tscale)
    # dk of a key whose exact gradient cancels between much larger terms (a
    # dominant feature fed by many (row, anchor) pairs of both signs) carries
    # the rounding of those terms: two unit roundoffs of their absolute sum
    # are allowed on top of the row bar
    slack_dk = 2 * UNIT_ROUNDOFF[wl.dtype] * np.stack([tscale[p] for p in pairs])
    errs, rows = {}, {}
    exps = [np.stack([ref[p][gi] for p in pairs]) for gi in range(len(NAMES))]
    big = max(np.linalg.norm(e) for e in exps)
    for gi, nm in enumerate(NAMES):
        got = np.stack([f64(grads[gi][b, h]) for b, h in pairs])
        exp = exps[gi]
        assert np.all(np.isfinite(got)), nm
        zero = np.linalg.norm(exp) <= 1e-6 * big      # zero by definition (n = 1)
        den = big if zero else np.linalg.norm(exp)
        errs[nm] = float(np.linalg.norm(got - exp) / den)
        if not zero:                                   # (a zero tensor has no row scale)
            slack = slack_dk if nm == "dk" else None
            rows[nm] = row_max_rel(got, exp, slack=slack)
            if rows[nm] > ROW_TOL[wl.dtype]:
                print(f"      worst {nm} row (value, seq, row, err, norm, local):",
                      row_max_rel(got, exp, where=True, slack=slack), flush=True)
    print("      " + " ".join(f"{k}={v:.2e}" for k, v in errs.items()), flush=True)
    print("      rows " + " ".join(f"{k}={v:.2e}" for k, v in rows.items()), flush=True)
    for nm, e in errs.items():
        assert e <= TOL[wl.dtype], (nm, e)
    for nm, e in rows.items():
        assert e <= ROW_TOL[wl.dtype], (nm, "row", e)
    return x, grads


@pytest.mark.parametrize("D,m,n,w,B,H", [
    (32, 32, 100, 20, 1, 2),      # window not a multiple of 32, ragged
    (64, 64, 333, 64, 1, 1),      # several query-sweep segments, ragged tail
    (32, 64, 70, 1, 2, 1),        # w = 1
    (64, 32, 47, 64, 1, 1),       # a chunk and a half
])
def test_backward_f32_structure(D, m, n, w, B, H):
    _run(Workload("f32_bwd", B, H, n, D, D, m, w, "f32", "fwdbwd", seed=31))


@pytest.mark.parametrize("D,m,n,w", [(128, 128, 700, 64), (64, 64, 513, 64), (128, 64, 300, 40),
                                     (128, 256, 400, 64), (32, 32, 200, 64), (64, 128, 257, 48)])
def test_backward_bf16_shapes(D, m, n, w):
    _run(Workload("bf16_bwd", 1, 2, n, D, D, m, w, "bf16", "fwdbwd", seed=32,
                  boost_frac=0.05 if m == 256 else 0.0, boost=4.0))


@pytest.mark.parametrize("D,m,n,w,dt", [
    (32, 32, 1, 64, "f32"),       # a single row
    (128, 128, 1, 64, "bf16"),
    (128, 128, 31, 64, "bf16"),   # one partial chunk
    (64, 64, 33, 5, "bf16"),      # chunk boundary + 1, short window
    (128, 256, 40, 64, "bf16"),   # two feature blocks, short sequence
])
def test_backward_edge_lengths(D, m, n, w, dt):
    _run(Workload("edge_bwd", 1, 2, n, D, D, m, w, dt, "fwdbwd", seed=34))


@pytest.mark.parametrize("D,m,w,n,dt", [(128, 64, 96, 400, "bf16"), (128, 64, 128, 433, "bf16"),
                                        (64, 64, 100, 300, "bf16"), (32, 32, 128, 290, "bf16"),
                                        (64, 64, 96, 250, "f32"), (32, 64, 128, 333, "f32"),
                                        (128, 64, 128, 40, "bf16")])
def test_backward_wide_windows(D, m, w, n, dt):
    """Windows of three and four anchor tiles (64 < w <= 128, w * m <= 8192):
    the du sweep stages NA + 1 row chunks and pairs chunk kt with kt + NA."""
    _run(Workload("wide_bwd", 1, 2, n, D, D, m, w, dt, "fwdbwd", seed=42))


@pytest.mark.parametrize("D,m,n,w,dt", [(128, 128, 250, 64, "bf16"), (64, 64, 200, 40, "f32")])
def test_backward_tile_grid_multiple_of_8(D, m, n, w, dt):
    """Tiles x heads a multiple of eight (here 8 x 4 and 7 x 8): the sweeps
    deal their tiles to the XCDs in contiguous runs, every row checked."""
    B, H = (2, 2) if n == 250 else (2, 4)
    _run(Workload("grid8_bwd", B, H, n, D, D, m, w, dt, "fwdbwd", seed=36))


def test_backward_layer16k_sampled_heads():
    _run(WORKLOADS["layer16k_bf16"], pairs=[(1, 9), (0, 2)])


def test_backward_stress64k_sampled_head():
    _run(WORKLOADS["stress64k_m256"], pairs=[(0, 21)])


def test_backward_bitwise_deterministic():
    """No atomics anywhere: two backward calls give identical bits."""
    wl = Workload("bf16_det", 1, 2, 700, 128, 128, 128, 64, "bf16", "fwdbwd", seed=33)
    x = make_inputs(wl, device=DEV, with_grad=True)
    out, stats = L.fwd(x["q"], x["k"], x["v"], x["r"], x["u"], x["omega"], wl.w)
    g1 = L.bwd(x["q"], x["k"], x["v"], x["r"], x["u"], x["omega"], wl.w, out, stats, x["dO"])
    g1 = tuple(t.clone() for t in g1)
    g2 = L.bwd(x["q"], x["k"], x["v"], x["r"], x["u"], x["omega"], wl.w, out, stats, x["dO"])
    torch.cuda.synchronize()
    for nm, a_, b_ in zip(NAMES, g1, g2):
        assert torch.equal(a_, b_), nm


@pytest.mark.parametrize("D,m,n,w,dt", [(128, 128, 700, 64, "bf16"), (128, 256, 300, 64, "bf16"),
                                        (32, 32, 100, 20, "f32")])
def test_backward_reusing_forward_states_is_bitwise_equal(D, m, n, w, dt):
    """linsimp_bwd_ex with LINSIMP_BWD_REUSE_STATES on the workspace the forward
    used gives the bits of the recomputing backward."""
    wl = Workload("reuse", 2, 2, n, D, D, m, w, dt, "fwdbwd", seed=35)
    x = make_inputs(wl, device=DEV, with_grad=True)
    d = L.dims_of(x["q"], x["v"], x["omega"], wl.w)
    ws = L.alloc_workspace(d, True, DEV)
    args = (x["q"], x["k"], x["v"], x["r"], x["u"], x["omega"], wl.w)
    out, stats = L.fwd(*args, workspace=ws)
    g_re = tuple(t.clone() for t in L.bwd(*args, out, stats, x["dO"], workspace=ws, reuse_states=True))
    g_rc = L.bwd(*args, out, stats, x["dO"])
    torch.cuda.synchronize()
    for nm, a_, b_ in zip(NAMES, g_re, g_rc):
        assert torch.equal(a_, b_), nm


@pytest.mark.parametrize("w,n", [(1, 70), (33, 97)])
def test_backward_two_feature_blocks_short_windows(w, n):
    """m = 256 (float32 du/dr partials per feature block, then summed) with
    one anchor tile per row (w <= 32), w = 1 included."""
    _run(Workload("m256_short_w", 1, 2, n, 128, 128, 256, w, "bf16", "fwdbwd", seed=36))


def test_reuse_flag_refuses_a_workspace_with_other_states():
    """linsimp_bwd_ex with LINSIMP_BWD_REUSE_STATES is refused (status -1,
    nothing launched) when the workspace holds the states of a forward with
    another k, v, omega or other dims, or when a prefill has overwritten them;
    the matching call goes through."""
    wl = Workload("reuse_guard", 1, 2, 100, 64, 64, 64, 64, "bf16", "fwdbwd", seed=38)
    x = make_inputs(wl, device=DEV, with_grad=True)
    d = L.dims_of(x["q"], x["v"], x["omega"], wl.w)
    ws = L.alloc_workspace(d, True, DEV)
    args = [x["q"], x["k"], x["v"], x["r"], x["u"], x["omega"], wl.w]
    out, stats = L.fwd(*args, workspace=ws)
    for pos, nm in ((1, "k"), (2, "v"), (5, "omega")):
        other = list(args)
        other[pos] = args[pos].clone()
        with pytest.raises(L.LinSimpError) as e:
            L.bwd(*other, out, stats, x["dO"], workspace=ws, reuse_states=True)
        assert e.value.status == -1 and "other k, v or omega" in str(e.value), nm
    with pytest.raises(L.LinSimpError) as e:             # other dims: another window
        L.bwd(*args[:6], 32, out, stats, x["dO"], workspace=ws, reuse_states=True)
    assert e.value.status == -1 and "other dims" in str(e.value)
    g = tuple(t.clone() for t in L.bwd(*args, out, stats, x["dO"], workspace=ws, reuse_states=True))
    ref = L.bwd(*args, out, stats, x["dO"])
    torch.cuda.synchronize()
    for nm, a_, b_ in zip(NAMES, g, ref):
        assert torch.equal(a_, b_), nm
    L.prefill(x["k"], x["v"], x["r"], x["u"], x["omega"], wl.w, workspace=ws)
    with pytest.raises(L.LinSimpError) as e:
        L.bwd(*args, out, stats, x["dO"], workspace=ws, reuse_states=True)
    assert e.value.status == -1 and "no forward" in str(e.value)
    torch.cuda.synchronize()

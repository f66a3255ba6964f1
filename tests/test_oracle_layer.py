"""Pins of the full-head oracle (oracle.layer) against independent facts.

Each test compares the oracle with something it does not share code with:
central finite differences of its own forward, torch autograd through torch's
library normalisations (F.normalize, F.rms_norm) over an independent
pair-form core, and invariances of the definitions (scale invariance of the
L2 normalisation and of RMSNorm, the channel gate reducing to the scalar one).
"""

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

from oracle import layer as LY


def _inputs(seed, n, D, Dv, m, scale=1.0):
    rng = np.random.default_rng(seed)
    q, k, r = (rng.standard_normal((n, D)) * scale for _ in range(3))
    v, u = (rng.standard_normal((n, Dv)) for _ in range(2))
    Om = rng.standard_normal((m, D))
    return q, k, v, r, u, Om


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


@pytest.mark.parametrize("channel_gate", [False, True])
def test_head_backward_matches_finite_differences(channel_gate):
    n, D, Dv, m, w = 5, 3, 2, 4, 3
    q, k, v, r, u, Om = _inputs(40, n, D, Dv, m)
    rng = np.random.default_rng(41)
    dy = rng.standard_normal((n, Dv))
    tau = 1.7
    gate = rng.standard_normal((n, Dv)) if channel_gate else -0.4
    dq, dk, dv, dr, du, dtau, dgate = LY.head_backward(q, k, v, r, u, Om, w, tau, gate, dy)

    def loss(xs, t=tau, g=gate):
        y, _ = LY.head_forward(*xs, Om, w, t, g)
        return float(np.sum(dy * y))

    args = [q, k, v, r, u]
    h = 1e-6
    for which, got in enumerate((dq, dk, dv, dr, du)):
        fd = np.zeros_like(args[which])
        for idx in np.ndindex(*args[which].shape):
            xp = [a.copy() for a in args]
            xm = [a.copy() for a in args]
            xp[which][idx] += h
            xm[which][idx] -= h
            fd[idx] = (loss(xp) - loss(xm)) / (2 * h)
        assert _rel(got, fd) < 1e-6, which
    fd_tau = (loss(args, t=tau + h) - loss(args, t=tau - h)) / (2 * h)
    assert abs(dtau - fd_tau) < 1e-6 * (1 + abs(fd_tau))
    if channel_gate:
        fd_g = np.zeros_like(gate)
        for idx in np.ndindex(*gate.shape):
            gp, gm = gate.copy(), gate.copy()
            gp[idx] += h
            gm[idx] -= h
            fd_g[idx] = (loss(args, g=gp) - loss(args, g=gm)) / (2 * h)
        assert _rel(dgate, fd_g) < 1e-6
    else:
        fd_g = (loss(args, g=gate + h) - loss(args, g=gate - h)) / (2 * h)
        assert abs(dgate - fd_g) < 1e-6 * (1 + abs(fd_g))


def _torch_head(q, k, v, r, u, Om, w, tau, gamma, rms_eps):
    """Independent torch head: library normalisations around a pair-form core."""
    qh, kh, rh = (Fn.normalize(x, dim=-1, eps=LY.NORM_EPS) for x in (q, k, r))
    qq = tau * qh
    m = Om.shape[0]

    def feat(x):
        return torch.exp(x @ Om.T - 0.5 * (x * x).sum(-1, keepdim=True)) / math.sqrt(m)

    chi = feat(kh)
    outs = []
    for i in range(q.shape[0]):
        lo = max(0, i - w + 1)
        f = feat(qq[i][None, :] * rh[lo: i + 1])
        kap = f @ chi[: i + 1].T
        num = (kap[:, :, None] * v[None, : i + 1, :] * u[lo: i + 1, None, :]).sum((0, 1))
        outs.append(num / kap.sum())
    ot = torch.stack(outs)
    return torch.sigmoid(gamma) * Fn.rms_norm(ot, (ot.shape[-1],), eps=rms_eps)


def test_head_matches_autograd_of_library_normalisations():
    n, D, Dv, m, w = 12, 4, 3, 6, 4
    q, k, v, r, u, Om = _inputs(42, n, D, Dv, m, scale=2.0)
    dy = np.random.default_rng(43).standard_normal((n, Dv))
    tau, gamma = 2.0, -2.0                        # the paper's initial gamma
    ts = [torch.tensor(x, requires_grad=True) for x in (q, k, v, r, u)]
    tt = torch.tensor(tau, dtype=torch.float64, requires_grad=True)
    tg = torch.tensor(gamma, dtype=torch.float64, requires_grad=True)
    y_t = _torch_head(*ts, torch.tensor(Om), w, tt, tg, LY.RMS_EPS)
    (y_t * torch.tensor(dy)).sum().backward()
    y, _ = LY.head_forward(q, k, v, r, u, Om, w, tau, gamma)
    assert _rel(y, y_t.detach().numpy()) < 1e-12
    grads = LY.head_backward(q, k, v, r, u, Om, w, tau, gamma, dy)
    for g, t in zip(grads[:5], ts):
        assert _rel(g, t.grad.numpy()) < 1e-10
    assert abs(grads[5] - tt.grad.item()) < 1e-10 * (1 + abs(tt.grad.item()))
    assert abs(grads[6] - tg.grad.item()) < 1e-10 * (1 + abs(tg.grad.item()))


def test_head_is_invariant_to_row_scales_of_q_k_r():
    n, D, Dv, m, w = 9, 4, 3, 5, 3
    q, k, v, r, u, Om = _inputs(44, n, D, Dv, m)
    rng = np.random.default_rng(45)
    sq, sk, sr = (rng.uniform(0.1, 10.0, size=(n, 1)) for _ in range(3))
    y0, _ = LY.head_forward(q, k, v, r, u, Om, w, 1.3, 0.5)
    y1, _ = LY.head_forward(q * sq, k * sk, v, r * sr, u, Om, w, 1.3, 0.5)
    assert _rel(y1, y0) < 1e-13


def test_rmsnorm_output_is_scale_free_and_unit_rms():
    n, D, Dv, m, w = 8, 3, 5, 4, 3
    q, k, v, r, u, Om = _inputs(46, n, D, Dv, m)
    gamma = 0.3
    y0, ot = LY.head_forward(q, k, v, r, u, Om, w, 1.0, gamma)
    # y / g has mean square 1 - eps/(ms + eps): unit RMS up to the epsilon
    ms = np.mean(ot * ot, axis=1)
    g = 1 / (1 + math.exp(-gamma))
    assert np.allclose(np.mean((y0 / g) ** 2, axis=1), ms / (ms + LY.RMS_EPS), rtol=1e-12)
    # scaling v by 3 scales o~ by 3 (o~ is linear in v); RMSNorm removes the
    # scale except through the epsilon: y1 = y0 sqrt(ms + e) / sqrt(ms + e/9)
    y1, _ = LY.head_forward(q, k, v * 3.0, r, u, Om, w, 1.0, gamma)
    ratio = np.sqrt(ms + LY.RMS_EPS) / np.sqrt(ms + LY.RMS_EPS / 9.0)
    assert _rel(y1, y0 * ratio[:, None]) < 1e-13


def test_channel_gate_with_constant_logits_is_the_head_gate():
    n, D, Dv, m, w = 7, 3, 4, 5, 2
    q, k, v, r, u, Om = _inputs(47, n, D, Dv, m)
    dy = np.random.default_rng(48).standard_normal((n, Dv))
    y_s, _ = LY.head_forward(q, k, v, r, u, Om, w, 1.5, -1.0)
    y_c, _ = LY.head_forward(q, k, v, r, u, Om, w, 1.5, np.full((n, Dv), -1.0))
    assert _rel(y_c, y_s) < 1e-15
    gs = LY.head_backward(q, k, v, r, u, Om, w, 1.5, -1.0, dy)
    gc = LY.head_backward(q, k, v, r, u, Om, w, 1.5, np.full((n, Dv), -1.0), dy)
    for a, b in zip(gs[:6], gc[:6]):
        assert _rel(a, b) < 1e-15
    assert abs(np.sum(gc[6]) - gs[6]) < 1e-12 * (1 + abs(gs[6]))


def test_zero_rows_take_the_floor_branch():
    n, D, Dv, m, w = 4, 3, 2, 4, 2
    q, k, v, r, u, Om = _inputs(49, n, D, Dv, m)
    q[1] = 0.0
    r[2] = 0.0
    dy = np.random.default_rng(50).standard_normal((n, Dv))
    y, _ = LY.head_forward(q, k, v, r, u, Om, w, 1.0, 0.0)
    assert np.all(np.isfinite(y))
    dq, dk, dv, dr, du, dtau, dg = LY.head_backward(q, k, v, r, u, Om, w, 1.0, 0.0, dy)
    for x in (dq, dk, dv, dr, du):
        assert np.all(np.isfinite(x))
    # below the floor x_hat = x / eps: the gradient is d x_hat / eps, which a
    # central difference that stays below the floor reproduces
    h = 1e-16
    qp, qm = q.copy(), q.copy()
    qp[1, 0] += h
    qm[1, 0] -= h
    lp = float(np.sum(dy * LY.head_forward(qp, k, v, r, u, Om, w, 1.0, 0.0)[0]))
    lm = float(np.sum(dy * LY.head_forward(qm, k, v, r, u, Om, w, 1.0, 0.0)[0]))
    assert abs((lp - lm) / (2 * h) - dq[1, 0]) < 1e-5 * (1 + abs(dq[1, 0]))

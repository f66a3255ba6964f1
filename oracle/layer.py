"""Plain float64 CPU oracle of the full LinSimp head (test infrastructure only).

The core (``oracle.linsimp``) starts at the composite query.  This module adds
the two steps either side of it, as the paper defines the head:

    q_hat = q / |q|,  k_hat = k / |k|,  r_hat = r / |r|        Sec. 3.1
    core inputs: tau * q_hat, k_hat, r_hat, v, u               Sec. 3.1 (per-head temperature on the query)
    o~ = core(tau * q_hat, k_hat, v, r_hat, u)                  Sec. 3.2-3.3
    y  = g * RMSNorm(o~),  g = sigmoid(gamma)                   eq:gated-output (per-head scalar gate)
    y  = g_i (*) RMSNorm(o~_i),  g_i = sigmoid(l_i) in (0,1)^Dv  Sec. 3.3 (channel-wise, input-dependent gate;
                                                                l_i = W_g x_i + b_g is given as an input)

Readings (the paper does not spell these out; each is repeated in the design
notes of the repository):

* L2 normalisation divides by max(|x|, norm_eps), norm_eps = 1e-12 (the
  usual guard for an all-zero row); below the floor the map is x / norm_eps.
* RMSNorm(x) = x / sqrt(mean(x^2) + rms_eps) with rms_eps = 1e-6 and no
  learned scale (eq:gated-output writes g * rmsnorm(o~) with g the only
  learned factor).
* tau and gamma are one float per head.  The channel-wise gate takes the
  projected logits l = W_g x + b_g as an input tensor [n, Dv]; the projection
  itself belongs to the surrounding model.

Gradients are the exact derivatives of these definitions:

    RMSNorm:  o_hat = o~ * rho, rho = (mean(o~^2) + e)^(-1/2)
              d o~  = rho * (d o_hat - o_hat * (d o_hat . o_hat) / Dv)
    gate:     d o_hat = g (*) dy;   dgamma = sum dy (*) o_hat * g (1 - g)
              (channel-wise: dl = dy (*) o_hat (*) g (*) (1 - g))
    L2 norm:  d x = (d x_hat - x_hat (x_hat . d x_hat)) / |x|   (|x| > norm_eps)
              d x = d x_hat / norm_eps                            (otherwise)
    temperature: d x_hat(q) = tau * d(core q);  dtau = sum_i q_hat_i . d(core q)_i

Shapes for one head: q, k, r [n, D]; v, u [n, Dv]; Omega [m, D].
"""

from __future__ import annotations

import numpy as np

from . import linsimp

NORM_EPS = 1e-12
RMS_EPS = 1e-6


def _f64(*xs):
    return [np.asarray(x, dtype=np.float64) for x in xs]


def sigmoid(x):
    x = np.asarray(x, np.float64)
    return 1.0 / (1.0 + np.exp(-x))


def l2_normalize(x, norm_eps=NORM_EPS):
    """Rows of x divided by max(|x|, norm_eps) (Sec. 3.1, x_hat = x / |x|).
    Returns (x_hat, norm) with norm = max(|x|, norm_eps) per row."""
    (x,) = _f64(x)
    nrm = np.maximum(np.sqrt(np.sum(x * x, axis=-1, keepdims=True)), norm_eps)
    return x / nrm, nrm[..., 0]


def rmsnorm(o, rms_eps=RMS_EPS):
    """o / sqrt(mean(o^2) + rms_eps) per row (eq:gated-output).  Returns
    (o_hat, rho) with rho = 1 / sqrt(mean(o^2) + rms_eps)."""
    (o,) = _f64(o)
    rho = 1.0 / np.sqrt(np.mean(o * o, axis=-1, keepdims=True) + rms_eps)
    return o * rho, rho[..., 0]


def gate_values(gate, n, Dv):
    """g as an [n, Dv] array: a scalar gamma (per-head gate, eq:gated-output)
    or logits [n, Dv] (channel-wise gate)."""
    gate = np.asarray(gate, np.float64)
    if gate.ndim == 0:
        return np.full((n, Dv), sigmoid(gate))
    return sigmoid(gate)


def head_forward(q, k, v, r, u, Omega, w, tau, gate, norm_eps=NORM_EPS, rms_eps=RMS_EPS,
                 eps=linsimp.EPS):
    """y of one head: normalise, core, gated RMSNorm.  Returns (y, o_tilde)."""
    q, k, v, r, u, Omega = _f64(q, k, v, r, u, Omega)
    qh, _ = l2_normalize(q, norm_eps)
    kh, _ = l2_normalize(k, norm_eps)
    rh, _ = l2_normalize(r, norm_eps)
    ot = linsimp.forward_recurrent(float(tau) * qh, kh, v, rh, u, Omega, w, eps)
    oh, _ = rmsnorm(ot, rms_eps)
    g = gate_values(gate, *ot.shape)
    return g * oh, ot


def _l2_backward(x, dxh, norm_eps):
    """Gradient through x_hat = x / max(|x|, norm_eps), row by row."""
    nrm = np.sqrt(np.sum(x * x, axis=-1, keepdims=True))
    big = nrm > norm_eps
    xh = x / np.maximum(nrm, norm_eps)
    proj = dxh - xh * np.sum(xh * dxh, axis=-1, keepdims=True)
    return np.where(big, proj / np.maximum(nrm, norm_eps), dxh / norm_eps)


def head_backward(q, k, v, r, u, Omega, w, tau, gate, dy, norm_eps=NORM_EPS, rms_eps=RMS_EPS,
                  eps=linsimp.EPS, parts=None):
    """Exact gradient of sum(dy * y) for one head.

    Returns (dq, dk, dv, dr, du, dtau, dgate): dgate is a float (d gamma) for
    the per-head gate and an [n, Dv] array (d logits) for the channel-wise one.
    If ``parts`` is a dict it receives the two inner products behind dtau and
    dgamma as their factors: q_hat and the core gradient of the scaled query
    (dtau = sum q_hat * dq_core), and dy and o_hat g (1 - g) (dgamma = their sum
    of products).
    """
    q, k, v, r, u, Omega, dy = _f64(q, k, v, r, u, Omega, dy)
    qh, _ = l2_normalize(q, norm_eps)
    kh, _ = l2_normalize(k, norm_eps)
    rh, _ = l2_normalize(r, norm_eps)
    tau = float(tau)
    ot = linsimp.forward_recurrent(tau * qh, kh, v, rh, u, Omega, w, eps)
    oh, rho = rmsnorm(ot, rms_eps)
    n, Dv = ot.shape
    g = gate_values(gate, n, Dv)
    # gate and RMSNorm
    dgl = dy * oh * g * (1.0 - g)
    dgate = float(np.sum(dgl)) if np.ndim(gate) == 0 else dgl
    doh = g * dy
    dot = rho[:, None] * (doh - oh * np.sum(doh * oh, axis=-1, keepdims=True) / Dv)
    # core
    dqc, dkh, dv, drh, du = linsimp.backward(tau * qh, kh, v, rh, u, Omega, w, dot, eps)
    # temperature and L2 normalisation
    dtau = float(np.sum(qh * dqc))
    if parts is not None:
        parts.update(q_hat=qh, dq_core=dqc, dy=dy, gate_factor=oh * g * (1.0 - g))
    dq = _l2_backward(q, tau * dqc, norm_eps)
    dk = _l2_backward(k, dkh, norm_eps)
    dr = _l2_backward(r, drh, norm_eps)
    return dq, dk, dv, dr, du, dtau, dgate

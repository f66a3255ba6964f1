"""Planted mistakes in the oracle, on the CPU.

Each plausible slip in a building block of the oracle, or in the order of its
recurrence, must be caught by a reference that shares none of the oracle's
code: the pure-Python brute force of oracle.brute (the definition written as
loops), the closed form of row 0 (one pair: out_0 = v_0 (*) u_0) and the
joint normaliser (v = u = 1 gives out = 1).  The unmodified oracle passes the
same checks.  This shows that the pins have teeth; it is not a test of the
GPU path.
"""

import numpy as np
import pytest

from oracle import brute
from oracle import linsimp as O


def _inputs(seed, n=6, D=3, Dv=2, m=3):
    rng = np.random.default_rng(seed)
    f = lambda *s: 0.5 * rng.standard_normal(s)   # noqa: E731
    return f(n, D), f(n, D), f(n, Dv), f(n, D), f(n, Dv), rng.standard_normal((m, D))


def _failed_checks(fwd):
    """Names of the independent checks that `fwd` (same signature as
    O.forward_recurrent) fails."""
    failed = []
    q, k, v, r, u, Om = _inputs(5)
    w = 3
    got = fwd(q, k, v, r, u, Om, w)
    ref = np.array(brute.output(q.tolist(), k.tolist(), v.tolist(), r.tolist(), u.tolist(), Om.tolist(), w))
    if not np.allclose(got, ref, rtol=1e-10, atol=1e-12):
        failed.append("brute force")
    if not np.allclose(got[0], v[0] * u[0], rtol=1e-12, atol=1e-14):
        failed.append("row 0")
    ones = fwd(q, k, np.ones_like(v), r, np.ones_like(u), Om, w)
    if not np.allclose(ones, 1.0, rtol=1e-12):
        failed.append("joint normaliser")
    return failed


def test_unmodified_oracle_passes_the_checks():
    assert _failed_checks(O.forward_recurrent) == []
    assert _failed_checks(O.forward_pair) == []
    assert _failed_checks(lambda *a: O.forward_chunked(*a, chunk=2, feature_block=2)) == []
    assert _failed_checks(lambda *a: O.forward_logspace(*a)[0]) == []


def _phi_no_norm_term(X, Omega):
    X, Omega = np.asarray(X, float), np.asarray(Omega, float)
    return np.exp(X @ Omega.T) / np.sqrt(Omega.shape[0])


def _phi_plus_norm_term(X, Omega):
    X, Omega = np.asarray(X, float), np.asarray(Omega, float)
    return np.exp(X @ Omega.T + 0.5 * np.sum(X * X, axis=-1, keepdims=True)) / np.sqrt(Omega.shape[0])


def _phi_omega_transposed(X, Omega):
    X, Omega = np.asarray(X, float), np.asarray(Omega, float)
    return np.exp(X @ Omega - 0.5 * np.sum(X * X, axis=-1, keepdims=True)) / np.sqrt(Omega.shape[0])


# building-block mutations: (module attribute, replacement)
BLOCK_MUTANTS = {
    "feature map without the -|x|^2/2 term": ("phi", _phi_no_norm_term),
    "feature map with +|x|^2/2": ("phi", _phi_plus_norm_term),
    "feature map with Omega transposed": ("phi", _phi_omega_transposed),
    "window one anchor too wide": ("anchor_window", lambda i, w: np.arange(max(0, i - w), i + 1)),
    "window without the anchor c = i": ("anchor_window", lambda i, w: np.arange(max(0, i - w), i)),
    "window one anchor too narrow": ("anchor_window", lambda i, w: np.arange(max(0, i - w + 2), i + 1)),
    "composite query q + r": ("composite_query", lambda q_i, r_C: np.asarray(q_i)[None, :] + np.asarray(r_C)),
    "composite query without the anchor": ("composite_query", lambda q_i, r_C: np.repeat(np.asarray(q_i)[None, :], len(r_C), 0)),
}


@pytest.mark.parametrize("name", list(BLOCK_MUTANTS))
def test_planted_building_block_mistake_is_caught(name, monkeypatch):
    attr, fake = BLOCK_MUTANTS[name]
    monkeypatch.setattr(O, attr, fake)
    assert _failed_checks(O.forward_recurrent), name
    assert _failed_checks(O.forward_pair), name


def _recurrent_variant(q, k, v, r, u, Omega, w, *, update_after=False, per_anchor=False, drop_u=False):
    """The recurrent form with one structural slip switched on."""
    n, Dv = v.shape
    m = Omega.shape[0]
    M, a = np.zeros((m, Dv)), np.zeros(m)
    out = np.zeros((n, Dv))
    for i in range(n):
        chi = O.phi(k[i], Omega)
        if not update_after:
            M += np.outer(chi, v[i])
            a += chi
        C = O.anchor_window(i, w)
        F = O.phi(O.composite_query(q[i], r[C]), Omega)
        NA = F @ M                                   # [|C|, Dv]
        if not drop_u:
            NA = NA * u[C]
        if per_anchor:
            out[i] = np.sum(NA / (F @ a + 1e-30)[:, None], axis=0)
        else:
            out[i] = NA.sum(axis=0) / (np.sum(F @ a) + 1e-30)
        if update_after:
            M += np.outer(chi, v[i])
            a += chi
    return out


STRUCTURAL_MUTANTS = {
    "state updated after the readout (j < i)": dict(update_after=True),
    "one normaliser per anchor instead of the joint one": dict(per_anchor=True),
    "anchor values u left out": dict(drop_u=True),
}


@pytest.mark.parametrize("name", list(STRUCTURAL_MUTANTS))
def test_planted_structural_mistake_is_caught(name):
    kw = STRUCTURAL_MUTANTS[name]
    assert _failed_checks(lambda *a: _recurrent_variant(*a)) == []      # the switch-off copy is right
    assert _failed_checks(lambda *a: _recurrent_variant(*a, **kw)), name


def _fd_failures(grads_fn):
    """Central finite differences of the recurrent form (the definition) at a
    few coordinates of every input against `grads_fn`'s analytic gradient."""
    q, k, v, r, u, Om = _inputs(9, n=5)
    w = 3
    dO = np.random.default_rng(10).standard_normal(v.shape)
    grads = grads_fn(q, k, v, r, u, Om, w, dO)
    xs = [q, k, v, r, u]
    failed = []
    h = 1e-6
    for gi, (x, g) in enumerate(zip(xs, grads)):
        for (a, b) in ((0, 0), (2, 1), (4, 0)):
            xp, xm = [t.copy() for t in xs], [t.copy() for t in xs]
            xp[gi][a, b] += h
            xm[gi][a, b] -= h
            fd = (np.sum(dO * O.forward_recurrent(*xp, Om, w)) - np.sum(dO * O.forward_recurrent(*xm, Om, w))) / (2 * h)
            if abs(fd - g[a, b]) > 1e-6 * max(1.0, abs(fd)):
                failed.append((gi, a, b))
    return failed


def test_backward_slips_are_caught_by_finite_differences():
    assert _fd_failures(O.backward) == []
    swapped = lambda *a: (lambda g: (g[3], g[1], g[2], g[0], g[4]))(O.backward(*a))   # noqa: E731  dq <-> dr
    assert _fd_failures(swapped)
    halved_du = lambda *a: (lambda g: (*g[:4], 0.5 * g[4]))(O.backward(*a))          # noqa: E731
    assert _fd_failures(halved_du)


# ---- the full head (oracle.layer) ----

def _head_reference_failures(head_forward):
    """Compare a head forward against torch's library normalisations around an
    independent pair-form core (the pin of tests/test_oracle_layer.py)."""
    import torch
    from test_oracle_layer import _inputs as head_inputs, _torch_head
    from oracle import layer as LY
    n, D, Dv, m, w = 9, 4, 3, 6, 4
    q, k, v, r, u, Om = head_inputs(42, n, D, Dv, m, scale=2.0)
    tau, gamma = 2.0, -2.0
    ref = _torch_head(*(torch.tensor(x) for x in (q, k, v, r, u)), torch.tensor(Om), w,
                      torch.tensor(tau, dtype=torch.float64), torch.tensor(gamma, dtype=torch.float64),
                      LY.RMS_EPS).numpy()
    y, _ = head_forward(q, k, v, r, u, Om, w, tau, gamma)
    return not np.allclose(y, ref, rtol=1e-10, atol=1e-12)


HEAD_MUTANTS = {
    "temperature on the key instead of the query": "tau_on_k",
    "RMSNorm over mean |x| instead of mean x^2": "rms_abs",
    "gate sigmoid(-gamma)": "gate_sign",
    "r left unnormalised": "no_r_norm",
}


def _mutant_head(kind):
    from oracle import layer as LY

    def head_forward(q, k, v, r, u, Omega, w, tau, gate, **kw):
        qh, _ = LY.l2_normalize(q)
        kh, _ = LY.l2_normalize(k)
        rh = np.asarray(r, float) if kind == "no_r_norm" else LY.l2_normalize(r)[0]
        qs, ks = (qh, tau * kh) if kind == "tau_on_k" else (tau * qh, kh)
        ot = O.forward_recurrent(qs, ks, v, rh, u, Omega, w)
        if kind == "rms_abs":
            oh = ot / np.sqrt(np.mean(np.abs(ot), axis=-1, keepdims=True) + LY.RMS_EPS)
        else:
            oh, _ = LY.rmsnorm(ot)
        g = LY.gate_values(-gate if kind == "gate_sign" else gate, *ot.shape)
        return g * oh, ot
    return head_forward


def test_head_reference_accepts_the_oracle_and_catches_planted_slips():
    from oracle import layer as LY
    assert not _head_reference_failures(LY.head_forward)
    for name, kind in HEAD_MUTANTS.items():
        assert _head_reference_failures(_mutant_head(kind)), name

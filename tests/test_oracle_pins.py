"""Pins of the CPU oracle against facts the paper and the mathematics fix.

None of these re-types the oracle's own formula: each compares it with an
independent computation (pure-Python brute force, a closed form, a library
routine, an invariant that a plausible mistake would break).
"""

import math

import numpy as np
import pytest
import torch

from oracle import brute, features, montecarlo
from oracle import linsimp as O


def _inputs(seed, n, D, Dv, m, scale=None):
    rng = np.random.default_rng(seed)
    s = D ** -0.25 if scale is None else scale
    q, k, r = (rng.standard_normal((n, D)) * s for _ in range(3))
    v, u = (rng.standard_normal((n, Dv)) * s for _ in range(2))
    Om = rng.standard_normal((m, D))
    return q, k, v, r, u, Om


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


# --------------------------------------------------------------------------
# North-star check 1: the score rewrite (Sec. 3.1 eq:two-views)
# --------------------------------------------------------------------------

def test_score_rewrite_matches_triple_sum():
    q, k, _, r, _, _ = _inputs(1, 6, 5, 2, 3)
    s = O.trilinear_score(q, k, r)
    ql, kl, rl = q.tolist(), k.tolist(), r.tolist()
    for i in range(6):
        for j in range(6):
            for c in range(6):
                ref = brute.score(ql, kl, rl, i, j, c)
                assert abs(s[i, j, c] - ref) <= 1e-13 * (1 + abs(ref))
                # the other orientation of eq:two-views
                alt = float(np.dot(q[i] * k[j], r[c]))
                assert abs(alt - ref) <= 1e-13 * (1 + abs(ref))


# --------------------------------------------------------------------------
# North-star checks 2 and 3: recurrent = parallel, brute force on tiny n
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed,n,D,Dv,m,w", [(2, 7, 3, 2, 5, 3), (3, 8, 4, 3, 8, 4),
                                              (4, 5, 2, 2, 3, 1), (5, 6, 3, 1, 4, 8)])
def test_brute_force_tiny(seed, n, D, Dv, m, w):
    q, k, v, r, u, Om = _inputs(seed, n, D, Dv, m, scale=0.7)
    ref = np.array(brute.output(q.tolist(), k.tolist(), v.tolist(), r.tolist(),
                                u.tolist(), Om.tolist(), w))
    assert _rel(O.forward_pair(q, k, v, r, u, Om, w), ref) < 1e-12
    assert _rel(O.forward_recurrent(q, k, v, r, u, Om, w), ref) < 1e-12
    assert _rel(O.forward_logspace(q, k, v, r, u, Om, w)[0], ref) < 1e-12
    assert _rel(O.forward_chunked(q, k, v, r, u, Om, w, chunk=3, feature_block=2), ref) < 1e-12


def test_recurrent_equals_parallel_and_chunked():
    q, k, v, r, u, Om = _inputs(6, 77, 8, 6, 16)
    w = 5
    rec = O.forward_recurrent(q, k, v, r, u, Om, w)
    assert _rel(O.forward_pair(q, k, v, r, u, Om, w), rec) < 1e-12
    # several chunk sizes, a ragged tail (77 = 4*16 + 13) and feature blocks
    for ch, fb in ((16, 4), (32, 16), (7, 5)):
        assert _rel(O.forward_chunked(q, k, v, r, u, Om, w, chunk=ch, feature_block=fb), rec) < 1e-12


# --------------------------------------------------------------------------
# North-star check 4: Monte-Carlo convergence (Lemma 1 and its variance)
# --------------------------------------------------------------------------

def test_lemma1_unbiased_mean():
    rng = np.random.default_rng(7)
    x = np.array([0.3, -0.2, 0.5, 0.1])
    y = np.array([-0.4, 0.25, 0.35, -0.3])
    m = 400_000
    Om = rng.standard_normal((m, 4))
    est = montecarlo.kernel_estimate(x, y, Om)
    sigma = math.sqrt(montecarlo.estimate_variance(x, y, m))
    assert abs(est - math.exp(x @ y)) < 5 * sigma
    # a feature map without the |x|^2/2 correction would be off by e^{(|x|^2+|y|^2)/2}
    assert abs(math.exp(x @ y) * math.exp(0.5 * (x @ x + y @ y)) - est) > 50 * sigma


def test_lemma1_closed_form_variance():
    rng = np.random.default_rng(8)
    x = np.array([0.2, -0.1, 0.3])
    y = np.array([0.1, 0.2, -0.25])
    m, trials = 8, 20_000
    ests = np.array([montecarlo.kernel_estimate(x, y, rng.standard_normal((m, 3)))
                     for _ in range(trials)])
    var_cf = montecarlo.estimate_variance(x, y, m)
    assert abs(ests.mean() - math.exp(x @ y)) < 5 * math.sqrt(var_cf / trials)
    assert abs(ests.var() / var_cf - 1.0) < 0.05


def test_output_converges_to_exact_window_kernel():
    """As m grows the estimator tends to o^(w) (App. A eq:exact-window-app);
    the error falls roughly like m^{-1/2} (the ratio is biased at finite m)."""
    # small input norms keep the log-normal feature products light-tailed, so
    # the Monte-Carlo error is in its m^{-1/2} regime already at m = 64
    q, k, v, r, u, _ = _inputs(9, 12, 4, 3, 1, scale=0.35)
    w = 4
    exact = O.exact_window(q, k, v, r, u, w)
    # the exact operator itself against pure-Python brute force
    bref = np.array(brute.exact_output(q.tolist(), k.tolist(), v.tolist(), r.tolist(),
                                       u.tolist(), w))
    assert _rel(exact, bref) < 1e-12
    errs = []
    for m in (64, 4096, 262_144):
        e = []
        for s in range(4):
            Om = np.random.default_rng(100 + s).standard_normal((m, 4))
            e.append(_rel(O.forward_recurrent(q, k, v, r, u, Om, w), exact))
        errs.append(np.mean(e))
    assert errs[0] > errs[1] > errs[2]
    slopes = np.diff(np.log(errs)) / np.log(64.0)      # m grows 64x per step
    assert np.all(np.abs(slopes + 0.5) < 0.15), slopes
    assert errs[2] < 2e-3


# --------------------------------------------------------------------------
# Special cases with closed forms
# --------------------------------------------------------------------------

def test_row0_is_v0_times_u0():
    for seed, m in ((10, 3), (11, 64)):
        q, k, v, r, u, Om = _inputs(seed, 5, 6, 4, m)
        o = O.forward_recurrent(q, k, v, r, u, Om, 3)
        assert np.allclose(o[0], v[0] * u[0], rtol=1e-13, atol=0)


def test_normalisation_is_joint():
    q, k, v, r, u, Om = _inputs(12, 40, 6, 5, 12)
    ones = np.ones_like(v)
    o = O.forward_recurrent(q, k, ones, r, ones, Om, 7)
    assert np.allclose(o, 1.0, rtol=1e-13, atol=0)
    # every output coordinate lies in the hull of the pair values v_j (*) u_c
    w = 7
    o = O.forward_recurrent(q, k, v, r, u, Om, w)
    for i in range(40):
        C = O.anchor_window(i, w)
        vals = (v[: i + 1][None, :, :] * u[C][:, None, :]).reshape(-1, v.shape[1])
        assert np.all(o[i] <= vals.max(0) + 1e-12) and np.all(o[i] >= vals.min(0) - 1e-12)


def test_unit_anchors_reduce_to_softmax_attention_as_m_grows():
    """r = 1, u = 1: every anchor sends the same query, so the layer is causal
    positive-random-feature linear attention (Performer), independent of w, and
    tends to causal softmax attention with scale 1 as m grows (Lemma 1)."""
    q, k, v, _, _, _ = _inputs(13, 10, 4, 3, 1, scale=0.5)
    ones_r = np.ones_like(q)
    ones_u = np.ones_like(v)
    Om = np.random.default_rng(14).standard_normal((200_000, 4))
    o3 = O.forward_recurrent(q, k, v, ones_r, ones_u, Om, 3)
    o9 = O.forward_recurrent(q, k, v, ones_r, ones_u, Om, 9)
    assert _rel(o3, o9) < 1e-13
    sdpa = torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(q)[None, None], torch.tensor(k)[None, None], torch.tensor(v)[None, None],
        is_causal=True, scale=1.0)[0, 0].numpy()
    assert _rel(o3, sdpa) < 1e-2


def test_window_one_factorises_u():
    """w = 1: o~_i = u_i (*) LinAttn(q_i (*) r_i; k; v)."""
    q, k, v, r, u, Om = _inputs(15, 30, 5, 4, 16)
    o = O.forward_recurrent(q, k, v, r, u, Om, 1)
    lin = O.forward_recurrent(q * r, k, v, np.ones_like(r), np.ones_like(u), Om, 1)
    assert _rel(o, u * lin) < 1e-13


def test_window_at_least_n_is_global_anchor_form():
    """w >= n: every c <= i is an anchor (App. E item 2, one global orientation)."""
    q, k, v, r, u, Om = _inputs(16, 9, 3, 2, 6, scale=0.8)
    n = 9
    ref = np.zeros((n, 2))
    chi = O.phi(k, Om)
    for i in range(n):                   # direct global sum, written independently
        num, den = np.zeros(2), 0.0
        for c in range(i + 1):
            f = O.phi(q[i] * r[c], Om)
            for j in range(i + 1):
                kap = f @ chi[j]
                num += kap * v[j] * u[c]
                den += kap
        ref[i] = num / den
    assert _rel(O.forward_recurrent(q, k, v, r, u, Om, n), ref) < 1e-12
    assert _rel(O.forward_recurrent(q, k, v, r, u, Om, 5 * n), ref) < 1e-12


# --------------------------------------------------------------------------
# Invariances
# --------------------------------------------------------------------------

def test_logspace_form_matches_and_survives_underflow():
    q, k, v, r, u, Om = _inputs(17, 50, 8, 4, 16)
    o_ls, L, R, Zh = O.forward_logspace(q, k, v, r, u, Om, 6)
    assert _rel(o_ls, O.forward_recurrent(q, k, v, r, u, Om, 6)) < 1e-12
    assert np.all(np.diff(R) >= 0)        # the key shift is a running maximum
    # keys so large that every fp64 feature underflows without the shift
    kb = k * 60.0
    o_ls = O.forward_logspace(q, kb, v, r, u, Om, 6)[0]
    assert np.allclose(o_ls[0], v[0] * u[0], rtol=1e-12, atol=0)
    assert np.all(np.isfinite(o_ls))


def test_causality_bitwise():
    q, k, v, r, u, Om = _inputs(18, 40, 6, 4, 8)
    base = O.forward_recurrent(q, k, v, r, u, Om, 5)
    t = 23
    rng = np.random.default_rng(19)
    q2, k2, v2, r2, u2 = (x.copy() for x in (q, k, v, r, u))
    for x in (q2, k2, v2, r2, u2):
        x[t + 1:] = rng.standard_normal(x[t + 1:].shape) * 3
    pert = O.forward_recurrent(q2, k2, v2, r2, u2, Om, 5)
    assert np.array_equal(base[: t + 1], pert[: t + 1])
    assert not np.allclose(base[t + 1:], pert[t + 1:])


def test_feature_bank_row_permutation_and_duplication():
    q, k, v, r, u, Om = _inputs(20, 30, 5, 3, 10)
    base = O.forward_recurrent(q, k, v, r, u, Om, 4)
    perm = np.random.default_rng(21).permutation(10)
    assert _rel(O.forward_recurrent(q, k, v, r, u, Om[perm], 4), base) < 1e-13
    # duplicating every row halves each feature squared: the kernel is unchanged
    dup = np.concatenate([Om, Om])
    assert _rel(O.forward_recurrent(q, k, v, r, u, dup, 4), base) < 1e-13


# --------------------------------------------------------------------------
# Gradients: finite differences and autograd of an independent pair form
# --------------------------------------------------------------------------

def test_backward_matches_finite_differences():
    n, D, Dv, m, w = 6, 3, 2, 4, 3
    q, k, v, r, u, Om = _inputs(22, n, D, Dv, m, scale=0.8)
    dO = np.random.default_rng(23).standard_normal((n, Dv))
    grads = O.backward(q, k, v, r, u, Om, w, dO)
    args = [q, k, v, r, u]

    def loss(xs):
        return float(np.sum(dO * O.forward_recurrent(*xs, Om, w)))

    h = 1e-6
    for which in range(5):
        fd = np.zeros_like(args[which])
        for idx in np.ndindex(*args[which].shape):
            xp = [a.copy() for a in args]
            xm = [a.copy() for a in args]
            xp[which][idx] += h
            xm[which][idx] -= h
            fd[idx] = (loss(xp) - loss(xm)) / (2 * h)
        assert _rel(grads[which], fd) < 1e-7, which


def _torch_pair_form(q, k, v, r, u, Om, w):
    """An independent pair-form forward in torch (fp64), for autograd."""
    n = q.shape[0]
    m = Om.shape[0]

    def feat(x):
        return torch.exp(x @ Om.T - 0.5 * (x * x).sum(-1, keepdim=True)) / math.sqrt(m)

    outs = []
    chi = feat(k)
    for i in range(n):
        lo = max(0, i - w + 1)
        f = feat(q[i][None, :] * r[lo: i + 1])            # [c, m]
        kap = f @ chi[: i + 1].T                          # [c, j]
        num = (kap[:, :, None] * v[None, : i + 1, :] * u[lo: i + 1, None, :]).sum((0, 1))
        outs.append(num / kap.sum())
    return torch.stack(outs)


def test_backward_matches_autograd_of_pair_form():
    n, D, Dv, m, w = 20, 4, 3, 8, 5
    q, k, v, r, u, Om = _inputs(24, n, D, Dv, m)
    dO = np.random.default_rng(25).standard_normal((n, Dv))
    ts = [torch.tensor(x, requires_grad=True) for x in (q, k, v, r, u)]
    out = _torch_pair_form(*ts, torch.tensor(Om), w)
    (out * torch.tensor(dO)).sum().backward()
    grads = O.backward(q, k, v, r, u, Om, w, dO)
    for g, t in zip(grads, ts):
        assert _rel(g, t.grad.numpy()) < 1e-10


# --------------------------------------------------------------------------
# Decode (Theorem 1)
# --------------------------------------------------------------------------

def test_decode_matches_forward_rows_and_resumes():
    n, D, Dv, m, w = 30, 5, 4, 8, 6
    q, k, v, r, u, Om = _inputs(26, n, D, Dv, m)
    full = O.forward_recurrent(q, k, v, r, u, Om, w)
    P = 4
    st = O.prefill_state(k[:P], v[:P], r[:P], u[:P], Om, w)
    saved = None
    for t in range(P, n):                    # runs several times round the ring
        o, st = O.decode_step(st, q[t], k[t], v[t], r[t], u[t], Om, w)
        assert _rel(o, full[t]) < 1e-12
        if t == 17:
            saved = {kk: (vv.copy() if isinstance(vv, np.ndarray) else vv) for kk, vv in st.items()}
    # resume from a saved state
    st2 = saved
    for t in range(18, n):
        o, st2 = O.decode_step(st2, q[t], k[t], v[t], r[t], u[t], Om, w)
        assert _rel(o, full[t]) < 1e-12
    # prefill of the whole prefix equals the stepped state
    ref = O.prefill_state(k, v, r, u, Om, w)
    assert _rel(st["M"], ref["M"]) < 1e-12 and _rel(st["a"], ref["a"]) < 1e-12
    assert np.array_equal(st["ring_r"], ref["ring_r"])


# --------------------------------------------------------------------------
# Orthogonal random-feature bank (App. B.1)
# --------------------------------------------------------------------------

def test_orthogonal_bank_structure_and_sign_fix():
    rng = np.random.default_rng(27)
    D = 6
    Om = features.orthogonal_bank(rng, 2 * D, D)
    for blk in (Om[:D], Om[D:]):
        dirs = blk / np.linalg.norm(blk, axis=1, keepdims=True)
        assert np.allclose(dirs @ dirs.T, np.eye(D), atol=1e-12)
    # Haar factor: with the sign fix the first direction's first coordinate is
    # symmetric about 0; without it (Householder QR) it always has one sign.
    s_fix = [np.sign(features.orthogonal_bank(rng, D, D)[0, 0]) for _ in range(400)]
    s_raw = [np.sign(features.orthogonal_bank(rng, D, D, sign_correct=False)[0, 0])
             for _ in range(400)]
    assert abs(np.mean(s_fix)) < 0.2
    assert abs(np.mean(s_raw)) > 0.9
    # marginal rows are N(0, I): Lemma 1 holds with this bank too
    x = np.array([0.3, -0.1, 0.2, 0.0, 0.1, -0.2])
    y = np.array([0.1, 0.2, -0.3, 0.25, 0.0, 0.1])
    Om = features.orthogonal_bank(rng, 120_000, D)
    est = montecarlo.kernel_estimate(x, y, Om)
    assert abs(est / math.exp(x @ y) - 1) < 5e-3


def test_orthogonal_block_reconstructs_and_has_positive_diagonal():
    rng = np.random.default_rng(70)
    D = 16
    G = rng.standard_normal((D, D))
    radii = np.sqrt(rng.chisquare(D, size=D))
    Om = features.orthogonal_block(G, radii)
    # row norms are the radii; directions are orthonormal
    assert np.allclose(np.linalg.norm(Om, axis=1), radii, rtol=1e-13)
    Qt = Om / radii[:, None]
    assert np.allclose(Qt @ Qt.T, np.eye(D), atol=1e-13)
    # Q^T G is upper triangular with a positive diagonal (the sign-fixed R):
    # a Gram-Schmidt of G's columns, computed independently, gives the same Q
    R = Qt @ G
    assert np.allclose(np.tril(R, -1), 0, atol=1e-12)
    assert np.all(np.diag(R) > 0)
    Qgs = np.zeros((D, D))
    for a in range(D):
        x = G[:, a].copy()
        for b in range(a):
            x -= (Qgs[:, b] @ G[:, a]) * Qgs[:, b]
        for b in range(a):                       # second pass (re-orthogonalise)
            x -= (Qgs[:, b] @ x) * Qgs[:, b]
        Qgs[:, a] = x / np.linalg.norm(x)
    assert np.allclose(Qgs.T, Qt, atol=1e-11)
    # without the fix the factor is Householder's: first column of Q is
    # -sign(G[0,0]) G[:,0] / |G[:,0]| (R_00 = -sign(G_00)|G_:0|)
    raw = features.orthogonal_block(G, np.ones(D), sign_correct=False)
    assert np.allclose(raw[0], -np.sign(G[0, 0]) * G[:, 0] / np.linalg.norm(G[:, 0]), atol=1e-13)


def test_orthogonal_bank_from_stacks_blocks_in_order_and_truncates():
    """orthogonal_bank_from (the reference of the device sampler): block b
    comes from draw b and nothing else, blocks are stacked in draw order and
    the last one is cut at m rows.  Pinned by properties of App. B.1's
    construction, not by re-calling it: the rows of block b, divided by
    radii[b], are orthonormal and Q_b^T G_b is upper triangular with a
    positive diagonal (the sign-fixed R of G_b = Q_b R_b); a truncated block
    keeps the leading rows, so those rows of Q^T G stay zero left of the
    diagonal."""
    rng = np.random.default_rng(72)
    D, nb = 8, 3
    G = rng.standard_normal((nb, D, D))
    radii = np.sqrt(rng.chisquare(D, size=(nb, D)))
    for m in (nb * D, nb * D - 3, D + 1, 5):
        Om = features.orthogonal_bank_from(G, radii, m)
        assert Om.shape == (m, D)
        for b in range(-(-m // D)):
            rows = Om[b * D: min(m, (b + 1) * D)]
            k = rows.shape[0]
            assert np.allclose(np.linalg.norm(rows, axis=1), radii[b, :k], rtol=1e-13)
            Qt = rows / radii[b, :k, None]
            assert np.allclose(Qt @ Qt.T, np.eye(k), atol=1e-13)
            R = Qt @ G[b]                     # the leading k rows of R_b
            assert np.allclose(np.tril(R, -1), 0, atol=1e-12)
            assert np.all(np.diag(R[:, :k]) > 0)
            if k >= 2:                        # draw b is the one that fits, not another's
                other = Qt @ G[(b + 1) % nb]
                assert not np.allclose(np.tril(other, -1), 0, atol=1e-6)
    # the same draws replayed through the sampler give the same bank
    m, D2 = 20, 6
    r1 = np.random.default_rng(73)
    Gs, Rs = [], []
    for _ in range(-(-m // D2)):
        Gs.append(r1.standard_normal((D2, D2)))
        Rs.append(np.sqrt(r1.chisquare(D2, size=D2)))
    assert np.array_equal(features.orthogonal_bank_from(np.stack(Gs), np.stack(Rs), m),
                          features.orthogonal_bank(np.random.default_rng(73), m, D2))
    # without the sign fix each block is Householder's factor of its own draw
    raw = features.orthogonal_bank_from(G, np.ones((nb, D)), 2 * D, sign_correct=False)
    for b in range(2):
        g0 = G[b][:, 0]
        assert np.allclose(raw[b * D], -np.sign(g0[0]) * g0 / np.linalg.norm(g0), atol=1e-13)


def _kernel_error(rng, m, D, sign_correct, pairs):
    """RMS relative error of the kernel estimate of Lemma 1 over fixed pairs,
    one bank of m rows."""
    Om = features.orthogonal_bank(rng, m, D, sign_correct)
    errs = []
    for x, y in pairs:
        est = montecarlo.kernel_estimate(x, y, Om)
        errs.append(est / montecarlo.exact_kernel(x, y) - 1.0)
    return float(np.sqrt(np.mean(np.square(errs))))


def test_sign_fix_gives_the_inverse_sqrt_m_trend():
    """App. B.1 diagnostic: with the sign correction the kernel error falls like
    m^{-1/2}; without it (Householder factor) it stays at a bias floor."""
    D = 16
    prng = np.random.default_rng(71)
    pairs = []
    for _ in range(16):
        x, y = prng.standard_normal(D), prng.standard_normal(D)
        pairs.append((0.5 * x / np.linalg.norm(x), 0.5 * y / np.linalg.norm(y)))
    ms = [256, 4096, 65536]
    fixed = [np.mean([_kernel_error(np.random.default_rng(100 + 7 * s + i), m, D, True, pairs)
                      for s in range(4)]) for i, m in enumerate(ms)]
    raw = [np.mean([_kernel_error(np.random.default_rng(200 + 7 * s + i), m, D, False, pairs)
                    for s in range(4)]) for i, m in enumerate(ms)]
    slope = np.polyfit(np.log(ms), np.log(fixed), 1)[0]
    assert -0.65 < slope < -0.35, (slope, fixed)
    # the raw factor's error does not keep falling: it is far above the fixed
    # one at large m and drops by much less than 16x over a 256x range
    assert raw[-1] > 4 * fixed[-1], (raw, fixed)
    assert raw[0] / raw[-1] < 4, raw


def test_backward_dk_term_scale_bounds_relative_perturbations():
    """oracle.linsimp.backward's term_scale (the per-key scale of dk's summed
    terms taken in absolute value) leaves the gradients unchanged, is at
    least |dk_j|, and bounds the first-order change of dk_j when every query
    feature phi(z_ic)_p entering the state gradient is scaled by (1 + delta)
    with |delta| <= u (what a rounding of those features does)."""
    rng = np.random.default_rng(91)
    n, D, Dv, m, w = 30, 6, 5, 12, 7
    q, k, v, r, u, Om = _inputs(92, n, D, Dv, m)
    dO = rng.standard_normal((n, Dv))
    plain = O.backward(q, k, v, r, u, Om, w, dO)
    ts = {}
    g = O.backward(q, k, v, r, u, Om, w, dO, term_scale=ts)
    assert all(np.array_equal(a, b) for a, b in zip(plain, g))
    T = ts["dk"]
    assert np.all(T >= np.linalg.norm(g[1], axis=1) * (1 - 1e-12))
    # perturbed state gradient: dM_i = sum_c F_ic (1 + delta) dA_ic, da_i likewise
    uu = 1e-6
    chi = O.phi(k, Om)
    worst = 0.0
    for trial in range(3):
        G, h = np.zeros((m, Dv)), np.zeros(m)
        M, a = chi.T @ v, chi.sum(axis=0)
        dk = np.zeros_like(k)
        for i in range(n - 1, -1, -1):
            C = O.anchor_window(i, w)
            F = O.phi(O.composite_query(q[i], r[C]), Om)
            Z = np.sum(F @ a)
            o = np.sum((F @ M) * u[C], axis=0) / Z
            dN, dZ = dO[i] / Z, -np.dot(dO[i], o) / Z
            Fp = F * (1 + uu * rng.uniform(-1, 1, F.shape))
            G += Fp.T @ (dN[None, :] * u[C])
            h += dZ * Fp.sum(axis=0)
            dlam = (G @ v[i] + h) * chi[i]
            dk[i] = dlam @ Om - dlam.sum() * k[i]
            M, a = M - np.outer(chi[i], v[i]), a - chi[i]
        worst = max(worst, float(np.max(np.linalg.norm(dk - g[1], axis=1) / (uu * T))))
    assert worst <= 1.0 + 1e-6, worst
    assert worst > 1e-3, worst          # the bound is not vacuous

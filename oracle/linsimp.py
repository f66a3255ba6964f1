"""Plain float64 CPU oracle of the LinSimp layer core (test infrastructure only).

What is computed, for one head, with 0-based positions i = 0 .. n-1
(the paper counts from 1):

    phi(x)  = m^{-1/2} exp(Omega x - |x|^2/2 * 1)             Sec. 3.2, eq:prf
    z_ic    = q_i (*) r_c                                       Sec. 3.2 (composite query)
    M_i     = sum_{j<=i} phi(k_j) v_j^T ,  a_i = sum_{j<=i} phi(k_j)   eq:Mstate, eq:astate
    C_i     = {max(0, i-w+1), ..., i}                           Sec. 3.3 (anchor window)
    N_i     = sum_{c in C_i} [phi(z_ic)^T M_i] (*) u_c          eq:Ni
    Z_i     = sum_{c in C_i}  phi(z_ic)^T a_i                   eq:Zi
    o~_i    = N_i / (Z_i + eps),  eps = 1e-30                   eq:linearized-output

Readings taken where the paper leaves a choice (each is repeated in the
design notes of the repository):

* Input streams are used as given: the caller applies the L2 normalisation
  and the temperature of Sec. 3.1 (``q = tau*q_hat``, ``k = k_hat``,
  ``r = r_hat``) before calling.  The layer core starts at the composite
  query.  The gated RMSNorm of eq:gated-output is applied after the core.
* The 1/sqrt(m) factor is kept in both feature vectors exactly as eq:prf
  writes it (App. A, "Feature scaling", says the output does not depend on it).
* eps is added to Z as eq:linearized-output writes it (the unshifted Z).
  The log-space form adds it to the shifted Z; the two agree whenever
  Z >> eps, which every test case satisfies.
* The key-side log-space shift is a running (causal) maximum of the key log
  features, carried through the state as a scale; App. B.2 evaluates the key
  features without a shift.  Either way the exact output is the same.
* Omega is one [m, D] bank per head, an input (App. B.1: a fixed,
  non-trainable buffer).  Its sampler lives in ``oracle.features``.
* The gradient treats every stabilising shift as a constant (the shifts
  cancel in the ratio, App. B.2), i.e. it is the exact gradient of the
  function above.

Every array is float64.  Shapes: q, k, r [n, D]; v, u [n, Dv]; Omega [m, D].
"""

from __future__ import annotations

import numpy as np

EPS = 1e-30


def _f64(*xs):
    return [np.asarray(x, dtype=np.float64) for x in xs]


# ---------------------------------------------------------------------------
# Building blocks
# ---------------------------------------------------------------------------

def phi(X, Omega):
    """Positive random features, Sec. 3.2 eq:prf.

    phi(x) = m^{-1/2} exp(Omega x - |x|^2/2), elementwise exp.
    X: [..., D] -> [..., m].
    """
    X, Omega = _f64(X, Omega)
    m = Omega.shape[0]
    logf = X @ Omega.T - 0.5 * np.sum(X * X, axis=-1, keepdims=True)
    return np.exp(logf) / np.sqrt(m)


def log_features(X, Omega):
    """Log feature ell = Omega x - |x|^2/2 (App. B.2, without the 1/sqrt(m))."""
    X, Omega = _f64(X, Omega)
    return X @ Omega.T - 0.5 * np.sum(X * X, axis=-1, keepdims=True)


def anchor_window(i, w):
    """Anchor set C_i of Sec. 3.3, 0-based: {max(0, i-w+1), ..., i}."""
    return np.arange(max(0, i - w + 1), i + 1)


def composite_query(q_i, r_C):
    """z_ic = q_i (*) r_c for every anchor row of ``r_C`` (Sec. 3.2)."""
    return np.asarray(q_i, np.float64)[None, :] * np.asarray(r_C, np.float64)


def trilinear_score(q, k, r):
    """s_ijc via the rewrite of eq:score-rewrite-intro / eq:two-views.

    s_ijc = ((q_i (*) r_c)^T k_j; returned as an [n, n, n] array indexed
    [i, j, c].  Used to pin the rewrite against the explicit triple sum.
    """
    q, k, r = _f64(q, k, r)
    z = q[:, None, :] * r[None, :, :]          # [i, c, a]
    return np.einsum("ica,ja->ijc", z, k)


# ---------------------------------------------------------------------------
# Forward: four forms of the same function
# ---------------------------------------------------------------------------

def forward_pair(q, k, v, r, u, Omega, w, eps=EPS):
    """Pair form (App. A, "Why the normalization is still joint").

    Materialises every approximate pair weight
        kappa~_ijc = phi(z_ic)^T phi(k_j),  j <= i, c in C_i,
    and sums numerator and denominator over the same joint set.
    O(n^2 w m); for n up to a few hundred.
    """
    q, k, v, r, u, Omega = _f64(q, k, v, r, u, Omega)
    n, Dv = v.shape
    out = np.zeros((n, Dv))
    chi = phi(k, Omega)                         # [n, m]
    for i in range(n):
        C = anchor_window(i, w)
        F = phi(composite_query(q[i], r[C]), Omega)     # [|C|, m]
        kappa = F @ chi[: i + 1].T                      # [|C|, i+1]
        # numerator: sum_c sum_j kappa_cj (v_j (*) u_c)
        N = np.sum(u[C] * (kappa @ v[: i + 1]), axis=0)
        Z = kappa.sum()
        out[i] = N / (Z + eps)
    return out


def forward_recurrent(q, k, v, r, u, Omega, w, eps=EPS, return_Z=False):
    """Recurrent form: eq:Mstate, eq:astate token by token, then eq:Ni, eq:Zi,
    eq:linearized-output.  This is the definition the GPU path is judged
    against.
    """
    q, k, v, r, u, Omega = _f64(q, k, v, r, u, Omega)
    n, Dv = v.shape
    m = Omega.shape[0]
    M = np.zeros((m, Dv))
    a = np.zeros(m)
    out = np.zeros((n, Dv))
    Zs = np.zeros(n)
    for i in range(n):
        chi = phi(k[i], Omega)
        M += np.outer(chi, v[i])                        # eq:Mstate
        a += chi                                        # eq:astate
        C = anchor_window(i, w)
        F = phi(composite_query(q[i], r[C]), Omega)     # [|C|, m]
        N = np.sum((F @ M) * u[C], axis=0)              # eq:Ni (eq:swap-sum)
        Z = np.sum(F @ a)                               # eq:Zi
        out[i] = N / (Z + eps)                          # eq:linearized-output
        Zs[i] = Z
    return (out, Zs) if return_Z else out


def forward_logspace(q, k, v, r, u, Omega, w, eps=EPS):
    """Log-space form (App. B.2) with a causal key-side shift.

    Query side: ell_icp = omega_p^T z_ic - |z_ic|^2/2 and
    L_i = max over c in C_i and p of ell_icp; features exp(ell - L_i).
    Key side: lambda_jp = omega_p^T k_j - |k_j|^2/2 and the running maximum
    R_i = max_{j<=i, p} lambda_jp; the state is carried in the frame R_i,
        M^_i = e^{R_{i-1}-R_i} M^_{i-1} + e^{lambda_i - R_i} v_i^T / sqrt(m),
    so that M_i = e^{R_i} M^_i.  Both shifts multiply N_i and Z_i by the same
    factor e^{-(L_i+R_i)} and cancel in the ratio.

    Returns (out, L, R, Zhat) with Zhat = Z_i e^{-(L_i+R_i)} and eps added
    to Zhat.
    """
    q, k, v, r, u, Omega = _f64(q, k, v, r, u, Omega)
    n, Dv = v.shape
    m = Omega.shape[0]
    Mh = np.zeros((m, Dv))
    ah = np.zeros(m)
    R = -np.inf
    out = np.zeros((n, Dv))
    Ls, Rs, Zh = np.zeros(n), np.zeros(n), np.zeros(n)
    for i in range(n):
        lam = log_features(k[i], Omega)
        Rn = max(R, lam.max())
        scale = np.exp(R - Rn) if np.isfinite(R) else 0.0
        Mh = scale * Mh + np.outer(np.exp(lam - Rn), v[i]) / np.sqrt(m)
        ah = scale * ah + np.exp(lam - Rn) / np.sqrt(m)
        R = Rn
        C = anchor_window(i, w)
        ell = log_features(composite_query(q[i], r[C]), Omega)   # [|C|, m]
        L = ell.max()
        psi = np.exp(ell - L) / np.sqrt(m)
        N = np.sum((psi @ Mh) * u[C], axis=0)
        Z = np.sum(psi @ ah)
        out[i] = N / (Z + eps)
        Ls[i], Rs[i], Zh[i] = L, R, Z
    return out, Ls, Rs, Zh


def forward_chunked(q, k, v, r, u, Omega, w, chunk=32, feature_block=128, eps=EPS):
    """Chunked evaluation (App. C "Host preparation" and state reconstruction,
    with the query-side shift of App. B.2 taken per feature block).

    States: the key features are grouped into chunks of ``chunk`` tokens
    (right-padded with zero features); the state of row i is the exclusive
    prefix over earlier chunks (eq:Mstate, eq:astate summed chunk by chunk)
    plus the tokens j <= i of its own chunk.

    Readout: the log features of all anchors and all features of a row are
    formed at once.  The features are split into blocks of ``feature_block``;
    each block b is shifted by its own maximum L_b, giving partial sums
    (N_b, Z_b) of eq:Ni and eq:Zi scaled by e^{-L_b}.  The blocks are then
    merged with the common shift L = max_b L_b: N = sum_b e^{L_b - L} N_b and
    likewise Z.  The shift cancels in eq:linearized-output; eps is compared
    with the unshifted Z, so it enters as eps e^{-L}.
    """
    q, k, v, r, u, Omega = _f64(q, k, v, r, u, Omega)
    n, Dv = v.shape
    m = Omega.shape[0]
    nchunks = -(-n // chunk)
    feats = np.zeros((nchunks * chunk, m))
    feats[:n] = phi(k, Omega)
    vals = np.zeros((nchunks * chunk, Dv))
    vals[:n] = v
    feats = feats.reshape(nchunks, chunk, m)
    vals = vals.reshape(nchunks, chunk, Dv)
    # per-chunk totals, then the exclusive prefix over chunks
    tot_M = np.matmul(feats.transpose(0, 2, 1), vals)                  # [nchunks, m, Dv]
    tot_a = feats.sum(axis=1)                                          # [nchunks, m]
    before_M = np.cumsum(tot_M, axis=0) - tot_M
    before_a = np.cumsum(tot_a, axis=0) - tot_a
    blocks = [np.arange(p0, min(m, p0 + feature_block)) for p0 in range(0, m, feature_block)]
    out = np.zeros((n, Dv))
    for i in range(n):
        b, t = divmod(i, chunk)
        M_i = before_M[b] + feats[b, : t + 1].T @ vals[b, : t + 1]
        a_i = before_a[b] + feats[b, : t + 1].sum(axis=0)
        C = anchor_window(i, w)
        ell = log_features(composite_query(q[i], r[C]), Omega)       # [|C|, m]
        L_b = np.array([ell[:, P].max() for P in blocks])
        parts = []
        for P, Lb in zip(blocks, L_b):
            psi = np.exp(ell[:, P] - Lb) / np.sqrt(m)
            parts.append((np.sum((psi @ M_i[P]) * u[C], axis=0), np.sum(psi @ a_i[P])))
        L = L_b.max()
        scale = np.exp(L_b - L)
        N = sum(s * nb for s, (nb, _) in zip(scale, parts))
        Z = sum(s * zb for s, (_, zb) in zip(scale, parts))
        out[i] = N / (Z + eps * np.exp(-L))
    return out


# ---------------------------------------------------------------------------
# Exact-kernel operators that the estimator approximates (tests only)
# ---------------------------------------------------------------------------

def exact_window(q, k, v, r, u, w):
    """o_i^(w) of App. A eq:exact-window-app: the same window with the exact
    kernel kappa_ijc = exp(z_ic^T k_j).  The random-feature output converges
    to it as m grows (Lemma 1; the ratio is biased at finite m, Sec. 3.2)."""
    q, k, v, r, u = _f64(q, k, v, r, u)
    n, Dv = v.shape
    out = np.zeros((n, Dv))
    for i in range(n):
        C = anchor_window(i, w)
        kappa = np.exp(composite_query(q[i], r[C]) @ k[: i + 1].T)   # [|C|, i+1]
        out[i] = np.sum(u[C] * (kappa @ v[: i + 1]), axis=0) / kappa.sum()
    return out


# ---------------------------------------------------------------------------
# Backward: exact gradient of sum_i dO_i . o~_i
# ---------------------------------------------------------------------------

def backward(q, k, v, r, u, Omega, w, dO, eps=EPS, term_scale=None):
    """Exact gradient of L = sum_i dO_i . o~_i w.r.t. q, k, v, r, u.

    Follows the two sweeps of App. C ("Backward query sweep", "Backward
    state sweep") and the host differentiation of the key feature map:

      dN_i = g_i/(Z_i+eps),  dZ_i = -(g_i . o~_i)/(Z_i+eps)
      per anchor c:  dA_ic = dN_i (*) u_c,   du_c += dN_i (*) A_ic
                     dF_ic = M_i dA_ic + dZ_i a_i      (F_ic = phi(z_ic))
                     dell  = dF_ic (*) F_ic            (F = m^{-1/2} e^ell)
                     dz_ic = sum_p dell_p (omega_p - z_ic)   (d ell/d z = omega - z)
                     dq_i += dz_ic (*) r_c,  dr_c += dz_ic (*) q_i
      state:  dM_i = sum_c F_ic dA_ic^T,  da_i = dZ_i sum_c F_ic
              G_j = sum_{i>=j} dM_i,  h_j = sum_{i>=j} da_i   (adjoint of the
              prefix recurrences eq:Mstate / eq:astate)
              dchi_j = G_j v_j + h_j,  dv_j += G_j^T chi_j
      key map: dlambda_j = dchi_j (*) chi_j,  dk_j = sum_p dlambda_jp (omega_p - k_j)

    The rows are swept from the end of the sequence to the start, so G and h
    are running sums; the prefix state M_i is rebuilt on the way back by
    removing chi_i v_i^T (the recurrence run in reverse).

    If ``term_scale`` is a dict, its entry "dk" receives, per key j, the norm
    of the same sums taken over absolute values (|dA|, |dZ|, |v_j|, |Omega|,
    |k_j|): the first-order bound on what a relative perturbation u of every
    summed term can change in dk_j is u times that scale.  It does not change
    the gradients.
    """
    q, k, v, r, u, Omega, dO = _f64(q, k, v, r, u, Omega, dO)
    n, D = q.shape
    Dv = v.shape[1]
    m = Omega.shape[0]
    chi = phi(k, Omega)                              # [n, m]
    M = chi.T @ v                                    # M_{n-1}
    a = chi.sum(axis=0)                              # a_{n-1}
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    dr = np.zeros_like(r)
    du = np.zeros_like(u)
    G = np.zeros((m, Dv))
    h = np.zeros(m)
    if term_scale is not None:
        Ga, ha, Tk = np.zeros((m, Dv)), np.zeros(m), np.zeros(n)
    for i in range(n - 1, -1, -1):
        C = anchor_window(i, w)
        z = composite_query(q[i], r[C])              # [|C|, D]
        F = phi(z, Omega)                            # [|C|, m]
        A = F @ M                                    # [|C|, Dv]
        N = np.sum(A * u[C], axis=0)
        Z = np.sum(F @ a)
        o = N / (Z + eps)
        g = dO[i]
        dN = g / (Z + eps)
        dZ = -np.dot(g, o) / (Z + eps)
        dA = dN[None, :] * u[C]                      # [|C|, Dv]
        du[C] += dN[None, :] * A
        dF = dA @ M.T + dZ * a[None, :]              # [|C|, m]
        dell = dF * F
        dz = dell @ Omega - dell.sum(axis=1, keepdims=True) * z   # [|C|, D]
        dq[i] += np.sum(dz * r[C], axis=0)
        dr[C] += dz * q[i][None, :]
        G += F.T @ dA                                # dM_i
        h += dZ * F.sum(axis=0)                      # da_i
        dchi = G @ v[i] + h
        dv[i] += G.T @ chi[i]
        dlam = dchi * chi[i]
        dk[i] = dlam @ Omega - dlam.sum() * k[i]
        if term_scale is not None:
            Ga += F.T @ np.abs(dA)
            ha += abs(dZ) * F.sum(axis=0)
            t = (Ga @ np.abs(v[i]) + ha) * chi[i]
            Tk[i] = np.linalg.norm(t @ np.abs(Omega) + t.sum() * np.abs(k[i]))
        # rebuild M_{i-1}, a_{i-1}
        M = M - np.outer(chi[i], v[i])
        a = a - chi[i]
    if term_scale is not None:
        term_scale["dk"] = Tk
    return dq, dk, dv, dr, du


# ---------------------------------------------------------------------------
# Autoregressive decode (Theorem 1: the state is M, a and the last w (r, u))
# ---------------------------------------------------------------------------

def prefill_state(k, v, r, u, Omega, w):
    """State after a prefix of n tokens (Theorem 1): M_{n-1}, a_{n-1} and the
    rolling anchor buffer, token j held in slot j mod w."""
    k, v, r, u, Omega = _f64(k, v, r, u, Omega)
    n = k.shape[0]
    chi = phi(k, Omega)
    ring_r = np.zeros((w, r.shape[1]))
    ring_u = np.zeros((w, u.shape[1]))
    for j in range(max(0, n - w), n):
        ring_r[j % w] = r[j]
        ring_u[j % w] = u[j]
    return {"M": chi.T @ v, "a": chi.sum(axis=0), "ring_r": ring_r,
            "ring_u": ring_u, "pos": n}


def decode_step(state, q_t, k_t, v_t, r_t, u_t, Omega, w, eps=EPS):
    """One decode step (Theorem 1): append token t = pos, update M and a by
    eq:Mstate / eq:astate, push (r_t, u_t) into slot t mod w, and read q_t
    out over the min(t+1, w) most recent anchors, the new token included.
    Returns (out, new_state); ``state`` is not modified.
    """
    q_t, k_t, v_t, r_t, u_t, Omega = _f64(q_t, k_t, v_t, r_t, u_t, Omega)
    t = int(state["pos"])
    chi = phi(k_t, Omega)
    M = state["M"] + np.outer(chi, v_t)
    a = state["a"] + chi
    ring_r = state["ring_r"].copy()
    ring_u = state["ring_u"].copy()
    ring_r[t % w] = r_t
    ring_u[t % w] = u_t
    slots = [(t - s) % w for s in range(min(t + 1, w))]
    F = phi(composite_query(q_t, ring_r[slots]), Omega)
    N = np.sum((F @ M) * ring_u[slots], axis=0)
    Z = np.sum(F @ a)
    new = {"M": M, "a": a, "ring_r": ring_r, "ring_u": ring_u, "pos": t + 1}
    return N / (Z + eps), new

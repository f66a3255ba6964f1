"""Random-feature bank samplers (test infrastructure only).

``orthogonal_bank`` follows App. B.1 step by step:
  1. draw G in R^{D x D} with iid N(0,1) entries and factor G = QR;
  2. multiply each column of Q by sign(R_aa) (needed for a Haar-distributed
     orthogonal factor);
  3. take the rows of Q^T as directions and scale each by an independent
     chi_D radius;
  4. stack blocks until there are m rows.
Each row is then marginally N(0, I_D), so Lemma 1 still holds.

``orthogonal_block`` / ``orthogonal_bank_from`` take the random draws (G and
the chi_D radii) as inputs, so a device sampler can be compared with the same
draws.
"""

import numpy as np


def orthogonal_block(G, radii, sign_correct=True):
    """One block of App. B.1 from given draws: G [D, D] iid N(0, 1) and radii
    [D] (chi_D draws).  G = QR (Householder, numpy/LAPACK), columns of Q times
    sign(R_aa) when sign_correct, rows of Q^T scaled by the radii: [D, D]."""
    G = np.asarray(G, np.float64)
    Q, R = np.linalg.qr(G)
    if sign_correct:
        Q = Q * np.sign(np.diag(R))[None, :]
    return Q.T * np.asarray(radii, np.float64)[:, None]


def orthogonal_bank_from(G, radii, m, sign_correct=True):
    """Bank of m rows from per-block draws G [nb, D, D] and radii [nb, D]
    (nb = ceil(m / D) blocks stacked, the last one truncated)."""
    blocks = [orthogonal_block(G[b], radii[b], sign_correct) for b in range(len(G))]
    return np.concatenate(blocks, axis=0)[:m]


def orthogonal_bank(rng, m, D, sign_correct=True):
    """Orthogonal random-feature bank of App. B.1, [m, D] float64."""
    blocks = []
    rows = 0
    while rows < m:
        G = rng.standard_normal((D, D))
        radii = np.sqrt(rng.chisquare(D, size=D))
        blocks.append(orthogonal_block(G, radii, sign_correct))
        rows += D
    return np.concatenate(blocks, axis=0)[:m]

"""Random-feature bank samplers (test infrastructure only).

``orthogonal_bank`` follows App. B.1 step by step:
  1. draw G in R^{D x D} with iid N(0,1) entries and factor G = QR;
  2. multiply each column of Q by sign(R_aa) (needed for a Haar-distributed
     orthogonal factor);
  3. take the rows of Q^T as directions and scale each by an independent
     chi_D radius;
  4. stack blocks until there are m rows.
Each row is then marginally N(0, I_D), so Lemma 1 still holds.

``iid_bank`` is the plain Gaussian bank the synthetic workloads use.
"""

import numpy as np


def iid_bank(rng, m, D):
    """Omega with iid N(0, 1) entries, [m, D]."""
    return rng.standard_normal((m, D))


def orthogonal_bank(rng, m, D, sign_correct=True):
    """Orthogonal random-feature bank of App. B.1, [m, D] float64."""
    blocks = []
    rows = 0
    while rows < m:
        G = rng.standard_normal((D, D))
        Q, R = np.linalg.qr(G)
        if sign_correct:
            Q = Q * np.sign(np.diag(R))[None, :]
        radii = np.sqrt(rng.chisquare(D, size=D))
        blocks.append(Q.T * radii[:, None])
        rows += D
    return np.concatenate(blocks, axis=0)[:m]

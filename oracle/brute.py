"""Pure-Python brute force of the LinSimp output (test infrastructure only).

No numpy: nested loops over positions, anchors, features and coordinates,
straight from the definitions, for tiny inputs (n <= 8, D <= 4, m <= 8).
Inputs are lists of lists of floats.

    score     s_ijc = sum_a q_ia k_ja r_ca          Sec. 3.1 eq:trilinear-score
    feature   phi_p(x) = m^{-1/2} exp(sum_a Omega_pa x_a - sum_a x_a^2 / 2)   eq:prf
    weight    kappa~_ijc = sum_p phi_p(q_i (*) r_c) phi_p(k_j)
    output    o~_i = sum_{c in C_i, j<=i} kappa~_ijc (v_j (*) u_c)
                     / (sum_{c in C_i, j<=i} kappa~_ijc + eps)      App. A
"""

import math


def score(q, k, r, i, j, c):
    """Explicit triple sum of eq:trilinear-score (streams used as given)."""
    return sum(q[i][a] * k[j][a] * r[c][a] for a in range(len(q[i])))


def feature(x, Omega, p):
    """p-th coordinate of phi(x), eq:prf."""
    m = len(Omega)
    dot = sum(Omega[p][a] * x[a] for a in range(len(x)))
    sq = sum(xa * xa for xa in x)
    return math.exp(dot - 0.5 * sq) / math.sqrt(m)


def output(q, k, v, r, u, Omega, w, eps=1e-30):
    """o~_i for every i by summing every pair weight (j, c) explicitly."""
    n = len(q)
    Dv = len(v[0])
    m = len(Omega)
    out = []
    for i in range(n):
        num = [0.0] * Dv
        den = 0.0
        for c in range(max(0, i - w + 1), i + 1):
            z = [q[i][a] * r[c][a] for a in range(len(q[i]))]
            fz = [feature(z, Omega, p) for p in range(m)]
            for j in range(0, i + 1):
                kap = sum(fz[p] * feature(k[j], Omega, p) for p in range(m))
                den += kap
                for d in range(Dv):
                    num[d] += kap * v[j][d] * u[c][d]
        out.append([num[d] / (den + eps) for d in range(Dv)])
    return out


def exact_output(q, k, v, r, u, w):
    """Exact windowed operator of App. A eq:exact-window-app by brute force:
    kappa_ijc = exp(s_ijc) with the explicit triple-sum score."""
    n = len(q)
    Dv = len(v[0])
    out = []
    for i in range(n):
        num = [0.0] * Dv
        den = 0.0
        for c in range(max(0, i - w + 1), i + 1):
            for j in range(0, i + 1):
                kap = math.exp(score(q, k, r, i, j, c))
                den += kap
                for d in range(Dv):
                    num[d] += kap * v[j][d] * u[c][d]
        out.append([num[d] / den for d in range(Dv)])
    return out

"""Monte-Carlo tools for the random-feature kernel (test infrastructure only).

Lemma 1 (Sec. 3.2): for rows omega ~ N(0, I_D),
    E[phi(x)^T phi(y)] = exp(x^T y).
The proof uses the Gaussian moment-generating function
E[exp(omega^T s)] = exp(|s|^2 / 2).  The same function gives the second
moment, hence the variance of the estimate for m independent rows:

    Var[phi(x)^T phi(y)] = exp(2 x^T y) (exp(|x + y|^2) - 1) / m.

(Each term e^{omega^T (x+y) - (|x|^2+|y|^2)/2} has second moment
e^{2|x+y|^2 - |x|^2 - |y|^2}; subtracting the squared mean e^{2 x^T y}
leaves e^{2 x^T y}(e^{|x+y|^2} - 1).)
"""

import numpy as np

from .linsimp import phi


def kernel_estimate(x, y, Omega):
    """phi(x)^T phi(y) for one bank Omega [m, D] (the estimate of Lemma 1)."""
    return float(phi(x, Omega) @ phi(y, Omega))


def exact_kernel(x, y):
    """exp(x^T y), the kernel Lemma 1 says the estimate is unbiased for."""
    return float(np.exp(np.dot(np.asarray(x, np.float64), np.asarray(y, np.float64))))


def estimate_variance(x, y, m):
    """Closed-form variance of phi(x)^T phi(y) for m iid N(0, I) rows."""
    x = np.asarray(x, np.float64)
    y = np.asarray(y, np.float64)
    s = x + y
    return float(np.exp(2 * x @ y) * (np.exp(s @ s) - 1.0) / m)

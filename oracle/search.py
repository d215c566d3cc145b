"""SGD-based search for the dropout-pattern distribution K (Sec. III-C, Alg. 1).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Alg. 1 parameterises K by logits v (d = softmax(v)) and minimises

    L(d) = lambda1 * (d . p_u - p)**2 + lambda2 * (1/N) * sum_i d_i log d_i

with p_u = [(i - 1) / i for i = 1..N] (the drop rate of period i), by gradient
descent on v until the loss change falls below a threshold. The paper leaves
lambda1, lambda2 (summing to 1), the step size, the initial v and the threshold
open; the readings used are lambda1 = 0.99, v = 0, step 10, threshold 1e-15.

Two oracles are given:

* ``search_gd``   - the paper's iteration, step by step (softmax, the two loss
                    terms, the gradient w.r.t. v, a descent step, the stop rule);
* ``closed_form`` - the unique minimiser. L is strictly convex on the simplex,
                    so its stationarity conditions characterise it:
                    d_i proportional to exp(beta * p_u[i]) with
                    beta = -(2 * lambda1 * N / lambda2) * (mu(beta) - p),
                    mu(beta) = d(beta) . p_u. F(beta) = beta + (2 lambda1 N /
                    lambda2)(mu(beta) - p) is strictly increasing, so bisection
                    on beta finds it to machine precision.
"""

import math

import numpy as np


def drop_rates(n):
    """p_u: the global drop rate (i - 1) / i of each period i = 1..n (Alg. 1)."""
    return np.array([(i - 1) / i for i in range(1, n + 1)], dtype=np.float64)


def softmax(v):
    v = np.asarray(v, dtype=np.float64)
    e = np.exp(v - v.max())
    return e / e.sum()


def loss(d, p, lam1, lam2):
    """Alg. 1 loss: lambda1 * E_p + lambda2 * E_n (0 log 0 taken as 0)."""
    d = np.asarray(d, dtype=np.float64)
    n = d.size
    e_p = (float(d @ drop_rates(n)) - p) ** 2
    e_n = sum(x * math.log(x) for x in d if x > 0.0) / n
    return lam1 * e_p + lam2 * e_n


def grad_d(d, p, lam1, lam2):
    """Gradient of the loss with respect to d."""
    n = d.size
    pu = drop_rates(n)
    mu = float(d @ pu)
    return 2.0 * lam1 * (mu - p) * pu + (lam2 / n) * (np.log(d) + 1.0)


def grad_v(v, p, lam1, lam2):
    """Gradient of the loss with respect to the logits v (chain rule through
    softmax: dL/dv_j = d_j * (g_j - sum_i d_i g_i))."""
    d = softmax(v)
    g = grad_d(d, p, lam1, lam2)
    return d * (g - float(d @ g))


def search_gd(p, n, lam1=0.99, lr=10.0, threshold=1e-15, max_iters=1_000_000):
    """Alg. 1 as printed: gradient descent on v until |delta loss| < threshold.

    Returns (d, iterations, converged).
    """
    lam2 = 1.0 - lam1
    v = np.zeros(n, dtype=np.float64)
    prev = None
    for it in range(1, max_iters + 1):
        d = softmax(v)
        cur = loss(d, p, lam1, lam2)
        if prev is not None and abs(cur - prev) < threshold:
            return d, it, True
        prev = cur
        v = v - lr * grad_v(v, p, lam1, lam2)
    return softmax(v), max_iters, False


def gibbs(beta, n):
    """d_i proportional to exp(beta * p_u[i])."""
    return softmax(beta * drop_rates(n))


def closed_form(p, n, lam1=0.99):
    """The unique minimiser of the Alg. 1 loss, by bisection on beta."""
    lam2 = 1.0 - lam1
    if n == 1:
        return np.ones(1)
    c = 2.0 * lam1 * n / lam2
    pu = drop_rates(n)

    def f(beta):
        return beta + c * (float(gibbs(beta, n) @ pu) - p)

    lo, hi = -(c + 1.0), c + 1.0
    for _ in range(400):
        mid = 0.5 * (lo + hi)
        if f(mid) < 0.0:
            lo = mid
        else:
            hi = mid
        if hi - lo <= 1e-15 * max(1.0, abs(mid)):
            break
    return gibbs(0.5 * (lo + hi), n)


def distribution_for_rate(p, n, lam1=0.99):
    """K for target rate p: e_1 for p = 0 (no dropout), the minimiser otherwise.

    Rates outside [0, (n-1)/n) cannot be reached by periods 1..n and are rejected.
    """
    if not (0.0 <= p < (n - 1) / n) and not (p == 0.0 and n == 1):
        raise ValueError("p must satisfy 0 <= p < (n-1)/n")
    if p == 0.0:
        e = np.zeros(n)
        e[0] = 1.0
        return e
    return closed_form(p, n, lam1)


def global_rate(K):
    """p_g = sum_i k_i (i - 1) / i (Eq. 3)."""
    K = np.asarray(K, dtype=np.float64)
    return float(K @ drop_rates(K.size))


def kkt_residual(d, p, lam1):
    """Spread max - min of dL/dd: zero at the interior minimiser, where every
    partial derivative equals the simplex multiplier."""
    g = grad_d(np.asarray(d, dtype=np.float64), p, lam1, 1.0 - lam1)
    return float(g.max() - g.min())

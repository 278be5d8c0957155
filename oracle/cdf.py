"""Oracle: the ordinal-logistic coverage model and its fit.

Test infrastructure only (see the package docstring).  Float64 throughout.

Paper passages followed:
* Sec. IV-C, Eq. 6-8: the probability that an extra budget delta covers the routed set,
  p_delta(x) = Pr(delta >= delta* | x), is modelled as sigmoid(theta_delta - w.x) for
  delta = 0..N-k with non-decreasing thresholds theta, so p_delta is a CDF in delta.
* Sec. IV-D, "CDF Model Training", Eq. 11: every sample (x, delta*) gives the targets
  [delta >= delta*] for delta = 0..N-k; the loss of a sample is the sum over delta of
  the binary cross-entropy between p_delta(x) and its target.  The fit minimises the
  mean of that loss over the samples.

Readings (where the paper is silent):
* one model per MoE layer, fitted on that layer's samples (the overhead analysis of
  Sec. V-F counts about 2N CDF parameters per layer);
* x is the prefetch probability vector in ranked order, as in ``routing``;
* an optional L2 penalty ridge/2 * (|w|^2 + |theta|^2) keeps thresholds finite at levels
  that every sample (or no sample) reaches; ridge = 0 is the paper's loss exactly.

The optimiser (scipy L-BFGS) is a library step; the ordering of theta is enforced by
writing theta_0 = c_0 and theta_delta = theta_{delta-1} + softplus(c_delta).
"""
from __future__ import annotations

import numpy as np
from scipy.optimize import minimize


def _softplus(z):
    return np.logaddexp(0.0, z)


def _sigmoid(z):
    return 0.5 * (1.0 + np.tanh(0.5 * z))


def cumulative_targets(dstar, n_levels: int) -> np.ndarray:
    """Eq. 11 targets: row i, column delta holds 1 when delta >= delta*_i, else 0."""
    d = np.asarray(dstar, dtype=np.int64)
    levels = np.arange(n_levels, dtype=np.int64)
    return (levels[None, :] >= d[:, None]).astype(np.float64)


def coverage_prob(X, w, theta) -> np.ndarray:
    """Eq. 8 for every sample and level: [n, N-k+1]."""
    X = np.asarray(X, dtype=np.float64)
    s = X @ np.asarray(w, dtype=np.float64)
    return _sigmoid(np.asarray(theta, dtype=np.float64)[None, :] - s[:, None])


def cdf_loss(X, dstar, w, theta, ridge: float = 0.0) -> float:
    """Mean over samples of the Eq. 11 loss, plus the optional ridge term.

    With a = theta_delta - w.x: -log sigmoid(a) = softplus(-a) and
    -log(1 - sigmoid(a)) = softplus(a).
    """
    X = np.asarray(X, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    theta = np.asarray(theta, dtype=np.float64)
    a = theta[None, :] - (X @ w)[:, None]
    t = cumulative_targets(dstar, theta.size)
    per_sample = (t * _softplus(-a) + (1.0 - t) * _softplus(a)).sum(axis=1)
    return float(per_sample.mean() + 0.5 * ridge * (w @ w + theta @ theta))


def cdf_loss_grad(X, dstar, w, theta, ridge: float = 0.0):
    """Gradient of ``cdf_loss`` with respect to (w, theta).

    d/da of the per-level cross-entropy is sigmoid(a) - target; a grows with theta_delta
    and falls with w.x.
    """
    X = np.asarray(X, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    theta = np.asarray(theta, dtype=np.float64)
    n = X.shape[0]
    a = theta[None, :] - (X @ w)[:, None]
    r = _sigmoid(a) - cumulative_targets(dstar, theta.size)      # [n, L]
    g_theta = r.sum(axis=0) / n + ridge * theta
    g_w = -(X.T @ r.sum(axis=1)) / n + ridge * w
    return g_w, g_theta


def _theta_of(c):
    return np.concatenate([[c[0]], c[0] + np.cumsum(_softplus(c[1:]))])


def fit_cdf(X, dstar, n_levels: int, ridge: float = 0.0, max_iter: int = 5000):
    """Minimise the Eq. 11 loss over (w, theta) with theta non-decreasing.

    Start: w = 0, thresholds spaced 0.5 apart from -1 (a neutral point, not the answer).
    Returns (w [E], theta [n_levels]) as float64.
    """
    X = np.asarray(X, dtype=np.float64)
    dstar = np.asarray(dstar, dtype=np.int64)
    E = X.shape[1]
    L = int(n_levels)
    if dstar.min() < 0 or dstar.max() >= L:
        raise ValueError("delta* outside 0..N-k")

    def unpack(v):
        return v[:E], v[E:]

    def objective(v):
        w, c = unpack(v)
        theta = _theta_of(c)
        f = cdf_loss(X, dstar, w, theta, ridge)
        g_w, g_theta = cdf_loss_grad(X, dstar, w, theta, ridge)
        # theta_j = c_0 + sum_{1 <= i <= j} softplus(c_i)
        tail = np.cumsum(g_theta[::-1])[::-1]                  # sum_{j >= i} g_theta_j
        g_c = np.empty(L)
        g_c[0] = tail[0]
        g_c[1:] = _sigmoid(c[1:]) * tail[1:]
        return f, np.concatenate([g_w, g_c])

    c0 = np.full(L, np.log(np.expm1(0.5)))
    c0[0] = -1.0
    v0 = np.concatenate([np.zeros(E), c0])
    res = minimize(objective, v0, jac=True, method="L-BFGS-B",
                   options={"maxiter": max_iter, "maxfun": 4 * max_iter, "ftol": 1e-15,
                            "gtol": 1e-11})
    w, c = unpack(res.x)
    return w, _theta_of(c)

"""Pins of the oracle's ordinal coverage model and its Eq. 11 fit (CPU only).

* a loss value worked by hand;
* closed form: with uninformative features (x = 0) the optimum of Eq. 11 sets
  sigmoid(theta_delta) to the empirical CDF of delta*, so theta_delta = logit(F(delta));
* recovery: samples drawn from a known ordinal-logistic model give back its parameters
  (this fails if the sign of w.x or the direction of the targets is flipped);
* calibration: the Eq. 9 budget taken with the fitted model covers the routed set for
  at least a fraction tau of the samples, which is what p_delta = Pr(delta >= delta*)
  promises (Eq. 6);
* the analytic gradient matches central differences of the loss.
"""
import math

import numpy as np
import pytest

from oracle import cdf


def test_loss_hand_value():
    # one sample, two levels, w.x = 0, theta = (0, 0), delta* = 1: targets (0, 1), both
    # probabilities 1/2, so the loss is ln 2 + ln 2
    X = np.zeros((1, 3))
    got = cdf.cdf_loss(X, [1], np.zeros(3), np.zeros(2))
    assert got == pytest.approx(2.0 * math.log(2.0), rel=1e-15)
    # theta = (-1, 2), delta* = 0: targets (1, 1): softplus(1) + softplus(-2)
    got = cdf.cdf_loss(X, [0], np.zeros(3), np.array([-1.0, 2.0]))
    assert got == pytest.approx(math.log1p(math.e) + math.log1p(math.exp(-2.0)), rel=1e-14)


def test_targets_are_cumulative_indicators():
    t = cdf.cumulative_targets([0, 2, 3], 4)
    assert t.tolist() == [[1, 1, 1, 1], [0, 0, 1, 1], [0, 0, 0, 1]]


def test_closed_form_without_features():
    rng = np.random.default_rng(11)
    L = 6
    # every level below the last has 0 < F < 1; the last level always has F = 1
    probs = np.array([0.15, 0.25, 0.2, 0.15, 0.15, 0.10])
    dstar = rng.choice(L, size=4000, p=probs)
    X = np.zeros((dstar.size, 5))
    w, theta = cdf.fit_cdf(X, dstar, L)
    F = np.array([(dstar <= d).mean() for d in range(L)])
    want = np.log(F[:-1] / (1.0 - F[:-1]))
    np.testing.assert_allclose(theta[:-1], want, atol=2e-5)
    assert theta[-1] > want[-1] + 5.0          # F = 1 there: the threshold runs off
    assert np.abs(w).max() < 1e-8               # x carries no signal
    assert np.all(np.diff(theta) >= 0.0)


def _sample_model(rng, n, w, theta):
    X = rng.standard_normal((n, w.size))
    p = cdf.coverage_prob(X, w, theta)                       # Pr(delta* <= delta | x)
    u = rng.random(n)
    reach = p >= u[:, None]
    dstar = np.where(reach.any(axis=1), reach.argmax(axis=1), theta.size - 1)
    return X, dstar


def test_recovers_known_parameters():
    rng = np.random.default_rng(12)
    w_true = np.array([1.2, -0.7, 0.0, 0.4, -1.5])
    theta_true = np.array([-1.5, -0.4, 0.3, 1.1, 2.0, 40.0])  # last level: always covered
    X, dstar = _sample_model(rng, 30000, w_true, theta_true)
    w, theta = cdf.fit_cdf(X, dstar, theta_true.size)
    np.testing.assert_allclose(w, w_true, atol=0.08)
    np.testing.assert_allclose(theta[:-1], theta_true[:-1], atol=0.08)


@pytest.mark.parametrize("tau", [0.8, 0.9, 0.95])
def test_budget_rule_with_fitted_model_reaches_tau(tau):
    rng = np.random.default_rng(13)
    w_true = np.array([0.8, -0.5, 0.3])
    theta_true = np.array([-1.0, 0.0, 0.8, 1.5, 2.5, 50.0])
    X, dstar = _sample_model(rng, 20000, w_true, theta_true)
    w, theta = cdf.fit_cdf(X, dstar, theta_true.size)
    def budget(w_, theta_):
        ok = cdf.coverage_prob(X, w_, theta_) >= tau
        return np.where(ok.any(axis=1), ok.argmax(axis=1), theta_.size - 1)

    delta_hat = budget(w, theta)
    coverage = (delta_hat >= dstar).mean()
    assert coverage >= tau - 0.01
    # the fitted model spends about what the true model would
    assert abs(delta_hat.mean() - budget(w_true, theta_true).mean()) < 0.05


def test_gradient_matches_central_differences():
    rng = np.random.default_rng(14)
    X = rng.random((50, 4))
    dstar = rng.integers(0, 5, 50)
    w = rng.standard_normal(4)
    theta = np.sort(rng.standard_normal(5))
    g_w, g_t = cdf.cdf_loss_grad(X, dstar, w, theta, ridge=0.3)
    h = 1e-6
    for i in range(4):
        e = np.zeros(4)
        e[i] = h
        fd = (cdf.cdf_loss(X, dstar, w + e, theta, 0.3) -
              cdf.cdf_loss(X, dstar, w - e, theta, 0.3)) / (2 * h)
        assert g_w[i] == pytest.approx(fd, abs=1e-7)
    for i in range(5):
        e = np.zeros(5)
        e[i] = h
        fd = (cdf.cdf_loss(X, dstar, w, theta + e, 0.3) -
              cdf.cdf_loss(X, dstar, w, theta - e, 0.3)) / (2 * h)
        assert g_t[i] == pytest.approx(fd, abs=1e-7)


def test_ridge_keeps_unreached_levels_finite():
    rng = np.random.default_rng(15)
    dstar = rng.integers(1, 3, 500)            # delta* never 0 and never above 2
    X = rng.random((500, 3))
    w, theta = cdf.fit_cdf(X, dstar, 6, ridge=1e-3)
    assert np.all(np.isfinite(theta)) and np.abs(theta).max() < 60
    assert np.all(np.diff(theta) >= 0.0)
    p = cdf.coverage_prob(X, w, theta)
    assert p[:, 0].mean() < 0.05 and p[:, 2:].mean() > 0.95

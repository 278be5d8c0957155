"""Host side of the ordinal-model training stage against the oracle (CPU only).

The package fits the Eq. 11 objective with its own code (ordered thresholds through
bounded steps); the oracle fits it through softplus steps.  Both must reach the same
optimum of the same strictly convex objective on the same samples.  The samples here are
made by the oracle (the GPU collection step has its own test).
"""
import numpy as np
import pytest

from oracle import cdf as ocdf
from oracle import metrics, routing
from paper_2608_11688_amd import cdf_fit, configs, inputs


def test_delta_star_matches_oracle_enumeration():
    rng = np.random.default_rng(21)
    for N, k in [(8, 2), (32, 8), (64, 8), (5, 5)]:
        ranked = np.stack([rng.permutation(N) for _ in range(200)])
        routed = np.stack([rng.choice(N, k, replace=False) for _ in range(200)])
        got = cdf_fit.delta_star(ranked, routed, k)
        want = [metrics.delta_star(list(ranked[i]), list(routed[i]), k) for i in range(200)]
        assert got.tolist() == want


def oracle_samples(cfg, layer, n, seed=1):
    h_pre, h_post = inputs.hidden_states(cfg, layer, 32, -(-n // 32), seed)
    h_pre, h_post = h_pre.reshape(-1, cfg.d)[:n], h_post.reshape(-1, cfg.d)[:n]
    wg, wpf, bias = inputs.router_weights(cfg, layer)
    zp = routing.router_logits(h_pre, wpf, bias)
    q = routing.softmax(zp)
    zg = routing.router_logits(h_post, wg, bias)
    X, D = [], []
    for i in range(n):
        ranked = routing.rank_experts(zp[i])
        X.append(q[i][ranked])
        routed = routing.rank_experts(zg[i])[:cfg.k]
        D.append(metrics.delta_star(ranked, routed, cfg.k))
    return np.array(X), np.array(D)


@pytest.mark.parametrize("name,ridge", [("granite-1b-a400m", 1e-3), ("tiny", 1e-3),
                                        ("olmoe-1b-7b", 1e-2)])
def test_fit_matches_oracle_fit(name, ridge):
    cfg = configs.CONFIGS[name]
    X, D = oracle_samples(cfg, 0, 256)
    L = cfg.E - cfg.k + 1
    w_o, t_o = ocdf.fit_cdf(X, D, L, ridge=ridge)
    w_p, t_p, loss_p = cdf_fit.fit_layer(X, D, L, ridge=ridge)
    loss_o = ocdf.cdf_loss(X, D, w_o, t_o, ridge)
    assert loss_p == pytest.approx(loss_o, rel=1e-9)
    assert ocdf.cdf_loss(X, D, w_p, t_p, ridge) == pytest.approx(loss_p, rel=1e-12)
    np.testing.assert_allclose(ocdf.coverage_prob(X, w_p, t_p), ocdf.coverage_prob(X, w_o, t_o),
                               atol=1e-5)
    assert np.all(np.diff(t_p) >= 0.0)


def test_fit_rejects_out_of_range_samples():
    X = np.zeros((3, 4))
    with pytest.raises(ValueError):
        cdf_fit.fit_layer(X, [0, 1, 3], 3)
    with pytest.raises(ValueError):
        cdf_fit.fit_layer(X, [-1, 0, 0], 3)

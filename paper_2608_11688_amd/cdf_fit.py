"""Per-layer fit of the ordinal coverage model (paper Sec. IV-C Eq. 8, Sec. IV-D Eq. 11).

This is the method's separate training stage, run once before decoding; no decode step
calls it.  Samples come from the decode kernels themselves, run on held-out tokens:

* apex_prefetch_route with a static budget of N - k and k_max = N returns the whole
  ranked expert list and the prefetch probabilities;
* apex_gate_topk returns the routed set;
* delta* is the ranked position of the deepest routed expert, minus k, floored at 0
  (the smallest budget whose prefix holds the routed set, Eq. 3).

The model input x is the prefetch probability vector in ranked order, the same vector
the ORDINAL policy of apex_prefetch_route dots with w.  The fit minimises, in float64 on
the host, the mean over samples of the sum over delta = 0..N-k of the binary
cross-entropy between sigmoid(theta_delta - w.x) and [delta >= delta*], plus
ridge/2 * (|w|^2 + |theta|^2).  The ridge term keeps thresholds finite at levels that
all or none of the samples reach, and picks one w among those that differ by a constant
(the entries of x sum to one, so such a shift moves into theta).  theta is written as
theta_0 plus running sums of non-negative steps, which L-BFGS-B keeps ordered with
bounds.
"""
from __future__ import annotations

import time

import numpy as np
from scipy.optimize import minimize

from . import configs, inputs, native

DEFAULT_RIDGE = 1e-3
HOLDOUT_SEED = 1          # token streams disjoint from the decode runs (seed 0)


def delta_star(ranked: np.ndarray, routed: np.ndarray, k: int) -> np.ndarray:
    """ranked [n, N] expert ids, best first; routed [n, k] -> delta* [n] (int64)."""
    ranked = np.asarray(ranked, np.int64)
    routed = np.asarray(routed, np.int64)
    n, N = ranked.shape
    where = np.empty((n, N), np.int64)
    rows = np.arange(n)[:, None]
    where[rows, ranked] = np.arange(N)[None, :]
    deepest = where[rows, routed].max(axis=1)
    return np.maximum(deepest + 1 - k, 0)


def collect_samples(cfg: configs.MoEConfig, layer: int, tokens: int,
                    holdout_seed: int = HOLDOUT_SEED, model_seed: int = 0, streams: int = 64):
    """Run the router and gate kernels on `tokens` held-out tokens of one layer.

    Returns (x [tokens, N] float64: prefetch probabilities in ranked order,
    delta* [tokens] int64).
    """
    import torch
    if not torch.cuda.is_available():
        raise native.ApexLibraryMissing("collecting CDF samples needs the GPU kernels")
    E, k, d = cfg.E, cfg.k, cfg.d
    streams = max(1, min(streams, tokens))
    steps = -(-tokens // streams)
    h_pre, h_post = inputs.hidden_states(cfg, layer, streams, steps, holdout_seed)
    h_pre = h_pre.reshape(-1, d)[:tokens]
    h_post = h_post.reshape(-1, d)[:tokens]
    wg, wpf, bias = inputs.router_weights(cfg, layer, model_seed)
    dev = torch.device("cuda")

    def t(a):
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    n = h_pre.shape[0]
    pf_idx = torch.empty((n, E), dtype=torch.int32, device=dev)
    pf_count = torch.empty((n,), dtype=torch.int32, device=dev)
    pf_prob = torch.empty((n, E), dtype=torch.float32, device=dev)
    route_idx = torch.empty((n, k), dtype=torch.int32, device=dev)
    route_gate = torch.empty((n, k), dtype=torch.float32, device=dev)
    exec_idx = torch.empty_like(route_idx)
    exec_gate = torch.empty_like(route_gate)
    b = None if bias is None else t(bias.astype(np.float32))
    stream = torch.cuda.current_stream().cuda_stream
    # the whole ranked list: static budget N - k with k_max = N
    native.apex_prefetch_route(t(h_pre), t(wpf.view(np.int16)), b, n, d, E, k, E,
                               native.SEL_STATIC, 0.0, E - k, None, None, pf_idx, pf_count,
                               pf_prob, stream)
    native.apex_gate_topk(t(h_post), t(wg.view(np.int16)), b, n, d, E, k, native.MODE_EXACT,
                          None, 0, route_idx, route_gate, exec_idx, exec_gate, None, stream)
    torch.cuda.synchronize()
    ranked = pf_idx.cpu().numpy()
    if not (pf_count.cpu().numpy() == E).all():
        raise native.ApexError(native.APEX_E_INVAL, "full ranking expected from the router")
    prob = pf_prob.cpu().numpy().astype(np.float64)
    x = np.take_along_axis(prob, ranked.astype(np.int64), axis=1)
    return x, delta_star(ranked, route_idx.cpu().numpy(), k)


def _objective(v, x, dstar, n_levels, ridge):
    n, E = x.shape
    w, theta0, steps = v[:E], v[E], v[E + 1:]
    theta = theta0 + np.concatenate([[0.0], np.cumsum(steps)])
    s = x @ w
    a = theta[None, :] - s[:, None]                             # [n, L]
    covered = np.arange(n_levels)[None, :] >= dstar[:, None]
    # cross-entropy of sigmoid(a): -log sigmoid(a) if covered, -log(1 - sigmoid(a)) if not
    loss = np.where(covered, np.logaddexp(0.0, -a), np.logaddexp(0.0, a)).sum() / n
    loss += 0.5 * ridge * (w @ w + theta @ theta)
    resid = 1.0 / (1.0 + np.exp(-a)) - covered                   # d loss / d a, per sample
    g_theta = resid.sum(axis=0) / n + ridge * theta
    g_w = -(x.T @ resid.sum(axis=1)) / n + ridge * w
    # theta_j = theta0 + sum_{1 <= i <= j} steps_i
    from_right = np.cumsum(g_theta[::-1])[::-1]
    grad = np.concatenate([g_w, [from_right[0]], from_right[1:]])
    return loss, grad


def fit_layer(x, dstar, n_levels: int, ridge: float = DEFAULT_RIDGE, max_iter: int = 5000):
    """Fit (w, theta) for one layer; float64 results and the final mean loss."""
    x = np.asarray(x, np.float64)
    dstar = np.asarray(dstar, np.int64)
    if dstar.size == 0 or dstar.min() < 0 or dstar.max() >= n_levels:
        raise ValueError("delta* samples must lie in 0..N-k")
    E = x.shape[1]
    v0 = np.concatenate([np.zeros(E), [-1.0], np.full(n_levels - 1, 0.5)])
    bounds = [(None, None)] * (E + 1) + [(0.0, None)] * (n_levels - 1)
    res = minimize(_objective, v0, args=(x, dstar, n_levels, ridge), jac=True,
                   method="L-BFGS-B", bounds=bounds,
                   options={"maxiter": max_iter, "maxfun": 4 * max_iter, "ftol": 1e-15,
                            "gtol": 1e-11})
    w = res.x[:E]
    theta = res.x[E] + np.concatenate([[0.0], np.cumsum(res.x[E + 1:])])
    return w, theta, float(res.fun)


def fit_model(cfg: configs.MoEConfig, tokens: int = 2048, layers=None,
              ridge: float = DEFAULT_RIDGE, holdout_seed: int = HOLDOUT_SEED,
              model_seed: int = 0):
    """Fit every layer's model on held-out tokens.

    Returns ({layer: (w fp32 [N], theta fp32 [N-k+1])}, report dict).
    """
    layers = range(cfg.L) if layers is None else layers
    t0 = time.perf_counter()
    params, losses, mean_dstar = {}, [], []
    for l in layers:
        x, dstar = collect_samples(cfg, l, tokens, holdout_seed, model_seed)
        w, theta, loss = fit_layer(x, dstar, cfg.E - cfg.k + 1, ridge)
        params[l] = (w.astype(np.float32), theta.astype(np.float32))
        losses.append(loss)
        mean_dstar.append(float(dstar.mean()))
    report = {"tokens_per_layer": tokens, "ridge": ridge, "holdout_seed": holdout_seed,
              "mean_loss": float(np.mean(losses)), "mean_delta_star": float(np.mean(mean_dstar)),
              "fit_s": round(time.perf_counter() - t0, 2)}
    return params, report

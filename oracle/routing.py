"""Oracle: prefetch router, ranked expert list and adaptive prefetch-set selection.

Test infrastructure only (see the package docstring).  Float64 throughout.

Paper passages followed:
* Sec. IV-D, "Prefetch Router Architecture and Placement": the prefetch router is a
  linear layer giving one logit per expert, followed by a softmax.
* Sec. IV-B: the ranked list E = (e_1, ..., e_N), highest predicted score first, and
  the prefetched set K_p^(delta) = {e_1, ..., e_{k+delta}} (Eq. 1).
* Sec. IV-C: the ordinal-logistic coverage model p_delta(x) = sigmoid(theta_delta - w.x)
  (Eq. 8) and the budget rule delta_hat = min{delta : p_delta >= tau} (Eq. 9).
* Cumulative-probability rule of the workload definitions: take experts in ranked
  order until their prefetch probabilities sum to at least tau, clamped to [k, k_max].
* Static over-fetch baseline (Sec. V-A): delta fixed for every token.
* No-Prefetch baseline (Sec. V-A): nothing is prefetched; every routed expert that is
  not already resident is loaded after the gate.

Readings (where the paper is silent): equal scores rank the lower expert id first;
the ordinal model's input x is the prefetch probability vector sorted in descending
order (its length is the number of experts, which matches the parameter count the
overhead analysis of Sec. V-F gives); when no delta satisfies Eq. 9 the whole ranked
list is taken (delta_hat = N - k, which always covers, Eq. 3).
"""
from __future__ import annotations

import math

import numpy as np

from .bf16 import bf16_to_f64

CUMPROB, ORDINAL_CDF, STATIC, NONE = 0, 1, 2, 3


def router_logits(h: np.ndarray, w_bits: np.ndarray, bias=None) -> np.ndarray:
    """z[b, e] = sum_j W[e, j] h[b, j] (+ bias_e), in float64 (Sec. IV-D linear layer)."""
    w = bf16_to_f64(w_bits)
    z = np.asarray(h, dtype=np.float64) @ w.T
    if bias is not None:
        z = z + np.asarray(bias, dtype=np.float64)[None, :]
    return z


def softmax(z: np.ndarray) -> np.ndarray:
    """Row softmax, max-subtracted, float64."""
    z = np.asarray(z, dtype=np.float64)
    m = z.max(axis=-1, keepdims=True)
    p = np.exp(z - m)
    return p / p.sum(axis=-1, keepdims=True)


def rank_experts(z_row) -> list:
    """Ranked list E: expert ids by descending score, lower id first on equal scores."""
    return sorted(range(len(z_row)), key=lambda e: (-float(z_row[e]), e))


def logit(tau: float) -> float:
    if tau <= 0.0:
        return -math.inf
    if tau >= 1.0:
        return math.inf
    return math.log(tau / (1.0 - tau))


def select_cumprob(q_ranked, k: int, k_max: int, tau: float):
    """Smallest m whose ranked prefix mass reaches tau, clamped to [k, k_max].

    With S_j the mass of the first j ranked experts, the clamped m depends only on the
    comparisons S_j >= tau for j = k .. k_max - 1: m = k if S_k >= tau, else the first
    such j, else k_max.  Returns (m, margin), margin = the smallest |S_j - tau| among the
    comparisons that decide m (j from k up to min(m, k_max - 1)); infinite when the clamp
    alone fixes m (k = k_max).
    """
    E = len(q_ranked)
    s = 0.0
    m_star = E
    prefix = []
    for i in range(E):
        s += float(q_ranked[i])
        prefix.append(s)
        if s >= tau:
            m_star = i + 1
            break
    m = min(max(m_star, k), k_max)
    margin = math.inf
    for j in range(k, min(m, k_max - 1) + 1):
        if j > len(prefix):            # the crossing came earlier: S_j >= S_m* >= tau
            s_j = sum(float(q) for q in q_ranked[:j])
        else:
            s_j = prefix[j - 1]
        margin = min(margin, abs(s_j - tau))
    return m, margin


def select_ordinal(q_ranked, cdf_w, cdf_theta, k: int, k_max: int, tau: float):
    """Eq. 8-9: delta_hat = min{delta in 0..N-k : sigmoid(theta_delta - w.x) >= tau}.

    x = the prefetch probabilities in ranked (descending) order.  sigmoid(a) >= tau is
    tested as a >= logit(tau) (sigmoid is increasing).  m = min(k + delta_hat, k_max)
    depends only on the tests for delta = 0 .. k_max - k - 1.  Returns (m, delta_hat,
    margin), margin = the smallest |theta_delta - w.x - logit(tau)| among the tests that
    decide m (delta up to min(delta_hat, k_max - k - 1)).
    """
    E = len(q_ranked)
    s = float(np.dot(np.asarray(cdf_w, dtype=np.float64), np.asarray(q_ranked, dtype=np.float64)))
    thr = logit(tau)
    delta_hat = E - k
    for delta in range(E - k + 1):
        if float(cdf_theta[delta]) - s >= thr:
            delta_hat = delta
            break
    m = min(k + delta_hat, k_max)
    margin = math.inf
    if math.isfinite(thr):
        for delta in range(0, min(delta_hat, k_max - k - 1) + 1):
            margin = min(margin, abs(float(cdf_theta[delta]) - s - thr))
    return m, delta_hat, margin


def select_static(k: int, k_max: int, static_delta: int, E: int) -> int:
    return min(k + static_delta, k_max, E)


def prefetch_route(h_pre, w_pf_bits, b_pf, k, k_max, policy=CUMPROB, tau=0.9,
                   static_delta=0, cdf_w=None, cdf_theta=None):
    """One call of the prefetch stage (Sec. IV-A, step 1) for a batch of tokens.

    Returns a dict with
      pf_idx   int32 [B, k_max]  the prefetched set K_p in ranked order, -1 padded
      pf_count int32 [B]         its size m = k + delta_hat (after the clamp)
      prob     f64 [B, E]        prefetch softmax q_p
      ranked   int32 [B, E]      the full ranked list E
      margin   f64 [B]           smallest decision margin (near-tie accounting)
    """
    h_pre = np.atleast_2d(np.asarray(h_pre))
    z = router_logits(h_pre, w_pf_bits, b_pf)
    q = softmax(z)
    B, E = z.shape
    pf_idx = np.full((B, k_max), -1, np.int32)
    pf_count = np.zeros(B, np.int32)
    ranked = np.zeros((B, E), np.int32)
    margin = np.full(B, math.inf)
    for b in range(B):
        order = rank_experts(z[b])
        ranked[b] = order
        q_ranked = [q[b, e] for e in order]
        if policy == CUMPROB:
            m, mg = select_cumprob(q_ranked, k, k_max, tau)
        elif policy == ORDINAL_CDF:
            m, _, mg = select_ordinal(q_ranked, cdf_w, cdf_theta, k, k_max, tau)
        elif policy == STATIC:
            m, mg = select_static(k, k_max, static_delta, E), math.inf
        elif policy == NONE:
            m, mg = 0, math.inf
        else:
            raise ValueError(f"unknown policy {policy}")
        # ordering and cut of the ranked prefix: logit gaps of adjacent entries
        zs = [z[b, e] for e in order]
        for i in range(min(m, E - 1)):
            mg = min(mg, zs[i] - zs[i + 1])
        pf_idx[b, :m] = order[:m]
        pf_count[b] = m
        margin[b] = mg
    return dict(pf_idx=pf_idx, pf_count=pf_count, prob=q, ranked=ranked, margin=margin,
                logits=z)

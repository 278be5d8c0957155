"""Oracle: original-router top-k and the two execution modes.

Test infrastructure only.  Float64 throughout.

Paper passages followed:
* Sec. III-A: the router computes a probability distribution over the experts and
  selects the top-k; their outputs are combined by a weighted sum.
* Sec. IV-E, correctness-preserving mode: the executed set is exactly the routed set
  K_r (missing experts are fetched, never replaced).
* Sec. IV-E, stall-free mode and Algorithm 1: keep K_r intersected with the available
  set, and replace each missing routed expert by the highest-weight remaining available
  expert under the original router's softmax weights alpha.

Readings: the gates are alpha renormalised over the executed set, so they sum to one;
equal logits rank the lower expert id first; if fewer than k experts are available,
all of them are executed and the unused output positions are -1 with gate 0.

``gate_topk`` computes the stall-free set as the top-k of the available experts by
gate logit.  That this equals Algorithm 1 follows because every routed expert scores
at least as high as every unrouted one, so the routed experts that are available are
the best available ones and Algorithm 1 tops them up with the next best.  The literal
steps of Algorithm 1 are in ``stall_free_algorithm1`` and the tests check the two
against each other and against brute force.
"""
from __future__ import annotations

import math

import numpy as np

from .routing import rank_experts, router_logits, softmax

EXACT, STALL_FREE = 0, 1


def _ordered_pick(z_row, candidates, k):
    """First k of ``candidates`` by (descending logit, ascending id), plus the logit
    gaps that decide that order and cut."""
    order = sorted(candidates, key=lambda e: (-float(z_row[e]), e))
    sel = order[:k]
    margin = math.inf
    for i in range(min(k, len(order) - 1)):
        margin = min(margin, float(z_row[order[i]]) - float(z_row[order[i + 1]]))
    return sel, margin


def gate_topk(h_post, w_g_bits, b_g, k, mode=EXACT, avail=None):
    """Post-attention gate (Sec. III-A / IV-E) for a batch of tokens.

    avail: None (every expert available), bool [E] shared by the batch, or bool [B, E].
    Returns dict with route_idx/route_gate (exact K_r and its renormalised alpha),
    exec_idx/exec_gate (the executed set; equal to the route in EXACT mode), prob
    (alpha) and margin (smallest deciding logit gap, for near-tie accounting).
    """
    h_post = np.atleast_2d(np.asarray(h_post))
    z = router_logits(h_post, w_g_bits, b_g)
    alpha = softmax(z)
    B, E = z.shape
    route_idx = np.full((B, k), -1, np.int32)
    route_gate = np.zeros((B, k))
    exec_idx = np.full((B, k), -1, np.int32)
    exec_gate = np.zeros((B, k))
    margin = np.full(B, math.inf)
    for b in range(B):
        K_r, mg = _ordered_pick(z[b], range(E), k)
        route_idx[b, :k] = K_r
        ssum = sum(alpha[b, e] for e in K_r)
        route_gate[b, :k] = [alpha[b, e] / ssum for e in K_r]
        if mode == EXACT:
            K_x = K_r
        elif mode == STALL_FREE:
            if avail is None:
                A = list(range(E))
            else:
                a = np.asarray(avail)
                row = a[b] if a.ndim == 2 else a
                A = [e for e in range(E) if row[e]]
            K_x, mg2 = _ordered_pick(z[b], A, k)
            mg = min(mg, mg2)
        else:
            raise ValueError(f"unknown mode {mode}")
        margin[b] = mg
        n = len(K_x)
        exec_idx[b, :n] = K_x
        if n:
            ssum = sum(alpha[b, e] for e in K_x)
            exec_gate[b, :n] = [alpha[b, e] / ssum for e in K_x]
    return dict(route_idx=route_idx, route_gate=route_gate, exec_idx=exec_idx,
                exec_gate=exec_gate, prob=alpha, margin=margin, logits=z)


def stall_free_algorithm1(K_r, q_r, K_p):
    """Algorithm 1 (Sec. IV-E) as its steps read, for pinning ``gate_topk``.

    K_r: routed experts; q_r: original-router logits over all N experts; K_p: the
    prefetched (available) experts.  Candidates are ranked by alpha = softmax(q_r),
    equal weights taking the lower id first.  Returns the executed set as a Python set.
    """
    alpha = softmax(np.asarray(q_r, dtype=np.float64)[None, :])[0]
    K_r, K_p = set(K_r), set(K_p)
    if K_r <= K_p:                          # every routed expert is available
        return set(K_r)
    kept = K_r & K_p                        # correctly prefetched routed experts
    missing = K_r - K_p
    candidates = K_p - kept
    ranked = sorted(candidates, key=lambda e: (-alpha[e], e))
    return kept | set(ranked[:len(missing)])

"""Oracle: one MoE-decode step through every layer of a workload.

Test infrastructure only.  Composes the other oracle modules in the order of the
paper's two-stage runtime (Sec. IV-A and IV-D "Runtime Operation"):

  prefetch router on h_pre -> ranked list -> adaptive prefetch set K_p
  -> cache plan (copies of non-resident experts)
  -> original router on h_post -> K_r; executed set by mode (Sec. IV-E)
  -> correctness-preserving misses = K_r minus the resident set
  -> gated SwiGLU experts on h_post, plus the workload's shared experts (Sec. V-A:
     activated for every token, outside the adaptive decision), each with weight 1.

The experts run on x = h_post and y is the MoE output alone (no residual, no norm);
layers are not chained, each layer draws its own hidden-state stream.
"""
from __future__ import annotations

import numpy as np

from paper_2608_11688_amd import inputs

from . import ffn, gating, metrics, routing
from .residency import Residency


class LayerState:
    def __init__(self, cfg, layer, seed=0, policy=routing.CUMPROB, cdf=None, weights="bf16",
                 bits=None):
        """bits: an already drawn {expert: weights} dict of the same layer and seed to use
        (and add to) instead of a new one."""
        self.cfg, self.layer = cfg, layer
        self.wg, self.wpf, self.bias = inputs.router_weights(cfg, layer, seed)
        self.res = Residency(cfg.E, cfg.C)
        self.seed = seed
        self.policy = policy
        self.cdf = cdf if cdf is not None else (None, None)
        self.weights = weights
        self._bits = {} if bits is None else bits

    def expert_bits(self, e):
        if e not in self._bits:
            self._bits[e] = inputs.expert_weights(self.cfg, self.layer, e, self.seed)
        return self._bits[e]

    def shared_bits(self, s):
        key = ("shared", s)
        if key not in self._bits:
            self._bits[key] = inputs.shared_expert_weights(self.cfg, self.layer, s, self.seed)
        return self._bits[key]


def shared_ffn(h_post, n_shared, shared_bits, weights="bf16"):
    """Sum of the shared experts on every token: each with weight 1 (Sec. V-A)."""
    h = np.atleast_2d(np.asarray(h_post, np.float64))
    B = h.shape[0]
    idx = np.tile(np.arange(n_shared), (B, 1))
    return ffn.moe_ffn(h, idx, np.ones((B, n_shared)), shared_bits, weights=weights)


def layer_step(st: LayerState, t, h_pre, h_post, mode, tau, static_delta=0, run_ffn=True):
    cfg = st.cfg
    r = routing.prefetch_route(h_pre, st.wpf, st.bias, cfg.k, cfg.k_max, st.policy, tau,
                               static_delta, st.cdf[0], st.cdf[1])
    B = r["pf_idx"].shape[0]
    pf_lists = [list(r["pf_idx"][b, :r["pf_count"][b]]) for b in range(B)]
    copies = st.res.plan(pf_lists, t)
    R = st.res.resident()
    avail = np.array([e in R for e in range(cfg.E)])
    g = gating.gate_topk(h_post, st.wg, st.bias, cfg.k, mode, avail)
    misses = set()
    if mode == gating.EXACT:
        for b in range(B):
            misses |= set(int(e) for e in g["route_idx"][b]) - R
    y = None
    if run_ffn:
        y = ffn.moe_ffn(h_post, g["exec_idx"], g["exec_gate"], st.expert_bits,
                        weights=st.weights)
        if cfg.shared:
            y = y + shared_ffn(h_post, cfg.shared, st.shared_bits, st.weights)
    m = dict(
        overlap=[metrics.overlap(g["route_idx"][b], pf_lists[b], cfg.k) for b in range(B)],
        coverage=[metrics.full_coverage(g["route_idx"][b], pf_lists[b]) for b in range(B)],
        delta_star=[metrics.delta_star(r["ranked"][b], g["route_idx"][b], cfg.k) for b in range(B)],
        # Eq. 9: delta_hat lies in 0..N-k; the no-prefetch baseline takes no extra experts
        delta_hat=[max(int(r["pf_count"][b]) - cfg.k, 0) for b in range(B)],
        hits=[len(set(int(e) for e in g["route_idx"][b]) & R) / cfg.k for b in range(B)],
        copies=len(copies), misses=len(misses),
    )
    return dict(route=r, gate=g, copies=copies, resident=R, misses=misses, y=y, metrics=m)


def make_states(cfg, layers, seed=0, policy=routing.CUMPROB, cdf=None, weights="bf16",
                bits_from=None):
    """One LayerState per layer (the per-layer routers, cache and expert weights), each
    with an empty cache; bits_from: states of the same layers and seed whose drawn expert
    weights the new states share."""
    return {l: LayerState(cfg, l, seed, policy, None if cdf is None else cdf[l], weights,
                          None if bits_from is None else bits_from[l]._bits)
            for l in layers}


def run(cfg, batch, steps, mode=gating.EXACT, tau=None, seed=0, layers=None, run_ffn=True,
        policy=routing.CUMPROB, static_delta=0, cdf=None, weights="bf16", states=None,
        hidden=None):
    """Replay ``steps`` decode steps of ``batch`` tokens; yields (t, layer, result).

    cdf: {layer: (w, theta)} ordinal-model parameters when policy is ORDINAL_CDF;
    weights: "bf16", "fp8", "mxfp4" or "fp32" expert weights (see ``ffn``);
    states, hidden: the layers' states (``make_states``) and hidden states
    ({layer: (h_pre, h_post)} from the seeded generator) when the caller has drawn them
    already; drawn here otherwise.
    """
    tau = cfg.tau if tau is None else tau
    layers = range(cfg.L) if layers is None else layers
    if states is None:
        states = make_states(cfg, layers, seed, policy, cdf, weights)
    hs = hidden if hidden is not None else {
        l: inputs.hidden_states(cfg, l, batch, steps, seed) for l in layers}
    for t in range(steps):
        for l in layers:
            h_pre, h_post = hs[l][0][t], hs[l][1][t]
            yield t, l, layer_step(states[l], t, h_pre, h_post, mode, tau, static_delta, run_ffn)

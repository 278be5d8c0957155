"""Seeded synthetic inputs for the MoE-decode hot path.

This module only draws random numbers and stores them in the formats the hot path
consumes (fp32 hidden states, bf16 bit patterns for weights).  It holds none of the
method's arithmetic, so both the HIP path and the CPU oracle may take their inputs
from it.

Every tensor comes from its own stream
``Generator(PCG64(SeedSequence([seed, cfg_id, tag, layer, index])))`` so that any
single expert, layer or batch row can be regenerated on its own.

Recipe (the paper evaluates on text benchmarks; these generators stand in for the
hidden states such text would produce, at the models' shapes):

* pre-attention hidden state per (layer, batch row): an AR(1) process
  h_0 ~ N(0, I), h_t = 0.7 h_{t-1} + 0.714 z_t, z_t ~ N(0, I), stored as fp32;
* post-attention hidden state: h_post = h_pre + 0.3 N(0, I), fp32;
* expert weights W1, W3 (I x d) and W2 (d x I): N(0, 0.02^2), rounded to bf16 (RNE);
* gate router W_g = s N(0, 0.02^2) and prefetch router W_pf = W_g + 0.1 s N(0, 0.02^2),
  with s = 2 / (0.02 sqrt(1.09 d)) so that gate logits have standard deviation 2;
* optional per-expert logit bias b ~ N(0, 1) (Zipf-like expert load), shared by both
  routers.
"""
from __future__ import annotations

import numpy as np

from .configs import MoEConfig

# stream tags
TAG_H0, TAG_HZ, TAG_HPOST, TAG_WG, TAG_WPF, TAG_W1, TAG_W3, TAG_W2, TAG_BIAS, TAG_CDF, \
    TAG_MISC, TAG_WQKV, TAG_WO, TAG_KCACHE, TAG_VCACHE = range(1, 16)

AR_RHO = 0.7
AR_SIGMA = 0.714
POST_NOISE = 0.3
W_STD = 0.02
PF_NOISE = 0.1
GATE_LOGIT_STD = 2.0


def rng(seed: int, cfg_id: int, tag: int, layer: int = 0, index: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([int(seed), int(cfg_id), int(tag), int(layer), int(index)])))


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return ((u + (((u >> 16) & 1) + 0x7FFF)) >> 16).astype(np.uint16)


def hidden_states(cfg: MoEConfig, layer: int, rows: int, steps: int, seed: int = 0):
    """(h_pre, h_post), each fp32 [steps, rows, d]; one AR(1) stream per (layer, row)."""
    d = cfg.d
    h_pre = np.empty((steps, rows, d), np.float32)
    h_post = np.empty((steps, rows, d), np.float32)
    for r in range(rows):
        h = rng(seed, cfg.cfg_id, TAG_H0, layer, r).standard_normal(d)
        z = rng(seed, cfg.cfg_id, TAG_HZ, layer, r).standard_normal((steps, d))
        nz = rng(seed, cfg.cfg_id, TAG_HPOST, layer, r).standard_normal((steps, d))
        for t in range(steps):
            if t > 0:
                h = AR_RHO * h + AR_SIGMA * z[t]
            h_pre[t, r] = h
            h_post[t, r] = h_pre[t, r].astype(np.float64) + POST_NOISE * nz[t]
    return h_pre, h_post


def router_scale(d: int) -> float:
    return GATE_LOGIT_STD / (W_STD * np.sqrt((1.0 + POST_NOISE ** 2) * d))


def router_weights(cfg: MoEConfig, layer: int, seed: int = 0):
    """(W_g bits [E,d], W_pf bits [E,d], bias fp32 [E] or None)."""
    s = router_scale(cfg.d)
    base = rng(seed, cfg.cfg_id, TAG_WG, layer).standard_normal((cfg.E, cfg.d)) * (W_STD * s)
    noise = rng(seed, cfg.cfg_id, TAG_WPF, layer).standard_normal((cfg.E, cfg.d))
    w_pf = base + noise * (PF_NOISE * W_STD * s)
    bias = None
    if cfg.bias_skew:
        bias = rng(seed, cfg.cfg_id, TAG_BIAS, layer).standard_normal(cfg.E).astype(np.float32)
    return to_bf16_bits(base.astype(np.float32)), to_bf16_bits(w_pf.astype(np.float32)), bias


def _swiglu_weights(cfg: MoEConfig, layer: int, index: int, I: int, seed: int):
    out = []
    for tag, shape in ((TAG_W1, (I, cfg.d)), (TAG_W3, (I, cfg.d)), (TAG_W2, (cfg.d, I))):
        g = rng(seed, cfg.cfg_id, tag, layer, index)
        w = g.standard_normal(shape, dtype=np.float32)
        w *= np.float32(W_STD)
        out.append(to_bf16_bits(w))
    return tuple(out)


def expert_weights(cfg: MoEConfig, layer: int, expert: int, seed: int = 0):
    """(W1 bits [I,d], W3 bits [I,d], W2 bits [d,I]) of one routed SwiGLU expert."""
    return _swiglu_weights(cfg, layer, expert, cfg.I, seed)


def shared_expert_weights(cfg: MoEConfig, layer: int, s: int, seed: int = 0):
    """The same for shared expert s < cfg.shared (its own streams: index E + s), with
    intermediate size cfg.shared_I."""
    if not 0 <= s < cfg.shared:
        raise IndexError(f"{cfg.name} has {cfg.shared} shared experts")
    return _swiglu_weights(cfg, layer, cfg.E + s, cfg.shared_I, seed)


def attention_weights(cfg: MoEConfig, layer: int, seed: int = 0):
    """(W_qkv bits [(H + 2 G) * hd, d], W_o bits [d, H * hd]) of one decode-attention block.

    Rows of W_qkv: the H query heads, then the G key heads, then the G value heads, hd rows
    each.  Entries ~ N(0, 1/fan_in), so projections of unit-variance states have unit
    variance.
    """
    H, G, hd, d = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d
    w_qkv = rng(seed, cfg.cfg_id, TAG_WQKV, layer).standard_normal(((H + 2 * G) * hd, d),
                                                                   dtype=np.float32)
    w_qkv *= np.float32(1.0 / np.sqrt(d))
    w_o = rng(seed, cfg.cfg_id, TAG_WO, layer).standard_normal((d, H * hd), dtype=np.float32)
    w_o *= np.float32(1.0 / np.sqrt(H * hd))
    return to_bf16_bits(w_qkv), to_bf16_bits(w_o)


def kv_cache(cfg: MoEConfig, layer: int, rows: int, ctx: int, seed: int = 0):
    """(K bits, V bits), each [rows, G, ctx, hd] bf16, entries ~ N(0, 1): the cached keys
    and values of `ctx` earlier tokens of every sequence."""
    G, hd = cfg.n_kv_heads, cfg.head_dim
    k = rng(seed, cfg.cfg_id, TAG_KCACHE, layer).standard_normal((rows, G, ctx, hd),
                                                                 dtype=np.float32)
    v = rng(seed, cfg.cfg_id, TAG_VCACHE, layer).standard_normal((rows, G, ctx, hd),
                                                                 dtype=np.float32)
    return to_bf16_bits(k), to_bf16_bits(v)


def kv_cache_device(torch, cfg: MoEConfig, layer: int, rows: int, ctx: int, seed: int = 0,
                    device="cuda"):
    """Like ``kv_cache`` but drawn on the device (torch's generator, seeded from the same
    stream key), for caches too large to draw on the host: (K, V) int16 tensors holding
    bf16 bits, [rows, G, ctx, hd] each."""
    G, hd = cfg.n_kv_heads, cfg.head_dim
    out = []
    for tag in (TAG_KCACHE, TAG_VCACHE):
        key = np.random.SeedSequence([int(seed), int(cfg.cfg_id), tag, int(layer)])
        g = torch.Generator(device=device)
        g.manual_seed(int(key.generate_state(1, np.uint64)[0] & 0x7FFFFFFFFFFFFFFF))
        x = torch.randn((rows, G, ctx, hd), generator=g, device=device, dtype=torch.float32)
        out.append(x.to(torch.bfloat16).view(torch.int16))
    return tuple(out)


def cdf_params(cfg: MoEConfig, layer: int, seed: int = 0):
    """Random ordinal-model parameters (w fp32 [E], theta fp32 [E-k+1], non-decreasing).

    Used to exercise the ordinal selection rule where no fitted model is at hand.
    """
    g = rng(seed, cfg.cfg_id, TAG_CDF, layer)
    w = g.standard_normal(cfg.E).astype(np.float32)
    theta = np.sort(g.standard_normal(cfg.E - cfg.k + 1) * 2.0 + 1.0).astype(np.float32)
    return w, theta


def uniform(seed: int, tag_index: int, shape, lo=0.0, hi=1.0, cfg_id: int = 999):
    """Generic seeded uniforms for edge-case tests."""
    return rng(seed, cfg_id, TAG_MISC, 0, tag_index).uniform(lo, hi, size=shape)

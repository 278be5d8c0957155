"""Oracle: one decode-attention block, the window the expert prefetch overlaps.

Test infrastructure only (see the package docstring).  Float64.

Paper passages: Sec. IV-A places the prefetch router before each MoE layer's attention
block and issues the expert transfers while attention runs; Eq. 12 bounds the hidden
part of a transfer by the attention time.  The block itself is standard decode
attention, which the paper does not spell out.  Reading taken: grouped-query attention
with the published model shapes.  Per token b:
  [q; k; v] = W_qkv h[b]   (H query heads, then G key heads, then G value heads, hd each);
  the new key and value are stored at position pos of the bf16 cache (rounded to bf16);
  for query head i with key/value head g = i // (H / G):
      a_i = sum_j softmax_j(q_i . K_g[j] / sqrt(hd)) V_g[j]   over j = 0..pos;
  o[b] = W_o [a_0; ...; a_{H-1}].
"""
from __future__ import annotations

import numpy as np

from .bf16 import bf16_to_f64


def round_bf16(x) -> np.ndarray:
    """Nearest bf16 value of each float64 (ties to even), as float64."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                 # x = m * 2^e, |m| in [0.5, 1)
    return np.ldexp(np.rint(m * 256.0), e - 8)   # 8 significant bits; rint ties to even


def to_bf16_bits(x) -> np.ndarray:
    """bf16 bit patterns of float64 values that are already bf16 values."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    return (f.view(np.uint32) >> 16).astype(np.uint16)


def attend(q, K, V, scale):
    """softmax(K q * scale) weighted sum of V.  q [hd], K, V [n, hd]."""
    s = (np.asarray(K, np.float64) @ np.asarray(q, np.float64)) * scale
    p = np.exp(s - s.max())
    return (p / p.sum()) @ np.asarray(V, np.float64)


def attention_block(h, w_qkv_bits, w_o_bits, k_cache_bits, v_cache_bits, H, G, hd, pos):
    """One decode step of the block for a batch.

    h [B, d]; w_qkv bits [(H + 2G) hd, d]; w_o bits [d, H hd]; caches bf16 bits
    [B, G, >= pos, hd] holding the keys and values of positions 0..pos-1.
    Returns dict(o [B, d], k_new, v_new [B, G, hd] as stored (bf16 values)).
    """
    h = np.atleast_2d(np.asarray(h, dtype=np.float64))
    B = h.shape[0]
    qkv = h @ bf16_to_f64(w_qkv_bits).T
    q = qkv[:, :H * hd].reshape(B, H, hd)
    k_new = round_bf16(qkv[:, H * hd:(H + G) * hd].reshape(B, G, hd))
    v_new = round_bf16(qkv[:, (H + G) * hd:].reshape(B, G, hd))
    Kc = bf16_to_f64(k_cache_bits)[:, :, :pos]
    Vc = bf16_to_f64(v_cache_bits)[:, :, :pos]
    group = H // G
    a = np.zeros((B, H, hd))
    scale = 1.0 / np.sqrt(hd)
    for b in range(B):
        for i in range(H):
            g = i // group
            K = np.concatenate([Kc[b, g], k_new[b, g][None]], axis=0)
            V = np.concatenate([Vc[b, g], v_new[b, g][None]], axis=0)
            a[b, i] = attend(q[b, i], K, V, scale)
    o = a.reshape(B, H * hd) @ bf16_to_f64(w_o_bits).T
    return dict(o=o, k_new=k_new, v_new=v_new)

"""Pins of the oracle's decode-attention block (CPU only).

* closed forms of the attention sum: identical keys give the mean of the values; one
  position gives its value; a dominant score gives that position's value;
* torch's scaled_dot_product_attention (float64, keys and values repeated over the
  query groups) on random inputs, through the whole block;
* bf16 rounding of the stored key/value: nearest value, ties to even.
"""
import numpy as np
import pytest

from oracle import attention as att
from oracle.bf16 import bf16_to_f64


def test_identical_keys_average_the_values():
    rng = np.random.default_rng(61)
    K = np.tile(rng.standard_normal(16), (9, 1))
    V = rng.standard_normal((9, 16))
    np.testing.assert_allclose(att.attend(rng.standard_normal(16), K, V, 0.25), V.mean(0),
                               rtol=1e-13)


def test_single_position_and_dominant_score():
    rng = np.random.default_rng(62)
    V = rng.standard_normal((1, 8))
    np.testing.assert_allclose(att.attend(rng.standard_normal(8), rng.standard_normal((1, 8)),
                                          V, 1.0), V[0], rtol=1e-15)
    q = np.zeros(8)
    q[0] = 1.0
    K = np.zeros((5, 8))
    K[3, 0] = 1000.0                     # score 1000 against 0: weight 1 - O(e^-1000)
    V = rng.standard_normal((5, 8))
    np.testing.assert_allclose(att.attend(q, K, V, 1.0), V[3], rtol=1e-14)


def test_round_bf16():
    assert att.round_bf16(1.0) == 1.0
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: ties to even -> 1
    assert att.round_bf16(1.0 + 2.0 ** -8) == 1.0
    assert att.round_bf16(1.0 + 3 * 2.0 ** -8) == 1.0 + 2 * 2.0 ** -7
    assert att.round_bf16(-3.0) == -3.0
    x = np.random.default_rng(63).standard_normal(1000)
    r = att.round_bf16(x)
    assert np.array_equal(bf16_to_f64(att.to_bf16_bits(r)), r)     # exactly bf16 values
    assert np.all(np.abs(r - x) <= np.abs(x) * 2.0 ** -8)


@pytest.mark.parametrize("H,G,hd,pos", [(4, 2, 16, 7), (6, 3, 8, 1), (4, 4, 32, 0),
                                        (8, 2, 16, 33)])
def test_block_matches_torch_sdpa(H, G, hd, pos):
    torch = pytest.importorskip("torch")
    import torch.nn.functional as F
    rng = np.random.default_rng(64 + H + pos)
    B, d = 3, 40

    def bits(a):
        return (np.asarray(a, np.float32).view(np.uint32) >> 16).astype(np.uint16)

    w_qkv = bits(rng.standard_normal(((H + 2 * G) * hd, d)) / np.sqrt(d))
    w_o = bits(rng.standard_normal((d, H * hd)) / np.sqrt(H * hd))
    kc = bits(rng.standard_normal((B, G, pos + 2, hd)))
    vc = bits(rng.standard_normal((B, G, pos + 2, hd)))
    h = rng.standard_normal((B, d))
    got = att.attention_block(h, w_qkv, w_o, kc, vc, H, G, hd, pos)

    T = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    qkv = T(h) @ T(bf16_to_f64(w_qkv)).T
    q = qkv[:, :H * hd].reshape(B, H, 1, hd)
    k_new = T(got["k_new"]).reshape(B, G, 1, hd)
    v_new = T(got["v_new"]).reshape(B, G, 1, hd)
    K = torch.cat([T(bf16_to_f64(kc))[:, :, :pos], k_new], dim=2)
    V = torch.cat([T(bf16_to_f64(vc))[:, :, :pos], v_new], dim=2)
    K = K.repeat_interleave(H // G, dim=1)
    V = V.repeat_interleave(H // G, dim=1)
    a = F.scaled_dot_product_attention(q, K, V)               # [B, H, 1, hd]
    o = a.reshape(B, H * hd) @ T(bf16_to_f64(w_o)).T
    np.testing.assert_allclose(got["o"], o.numpy(), rtol=1e-10, atol=1e-12)
    # the stored key and value are the projections rounded to bf16
    k_exact = qkv[:, H * hd:(H + G) * hd].numpy().reshape(B, G, hd)
    np.testing.assert_array_equal(got["k_new"], att.round_bf16(k_exact))

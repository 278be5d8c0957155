"""Decode attention (apex_attention_decode) against the oracle's block.

The output must match to float32 rounding (max error 1e-4 of max |o|); the key and value
written into the caches must equal the oracle's bf16 rounding of the projections, or
differ by one bf16 step where the float32 and float64 projections straddle a rounding
boundary (counted, at most a few per mille).
"""
import numpy as np
import pytest

from oracle import attention as oatt
from paper_2608_11688_amd import configs, inputs, native

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as t
    return t


def dev(torch, a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).cuda()


def run_case(torch, cfg, B, ctx, layer=0):
    H, G, hd, d = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d
    ctx_max, pos = ctx + 1, ctx
    w_qkv, w_o = inputs.attention_weights(cfg, layer)
    kc, vc = inputs.kv_cache(cfg, layer, B, ctx_max)
    h = inputs.hidden_states(cfg, layer, B, 1)[0][0]
    k_dev, v_dev = dev(torch, kc), dev(torch, vc)
    o = torch.full((B, d), float("nan"), device="cuda")
    ws_bytes = native.apex_attention_workspace_bytes(B, H, G, hd, ctx_max)
    ws = torch.full((ws_bytes,), 0xAB, dtype=torch.uint8, device="cuda")
    native.apex_attention_decode(dev(torch, h), dev(torch, w_qkv), dev(torch, w_o), B, d, H, G, hd,
                                 k_dev, v_dev, ctx_max, pos, o, ws, ws_bytes)
    torch.cuda.synchronize()
    ref = oatt.attention_block(h, w_qkv, w_o, kc, vc, H, G, hd, pos)
    got = o.cpu().numpy().astype(np.float64)
    err = np.abs(got - ref["o"]).max() / np.abs(ref["o"]).max()
    assert err <= 1e-4, err
    # the cache holds the new key and value at pos and is untouched elsewhere
    k_out = k_dev.cpu().numpy().view(np.uint16)
    v_out = v_dev.cpu().numpy().view(np.uint16)
    assert np.array_equal(np.delete(k_out, pos, axis=2), np.delete(kc, pos, axis=2))
    assert np.array_equal(np.delete(v_out, pos, axis=2), np.delete(vc, pos, axis=2))
    off = 0
    for got_bits, want in ((k_out[:, :, pos], ref["k_new"]), (v_out[:, :, pos], ref["v_new"])):
        want_bits = oatt.to_bf16_bits(want)
        steps = np.abs(got_bits.astype(np.int32) - want_bits.astype(np.int32))
        assert steps.max() <= 1
        off += int((steps == 1).sum())
    assert off <= max(2, 0.005 * 2 * B * G * hd), off
    return err, off


@pytest.mark.parametrize("name,B,ctx", [
    ("tiny", 1, 0),                     # nothing cached: attends to the new token only
    ("granite-1b-a400m", 1, 1024),
    ("granite-1b-a400m", 4, 37),        # ragged split boundaries
    ("granite-3b-a800m", 2, 512),       # three query heads per key/value head
    ("olmoe-1b-7b", 1, 2048),           # head size 128, one query head per group
    ("mixtral-8x7b", 1, 1024),          # head size 128, four query heads per group
    ("mixtral-8x7b", 3, 100),
])
def test_attention_matches_oracle(torch, name, B, ctx):
    cfg = configs.CONFIGS[name]
    print(name, B, ctx, run_case(torch, cfg, B, ctx))


def test_attention_eight_heads_per_group(torch):
    cfg = configs.MoEConfig("att_g8", 440, L=1, d=512, E=4, k=1, I=64, C=4, k_max=4, tau=0.9,
                            steps=1, heads=8, kv_heads=1)
    print("g8", run_case(torch, cfg, 2, 300))


def test_attention_rejects_bad_shapes(torch):
    A = 4096
    with pytest.raises(native.ApexError):
        native.apex_attention_decode(A, A, A, 1, 512, 8, 3, 64, A, A, 10, 0, A, A, 1 << 20)
    with pytest.raises(native.ApexError):
        native.apex_attention_decode(A, A, A, 1, 512, 8, 1, 96, A, A, 10, 0, A, A, 1 << 20)
    with pytest.raises(native.ApexError):
        native.apex_attention_decode(A, A, A, 1, 512, 8, 8, 64, A, A, 10, 10, A, A, 1 << 20)

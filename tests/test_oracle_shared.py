"""Pins of the oracle's shared experts (Sec. V-A: DeepSeek's two shared experts run for
every token, outside the adaptive decision), CPU only.

* the shared sum against torch's own SwiGLU in float64 (an independent library);
* a decode layer-step with shared experts equals the same step without them plus that
  sum: the routing, cache and miss decisions do not see the shared experts;
* the shared experts' weights have their own seeded streams and intermediate size.
"""
import dataclasses

import numpy as np
import pytest

from oracle import decode, gating
from oracle.bf16 import bf16_to_f64
from paper_2608_11688_amd import configs, inputs

CFG = configs.MoEConfig("shared_pin", 430, L=1, d=64, E=8, k=2, I=32, C=4, k_max=4, tau=0.9,
                        steps=4, shared=2, I_shared=48)


def torch_shared_sum(h, cfg, layer):
    torch = pytest.importorskip("torch")
    x = torch.from_numpy(np.atleast_2d(np.asarray(h, np.float64)))
    y = torch.zeros_like(x)
    for s in range(cfg.shared):
        w1, w3, w2 = (torch.from_numpy(bf16_to_f64(w))
                      for w in inputs.shared_expert_weights(cfg, layer, s))
        y += torch.nn.functional.silu(x @ w1.T) * (x @ w3.T) @ w2.T
    return y.numpy()


def test_shared_sum_matches_torch():
    h = inputs.hidden_states(CFG, 0, 3, 1)[1][0]
    st = decode.LayerState(CFG, 0)
    got = decode.shared_ffn(h, CFG.shared, st.shared_bits)
    np.testing.assert_allclose(got, torch_shared_sum(h, CFG, 0), rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("mode", [gating.EXACT, gating.STALL_FREE])
def test_step_with_shared_is_step_without_plus_shared_sum(mode):
    plain = dataclasses.replace(CFG, shared=0)
    with_shared = list(decode.run(CFG, 2, 3, mode=mode))
    without = list(decode.run(plain, 2, 3, mode=mode))
    for (t, l, a), (_, _, b) in zip(with_shared, without):
        assert a["copies"] == b["copies"] and a["misses"] == b["misses"]
        assert np.array_equal(a["gate"]["exec_idx"], b["gate"]["exec_idx"])
        h_post = inputs.hidden_states(CFG, l, 2, 3)[1][t]
        np.testing.assert_allclose(a["y"], b["y"] + torch_shared_sum(h_post, CFG, l),
                                   rtol=1e-12, atol=1e-14)


def test_shared_weights_have_their_own_streams():
    w1, w3, w2 = inputs.shared_expert_weights(CFG, 0, 1)
    assert w1.shape == (CFG.I_shared, CFG.d) and w2.shape == (CFG.d, CFG.I_shared)
    other = inputs.shared_expert_weights(CFG, 0, 0)[0]
    assert not np.array_equal(w1, other)
    routed = [inputs.expert_weights(CFG, 0, e)[0][:CFG.I] for e in range(CFG.E)]
    assert all(not np.array_equal(w1[:CFG.I], r) for r in routed)
    with pytest.raises(IndexError):
        inputs.shared_expert_weights(CFG, 0, CFG.shared)

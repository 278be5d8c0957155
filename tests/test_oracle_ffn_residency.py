"""Pins of the oracle's SwiGLU FFN, cache replay, coverage metrics and decode step."""
import math

import numpy as np
import pytest
import torch

from oracle import decode, ffn, gating, metrics, routing
from oracle.bf16 import bf16_to_f64
from oracle.residency import Residency
from paper_2608_11688_amd import configs, inputs
from paper_2608_11688_amd.inputs import to_bf16_bits


def _rand_expert(rng, d, I):
    return tuple(to_bf16_bits(rng.standard_normal(s).astype(np.float32) * 0.1)
                 for s in ((I, d), (I, d), (d, I)))


def test_bf16_widening_known_patterns():
    bits = np.array([0x3F80, 0xBF80, 0x4049, 0x0000, 0x8000, 0x3C00, 0x7F7F], np.uint16)
    want = [1.0, -1.0, 3.140625, 0.0, -0.0, 2.0 ** -7, 3.3895313892515355e38]
    assert list(bf16_to_f64(bits)) == want


def test_silu_closed_forms():
    # silu(0) = 0; silu(ln 3) = (3/4) ln 3 since sigmoid(ln 3) = 3/4; silu(-ln 3) = -(1/4) ln 3
    assert ffn.silu(0.0) == 0.0
    assert abs(ffn.silu(math.log(3)) - 0.75 * math.log(3)) < 1e-15
    assert abs(ffn.silu(-math.log(3)) + 0.25 * math.log(3)) < 1e-15
    assert ffn.silu(-800.0) == 0.0            # no overflow to nan


def test_swiglu_against_torch_float64():
    rng = np.random.default_rng(20)
    d, I = 48, 80
    w1, w3, w2 = (bf16_to_f64(w) for w in _rand_expert(rng, d, I))
    x = rng.standard_normal(d)
    got = ffn.swiglu_expert(x, w1, w3, w2)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))
    ref = t(w2) @ (torch.nn.functional.silu(t(w1) @ t(x)) * (t(w3) @ t(x)))
    assert np.allclose(got, ref.numpy(), rtol=1e-12, atol=1e-14)


def test_swiglu_one_unit_closed_form():
    # d = I = 1 with W1 = 1, W3 = 2, W2 = 0.5 and x = ln 3: y = 0.5 * (3/4 ln3) * (2 ln3)
    x = np.array([math.log(3)])
    y = ffn.swiglu_expert(x, np.array([[1.0]]), np.array([[2.0]]), np.array([[0.5]]))
    assert abs(y[0] - 0.75 * math.log(3) ** 2) < 1e-15


def test_moe_ffn_zero_weights_linearity_and_skip():
    rng = np.random.default_rng(21)
    d, I, E, k, B = 32, 40, 6, 2, 3
    experts = {e: _rand_expert(rng, d, I) for e in range(E)}
    zero = tuple(np.zeros_like(w) for w in experts[0])
    x = rng.standard_normal((B, d))
    idx = np.array([[0, 3], [5, 1], [2, -1]])
    gate = np.array([[0.6, 0.4], [0.3, 0.7], [1.0, 0.0]])
    assert np.all(ffn.moe_ffn(x, idx, gate, lambda e: zero) == 0)
    y1 = ffn.moe_ffn(x, idx, gate, experts.__getitem__)
    y2 = ffn.moe_ffn(x, idx, 2 * gate, experts.__getitem__)
    assert np.allclose(y2, 2 * y1, rtol=1e-14)
    # token 2 runs one expert with gate 1: its row is that expert alone
    w = [bf16_to_f64(a) for a in experts[2]]
    assert np.allclose(y1[2], ffn.swiglu_expert(x[2], *w), rtol=1e-14)
    # a pass that skips expert 3 plus a pass with only expert 3 sum to the full output
    part_a = ffn.moe_ffn(x, idx, gate, experts.__getitem__, skip={3})
    part_b = ffn.moe_ffn(x, idx, gate, experts.__getitem__, skip={0, 1, 2, 4, 5})
    assert np.allclose(part_a + part_b, y1, rtol=1e-13, atol=1e-15)


def test_residency_hand_sequence():
    # E = 5, C = 2; start {0, 1}
    r = Residency(5, 2)
    assert r.plan([[1, 3]], 0) == [(3, 0)]           # 0 is the only resident outside T
    assert r.expert_of_slot == [3, 1]
    assert r.plan([[4]], 1) == [(4, 1)]              # 1 (last use 0) before 3 (0): id order
    assert r.expert_of_slot == [3, 4]
    assert r.plan([[3, 2]], 2) == [(2, 1)]           # 4 evicted, 3 kept
    assert r.expert_of_slot == [3, 2]
    # batch: three tokens want {0,1}, {1,2}, {1,4}; counts 1:3, then best rank 0 beats 2,4
    r2 = Residency(5, 2)
    assert r2.target([[0, 1], [1, 2], [4, 1]]) == [1, 0]


@pytest.mark.parametrize("E,C,B", [(8, 4, 1), (32, 16, 1), (40, 16, 8), (64, 24, 16)])
def test_residency_invariants(E, C, B):
    rng = np.random.default_rng(E + C + B)
    r = Residency(E, C)
    for t in range(80):
        lists = []
        for b in range(B):
            m = int(rng.integers(1, min(C, E) + 1))
            lists.append(list(rng.choice(E, size=m, replace=False)))
        before = r.resident()
        T = r.target(lists)
        copies = r.plan(lists, t)
        after = r.resident()
        assert len(after) == C and len(set(r.expert_of_slot)) == C
        assert set(T) <= after
        assert len(copies) == len(set(T) - before)
        assert set(e for e, _ in copies) == set(T) - before
        if B == 1:
            assert set(lists[0]) <= after
        # evicted experts are the least recently used among the residents outside T
        # (last use of experts outside T is not touched by the step)
        evicted = before - after
        kept_outside = (before & after) - set(T)
        for e in evicted:
            for f in kept_outside:
                assert (r.last_used[e], e) < (r.last_used[f], f)


def test_delta_star_enumeration_matches_rank_positions():
    rng = np.random.default_rng(30)
    for _ in range(200):
        E = int(rng.integers(3, 12))
        k = int(rng.integers(1, E + 1))
        ranked = list(rng.permutation(E))
        K_r = list(rng.choice(E, size=k, replace=False))
        ds = metrics.delta_star(ranked, K_r, k)
        assert ds == max(ranked.index(e) for e in K_r) + 1 - k
        # Eq. 5: full coverage iff delta >= delta*
        for delta in range(E - k + 1):
            assert metrics.full_coverage(K_r, ranked[:k + delta]) == (delta >= ds)
            assert (metrics.overlap(K_r, ranked[:k + delta], k) == 1.0) == (delta >= ds)


def test_decode_step_invariants_tiny():
    cfg = configs.TINY
    for mode in (gating.EXACT, gating.STALL_FREE):
        prev_res = None
        for t, l, out in decode.run(cfg, 1, 6, mode=mode):
            g = out["gate"]
            assert abs(g["exec_gate"][0].sum() - 1) < 1e-12
            R = out["resident"]
            if mode == gating.EXACT:
                assert np.array_equal(g["exec_idx"], g["route_idx"])
                assert out["misses"] == set(int(e) for e in g["route_idx"][0]) - R
            else:
                assert set(int(e) for e in g["exec_idx"][0]) <= R
            assert np.isfinite(out["y"]).all() and out["y"].shape == (1, cfg.d)
            m = out["metrics"]
            assert (m["delta_hat"][0] >= m["delta_star"][0]) == m["coverage"][0]


def test_inputs_are_seeded_and_shaped():
    cfg = configs.TINY
    a = inputs.hidden_states(cfg, 0, 2, 5, seed=3)
    b = inputs.hidden_states(cfg, 0, 2, 5, seed=3)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert a[0].dtype == np.float32 and a[0].shape == (5, 2, cfg.d)
    wg, wpf, bias = inputs.router_weights(cfg, 0)
    assert wg.shape == (cfg.E, cfg.d) and wg.dtype == np.uint16 and bias is None
    w1, w3, w2 = inputs.expert_weights(cfg, 0, 3)
    assert w1.shape == (cfg.I, cfg.d) and w2.shape == (cfg.d, cfg.I)
    # gate logits have standard deviation about 2 (the scaling the workloads ask for)
    h = inputs.hidden_states(configs.GRANITE_1B, 0, 1, 256)[1][:, 0]
    z = routing.router_logits(h, inputs.router_weights(configs.GRANITE_1B, 0)[0])
    assert 1.6 < z.std() < 2.4

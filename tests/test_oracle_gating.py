"""Pins of the oracle's gate top-k and the two execution modes (CPU only)."""
import itertools
import json
import os

import numpy as np
import pytest

from oracle import gating, metrics, routing
from paper_2608_11688_amd.inputs import to_bf16_bits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _identity_gate(z):
    """Weights and input that make the gate logits equal ``z`` exactly (bf16 values)."""
    z = np.asarray(z, np.float32)
    E = len(z)
    W = np.eye(E, dtype=np.float32)
    return to_bf16_bits(W), z[None, :]


def _brute_topk_subset(z, k, allowed):
    best, best_val = None, None
    for c in itertools.combinations(sorted(allowed), min(k, len(allowed))):
        v = sum(z[e] for e in c)
        if best_val is None or v > best_val:
            best, best_val = set(c), v
    return best


@pytest.mark.parametrize("E,k", [(8, 2), (8, 4), (6, 3), (5, 1)])
def test_exact_topk_is_best_k_subset_and_gates_renormalise(E, k):
    rng = np.random.default_rng(10 + E * 7 + k)
    for _ in range(40):
        z = rng.standard_normal(E) * 2
        W, h = _identity_gate(z)
        g = gating.gate_topk(h, W, None, k, gating.EXACT)
        zz = g["logits"][0]
        assert set(g["route_idx"][0]) == _brute_topk_subset(zz, k, range(E))
        assert np.array_equal(g["route_idx"], g["exec_idx"])
        assert abs(g["route_gate"][0].sum() - 1) < 1e-14
        alpha = g["prob"][0]
        ratio = g["route_gate"][0] / alpha[g["route_idx"][0]]
        assert np.allclose(ratio, ratio[0], rtol=1e-13)
        # route order is descending logit
        assert list(g["route_idx"][0]) == routing.rank_experts(zz)[:k]


@pytest.mark.parametrize("E,k", [(8, 2), (8, 4), (7, 3), (6, 5)])
def test_stall_free_equals_algorithm1_and_brute_force(E, k):
    rng = np.random.default_rng(100 + E * 7 + k)
    for _ in range(150):
        z = rng.standard_normal(E) * 2
        W, h = _identity_gate(z)
        na = int(rng.integers(k, E + 1))
        A = sorted(rng.choice(E, size=na, replace=False).tolist())
        avail = np.zeros(E, bool)
        avail[A] = True
        g = gating.gate_topk(h, W, None, k, gating.STALL_FREE, avail)
        zz = g["logits"][0]
        got = set(int(e) for e in g["exec_idx"][0] if e >= 0)
        K_r = set(int(e) for e in g["route_idx"][0])
        assert got == gating.stall_free_algorithm1(K_r, zz, A)
        assert got == _brute_topk_subset(zz, k, A)
        assert got <= set(A)
        assert abs(g["exec_gate"][0].sum() - 1) < 1e-14
        if K_r <= set(A):                     # Algorithm 1, all routed experts available
            assert list(g["exec_idx"][0]) == list(g["route_idx"][0])


def test_stall_free_with_everything_available_equals_exact():
    rng = np.random.default_rng(11)
    E, d, k = 16, 64, 4
    W = to_bf16_bits(rng.standard_normal((E, d)).astype(np.float32))
    h = rng.standard_normal((6, d)).astype(np.float32)
    ex = gating.gate_topk(h, W, None, k, gating.EXACT)
    sf = gating.gate_topk(h, W, None, k, gating.STALL_FREE, np.ones(E, bool))
    for key in ("exec_idx", "exec_gate", "route_idx", "route_gate"):
        assert np.array_equal(ex[key], sf[key])


def test_stall_free_fewer_available_than_k_and_per_token_masks():
    z = np.array([0.5, 2.0, -1.0, 1.0, 0.0])
    W, h = _identity_gate(z)
    avail = np.array([False, False, True, True, False])
    g = gating.gate_topk(h, W, None, 3, gating.STALL_FREE, avail)
    assert list(g["exec_idx"][0]) == [3, 2, -1]
    assert g["exec_gate"][0][2] == 0.0 and abs(g["exec_gate"][0][:2].sum() - 1) < 1e-15
    none = gating.gate_topk(h, W, None, 2, gating.STALL_FREE, np.zeros(5, bool))
    assert (none["exec_idx"] == -1).all() and (none["exec_gate"] == 0).all()
    # a [B, E] mask applies per token
    h2 = np.vstack([h, h])
    m2 = np.array([[1, 1, 1, 1, 1], [0, 0, 1, 1, 1]], bool)
    g2 = gating.gate_topk(h2, W, None, 2, gating.STALL_FREE, m2)
    assert list(g2["exec_idx"][0]) == [1, 3] and list(g2["exec_idx"][1]) == [3, 4]


def test_equal_logits_take_lower_id():
    W, h = _identity_gate([1.0, 2.0, 2.0, 2.0, 0.0])
    g = gating.gate_topk(h, W, None, 2, gating.EXACT)
    assert list(g["route_idx"][0]) == [1, 2]


def test_golden_worked_example_modes():
    g = json.load(open(os.path.join(GOLDEN, "worked_example_n8k4.json")))
    k = g["k"]
    zg = np.array(g["gate_logits"])
    W, h = _identity_gate(zg)
    ex = gating.gate_topk(h, W, None, k, gating.EXACT)
    assert list(ex["route_idx"][0]) == g["K_r"]
    for e, gate in g["exact_gates"].items():
        j = list(ex["route_idx"][0]).index(int(e))
        assert abs(ex["route_gate"][0][j] - gate) < g["gate_tol"]
    ranked = g["ranked"]
    assert metrics.delta_star(ranked, g["K_r"], k) == g["delta_star"]
    for delta, want in g["stall_free_exec_at_delta"].items():
        K_p = ranked[:k + int(delta)]
        avail = np.zeros(g["N"], bool)
        avail[K_p] = True
        sf = gating.gate_topk(h, W, None, k, gating.STALL_FREE, avail)
        assert set(sf["exec_idx"][0]) == set(want)
        assert gating.stall_free_algorithm1(g["K_r"], zg, K_p) == set(want)
        assert metrics.overlap(g["K_r"], K_p, k) == g["overlap_at_delta"][delta]

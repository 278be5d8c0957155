"""Pins of the oracle's prefetch router and selection rules (CPU only).

Each check compares the oracle with something other than its own formula: special
cases with a closed form, brute force over subsets, a library routine, invariants the
paper states, or the hand-worked fixture under tests/golden/.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import scipy.special

from oracle import routing
from paper_2608_11688_amd import configs, inputs
from paper_2608_11688_amd.inputs import to_bf16_bits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _bits(a):
    return to_bf16_bits(np.asarray(a, np.float32))


def test_logits_identity_rows_select_coordinates():
    # W = rows of the identity: z_e = h[col_e] exactly, plus the bias.
    rng = np.random.default_rng(1)
    d, E = 16, 5
    cols = [3, 0, 15, 7, 7]
    W = np.zeros((E, d), np.float32)
    for e, c in enumerate(cols):
        W[e, c] = 1.0
    h = rng.standard_normal((3, d)).astype(np.float32)
    bias = np.array([0.5, -1.0, 0.0, 2.0, 0.25], np.float32)
    z = routing.router_logits(h, _bits(W), bias)
    assert z.shape == (3, E)
    for b in range(3):
        for e, c in enumerate(cols):
            assert z[b, e] == float(h[b, c]) + float(bias[e])


def test_logits_scaled_one_hot_and_row_permutation():
    # a single nonzero weight 2^-3 at (e, e+1): z_e = h[e+1] / 8 exactly; permuting the
    # rows of W permutes the logits.
    d, E = 12, 6
    W = np.zeros((E, d), np.float32)
    for e in range(E):
        W[e, e + 1] = 0.125
    h = np.arange(d, dtype=np.float32)[None, :] - 4.0
    z = routing.router_logits(h, _bits(W))
    assert np.array_equal(z[0], (np.arange(1, E + 1) - 4.0) / 8.0)
    perm = [4, 2, 0, 5, 1, 3]
    zp = routing.router_logits(h, _bits(W[perm]))
    assert np.array_equal(zp[0], z[0][perm])


def test_softmax_closed_forms():
    # two experts: q_0 = logistic(z_0 - z_1); equal logits: uniform
    z = np.array([[0.7, -1.3]])
    q = routing.softmax(z)
    assert abs(q[0, 0] - scipy.special.expit(2.0)) < 1e-15
    assert np.allclose(routing.softmax(np.full((1, 7), 3.5)), 1 / 7, atol=0, rtol=1e-15)
    # shift invariance and normalisation on random rows
    rng = np.random.default_rng(2)
    zz = rng.standard_normal((5, 11)) * 4
    assert np.allclose(routing.softmax(zz), routing.softmax(zz + 123.0), rtol=1e-12)
    assert np.allclose(routing.softmax(zz).sum(-1), 1.0, rtol=1e-15)
    assert np.allclose(routing.softmax(zz), scipy.special.softmax(zz, axis=-1), rtol=1e-12)


def test_rank_matches_stable_argsort_and_breaks_ties_by_id():
    rng = np.random.default_rng(3)
    for _ in range(50):
        z = np.round(rng.standard_normal(13), 1)        # rounding makes ties common
        assert routing.rank_experts(z) == list(np.argsort(-z, kind="stable"))
    assert routing.rank_experts([1.0, 2.0, 2.0, 1.0]) == [1, 2, 0, 3]


def _brute_min_mass_subset(q, tau):
    E = len(q)
    for size in range(1, E + 1):
        if any(sum(q[i] for i in c) >= tau for c in itertools.combinations(range(E), size)):
            return size
    return E


@pytest.mark.parametrize("E,k,k_max", [(8, 2, 4), (6, 1, 6), (7, 3, 5), (5, 2, 5)])
def test_cumprob_equals_smallest_subset_reaching_tau(E, k, k_max):
    rng = np.random.default_rng(E * 100 + k)
    for trial in range(60):
        z = rng.standard_normal(E) * 2
        q = routing.softmax(z[None])[0]
        tau = float(rng.uniform(0.3, 0.99))
        ranked = routing.rank_experts(z)
        m, margin = routing.select_cumprob([q[e] for e in ranked], k, k_max, tau)
        if margin < 1e-9:
            continue
        m_star = _brute_min_mass_subset(q, tau)
        assert m == min(max(m_star, k), k_max)


def test_cumprob_edges_and_nesting():
    q = [0.5, 0.3, 0.15, 0.05]
    assert routing.select_cumprob(q, 1, 4, 0.0)[0] == 1
    assert routing.select_cumprob(q, 2, 4, 0.0)[0] == 2       # clamp up to k
    assert routing.select_cumprob(q, 1, 4, 1.0 + 1e-12)[0] == 4   # tau unreachable -> all
    assert routing.select_cumprob(q, 1, 3, 1.0 + 1e-12)[0] == 3   # then clamp to k_max
    ms = [routing.select_cumprob(q, 1, 4, t)[0] for t in np.linspace(0.01, 0.999, 40)]
    assert ms == sorted(ms)


def test_ordinal_closed_form_count_and_scipy_sigmoid():
    # with non-decreasing cut-points the failing deltas form a prefix, so
    # delta_hat = #{delta : theta_delta - s < logit(tau)} (capped at N-k)
    rng = np.random.default_rng(5)
    E, k = 9, 3
    for trial in range(200):
        z = rng.standard_normal(E) * 2
        q = routing.softmax(z[None])[0]
        qr = [q[e] for e in routing.rank_experts(z)]
        w = rng.standard_normal(E)
        theta = np.sort(rng.standard_normal(E - k + 1) * 2)
        tau = float(rng.uniform(0.05, 0.98))
        m, dh, margin = routing.select_ordinal(qr, w, theta, k, E, tau)
        s = float(np.dot(w, qr))
        thr = math.log(tau / (1 - tau))
        if margin < 1e-9:
            continue
        count = int(np.sum(theta - s < thr))
        assert dh == min(count, E - k)
        # the same decision read with a library sigmoid
        ok = [d for d in range(E - k + 1) if scipy.special.expit(theta[d] - s) >= tau]
        assert dh == (ok[0] if ok else E - k)
        assert m == k + dh


def test_ordinal_zero_weight_is_token_independent_and_monotone_in_tau():
    E, k = 8, 2
    theta = np.linspace(-2, 3, E - k + 1)
    rng = np.random.default_rng(6)
    outs = set()
    for _ in range(20):
        z = rng.standard_normal(E)
        q = routing.softmax(z[None])[0]
        outs.add(routing.select_ordinal(sorted(q, reverse=True), np.zeros(E), theta, k, E, 0.8)[1])
    assert len(outs) == 1
    q = routing.softmax(rng.standard_normal((1, E)))[0]
    w = rng.standard_normal(E)
    dh = [routing.select_ordinal(sorted(q, reverse=True), w, theta, k, E, t)[1]
          for t in np.linspace(0.01, 0.99, 50)]
    assert dh == sorted(dh)
    # no delta reaches tau: take the whole list (delta_hat = N - k), then clamp
    assert routing.select_ordinal(q, w, np.full(E - k + 1, -50.0), k, E, 0.9)[1] == E - k
    assert routing.select_ordinal(q, w, np.full(E - k + 1, -50.0), k, 5, 0.9)[0] == 5


def test_prefetch_route_full_list_and_static():
    rng = np.random.default_rng(7)
    E, d, k = 8, 32, 2
    W = _bits(rng.standard_normal((E, d)).astype(np.float32))
    h = rng.standard_normal((4, d)).astype(np.float32)
    r = routing.prefetch_route(h, W, None, k, E, routing.CUMPROB, 1.0 + 1e-9)
    assert (r["pf_count"] == E).all()
    for b in range(4):
        assert sorted(r["pf_idx"][b]) == list(range(E))
        assert list(r["pf_idx"][b]) == list(r["ranked"][b])
    r = routing.prefetch_route(h, W, None, k, 5, routing.STATIC, 0.9, static_delta=2)
    assert (r["pf_count"] == 4).all()
    assert (r["pf_idx"][:, 4:] == -1).all()
    assert (r["pf_idx"][:, :4] == r["ranked"][:, :4]).all()


def test_golden_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "worked_example_n8k4.json")))
    zp = np.array(g["prefetch_logits"])
    assert routing.rank_experts(zp) == g["ranked"]
    q = routing.softmax(zp[None])[0]
    qr = [q[e] for e in g["ranked"]]
    for tau, m_star in g["cumprob_m_star"].items():
        assert routing.select_cumprob(qr, 1, 8, float(tau))[0] == m_star


def test_overhead_table_parameter_counts():
    # The printed totals follow from a d x N router plus an ordinal model whose weight
    # vector has one entry per expert (the length select_ordinal takes, matching the
    # ranked probability vector) and N-k+1 cut-points; a weight vector over the d
    # hidden units would not reproduce them.
    g = json.load(open(os.path.join(GOLDEN, "overhead_params.json")))
    for row in g["rows"]:
        d, N, k, L = row["d"], row["N"], row["k"], row["layers"]
        q = routing.softmax(np.zeros((1, N)))[0]
        routing.select_ordinal(q, np.zeros(N), np.zeros(N - k + 1), k, N, 0.9)
        per_expert_w = L * (d * N + N + (N - k + 1))
        per_hidden_w = L * (d * N + d + (N - k + 1))
        assert round(per_expert_w / 1e6, 2) == row["printed_millions"]
        assert round(per_hidden_w / 1e6, 2) != row["printed_millions"]


def test_phi_and_deepseek_shapes_follow_the_overhead_table():
    # the Phi-7B and DeepSeek-16B workloads take d, N, k and the MoE layer count of the
    # overhead table's rows, and I from the total and active counts in the model names
    g = {r["model"]: r for r in json.load(open(os.path.join(GOLDEN, "overhead_params.json")))["rows"]}
    for cfg, row, total, active in ((configs.PHI_7B, g["Phi-7B"], 7.0e9, 2.4e9),
                                    (configs.DEEPSEEK_16B, g["DeepSeek-16B"], 16.0e9, 2.4e9)):
        assert (cfg.d, cfg.E, cfg.k, cfg.L) == (row["d"], row["N"], row["k"], row["layers"])
        I = (total - active) / (cfg.L * (cfg.E - cfg.k) * 3 * cfg.d)
        assert cfg.I == 64 * round(I / 64)
    assert configs.DEEPSEEK_16B.shared == 2 and configs.PHI_7B.shared == 0


def test_no_prefetch_policy_selects_nothing():
    cfg = configs.GRANITE_1B
    h = inputs.hidden_states(cfg, 0, 4, 1)[0][0]
    wg, wpf, bias = inputs.router_weights(cfg, 0)
    r = routing.prefetch_route(h, wpf, bias, cfg.k, cfg.k_max, routing.NONE)
    assert (r["pf_count"] == 0).all() and (r["pf_idx"] == -1).all()
    # the ranked list is still reported
    assert sorted(r["ranked"][0].tolist()) == list(range(cfg.E))


def test_no_prefetch_decode_keeps_the_initial_cache():
    from oracle import decode, gating
    cfg = configs.TINY
    seen = []
    for t, l, out in decode.run(cfg, 1, 12, mode=gating.EXACT, policy=routing.NONE,
                                run_ffn=False):
        assert out["copies"] == []
        assert sorted(out["resident"]) == list(range(cfg.C))
        routed = set(int(e) for e in out["gate"]["route_idx"][0])
        assert sorted(out["misses"]) == sorted(routed - set(range(cfg.C)))
        # nothing prefetched: no overlap, no extra experts (delta_hat >= 0, Eq. 9)
        assert out["metrics"]["overlap"] == [0.0] and out["metrics"]["delta_hat"] == [0]
        seen.append(len(out["misses"]))
    assert sum(seen) > 0

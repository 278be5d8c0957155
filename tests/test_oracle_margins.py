"""Pins of the oracle's decision margins (CPU only).

The GPU parity tests excuse an index-set mismatch only where the oracle reports a
deciding margin below 1e-5 (a near tie).  These tests fix what those margins are
without going through the oracle's own formulas:
* hand-made inputs whose margin is known by construction (an exact logit tie gives 0, a
  planted logit gap gives that gap, a prefix sum planted at tau +- eps gives eps);
* comparisons the clamp to [k, k_max] makes irrelevant are not counted;
* brute force: every perturbation of the deciding quantity smaller than the margin
  leaves the decision unchanged, and one just larger than the margin changes it.
"""
import math

import numpy as np
import pytest

from oracle import gating, routing
from paper_2608_11688_amd.inputs import to_bf16_bits


def identity_router(E, d):
    """bf16 bits of W = the first E rows of the d x d identity: z = h[:E] exactly."""
    W = np.zeros((E, d), np.float32)
    W[np.arange(E), np.arange(E)] = 1.0
    return to_bf16_bits(W)


def h_with(z, d, dtype=np.float32):
    h = np.zeros((1, d), dtype)
    h[0, :len(z)] = z
    return h


# ----------------------------------------------------------------- prefetch router
def test_prefetch_exact_tie_at_the_cut_has_margin_zero():
    # STATIC m = 3: experts 4 and 6 share the third-largest logit
    z = [0.0, 1.0, 3.0, -1.0, 2.0, 0.5, 2.0, -2.0]
    r = routing.prefetch_route(h_with(z, 16), identity_router(8, 16), None, 2, 4,
                               routing.STATIC, 0.9, static_delta=1)
    assert r["pf_count"][0] == 3
    assert list(r["pf_idx"][0, :3]) == [2, 4, 6]          # lower id first on the tie
    assert r["margin"][0] == 0.0


def test_prefetch_planted_gap_is_the_margin():
    # STATIC m = 3 over logits 4, 3, 2.75, 0.5, ...: the gaps that decide the ranked
    # prefix and its cut are 1, 0.25 and 2.25, so the margin is 0.25
    z = [0.5, 2.75, -3.0, 4.0, 3.0, 0.25]
    r = routing.prefetch_route(h_with(z, 8), identity_router(6, 8), None, 2, 5,
                               routing.STATIC, 0.9, static_delta=1)
    assert list(r["pf_idx"][0, :3]) == [3, 4, 1]
    assert r["margin"][0] == 0.25
    # the gaps past the cut do not count: 0.5 vs 0.25 (0.25 apart) sits below it
    z2 = [0.5, 2.0, -3.0, 4.0, 3.0, 0.4375]
    r2 = routing.prefetch_route(h_with(z2, 8), identity_router(6, 8), None, 2, 5,
                                routing.STATIC, 0.9, static_delta=1)
    assert r2["margin"][0] == 1.0


Q_BINARY = [0.5, 0.25, 0.125, 0.0625, 0.03125, 0.03125]   # prefix sums exact in fp64


@pytest.mark.parametrize("tau,k,k_max,m,margin", [
    # crossing inside the window [k, k_max - 1]: the margin is the distance eps
    (0.875 + 1e-6, 2, 4, 4, 1e-6),            # S_3 just below tau: m = 4
    (0.875 - 1e-6, 2, 4, 3, 1e-6),            # S_3 just above tau: m = 3
    (0.75 + 3e-6, 2, 5, 3, 3e-6),             # S_2 just below tau
    # the clamp decides: a crossing outside the window changes nothing
    (0.5 + 3e-6, 2, 4, 2, 0.25 - 3e-6),       # S_1 near tau, but m >= k = 2 anyway
    (0.9375 + 2e-6, 2, 4, 4, 0.0625 + 2e-6),  # S_4 near tau, but m <= k_max = 4 anyway
    (0.875 + 1e-6, 3, 3, 3, math.inf),        # k = k_max: tau decides nothing
])
def test_cumprob_margin_planted_at_tau(tau, k, k_max, m, margin):
    got_m, got_margin = routing.select_cumprob(Q_BINARY, k, k_max, tau)
    assert got_m == m
    if math.isinf(margin):
        assert math.isinf(got_margin)
    else:
        assert got_margin == pytest.approx(margin, rel=1e-9, abs=1e-15)


def cumprob_m(q, k, k_max, tau):
    """Brute force: the smallest m in [k, k_max] whose prefix mass reaches tau."""
    for m in range(k, k_max):
        if sum(q[:m]) >= tau:
            return m
    return k_max


def test_cumprob_margin_is_the_distance_to_a_changed_decision():
    rng = np.random.default_rng(7)
    for trial in range(400):
        E = int(rng.integers(3, 12))
        k = int(rng.integers(1, E))
        k_max = int(rng.integers(k, E + 1))
        q = np.sort(rng.dirichlet(np.full(E, 0.7)))[::-1]
        tau = float(rng.uniform(0.3, 0.999))
        m, margin = routing.select_cumprob(list(q), k, k_max, tau)
        assert m == cumprob_m(list(q), k, k_max, tau)
        if math.isinf(margin):
            assert k == k_max
            continue
        for f in (-0.999, -0.5, 0.5, 0.999):
            assert cumprob_m(list(q), k, k_max, tau + f * margin) == m, trial
        assert any(cumprob_m(list(q), k, k_max, tau + f * margin * (1 + 1e-9)) != m
                   for f in (-1.0, 1.0)), trial


@pytest.mark.parametrize("eps,k_max,m,margin", [
    (1e-6, 6, 4, 1e-6),     # theta_1 - s just below logit(tau): delta_hat = 2
    (-1e-6, 6, 3, 1e-6),    # just above: delta_hat = 1
    (1e-6, 3, 3, 0.5 + 1e-6),  # k_max = k + 1: only delta = 0 decides m (|0.5 - logit tau|)
])
def test_ordinal_margin_planted_at_the_threshold(eps, k_max, m, margin):
    # w = 0, so s = 0 and theta_delta itself is compared with logit(tau) = 1 + eps
    k, E = 2, 8
    theta = np.array([0.5, 1.0, 2.0, 3.0, 4.0, 5.0, 6.0])
    tau = 1.0 / (1.0 + math.exp(-(1.0 + eps)))
    got_m, _, got_margin = routing.select_ordinal(np.full(E, 1.0 / E), np.zeros(E), theta, k,
                                                  k_max, tau)
    assert got_m == m
    assert got_margin == pytest.approx(margin, rel=1e-6, abs=1e-12)


def ordinal_m(a, thr, k, k_max):
    for delta in range(len(a)):
        if a[delta] >= thr:
            return min(k + delta, k_max)
    return min(k + len(a) - 1, k_max)


def test_ordinal_margin_is_the_distance_to_a_changed_decision():
    rng = np.random.default_rng(8)
    for trial in range(400):
        E = int(rng.integers(3, 12))
        k = int(rng.integers(1, E))
        k_max = int(rng.integers(k, E + 1))
        q = np.sort(rng.dirichlet(np.ones(E)))[::-1]
        w = rng.standard_normal(E)
        theta = rng.normal(1.0, 2.0, E - k + 1)
        tau = float(rng.uniform(0.2, 0.95))
        m, _, margin = routing.select_ordinal(q, w, theta, k, k_max, tau)
        a = theta - float(w @ q)
        thr = math.log(tau / (1 - tau))
        assert m == ordinal_m(a, thr, k, k_max)
        if math.isinf(margin):
            assert k == k_max
            continue
        # shifting every theta by c moves each test by c
        for f in (-0.999, -0.5, 0.5, 0.999):
            assert ordinal_m(a + f * margin, thr, k, k_max) == m, trial
        assert any(ordinal_m(a + f * margin * (1 + 1e-9), thr, k, k_max) != m
                   for f in (-1.0, 1.0)), trial


# ----------------------------------------------------------------- gate
def test_gate_exact_tie_and_planted_gap():
    E, d = 6, 8
    W = identity_router(E, d)
    tie = gating.gate_topk(h_with([1.0, 3.0, 2.0, 2.0, 0.0, -1.0], d), W, None, 3)
    assert list(tie["route_idx"][0]) == [1, 2, 3] and tie["margin"][0] == 0.0
    # cut between 2.5 and 1.75 (0.75); order inside the top-3: 1 and 0.5
    gap = gating.gate_topk(h_with([2.5, 4.0, 3.0, 1.75, 0.0, -1.0], d), W, None, 3)
    assert list(gap["route_idx"][0]) == [1, 2, 0] and gap["margin"][0] == 0.5
    gap2 = gating.gate_topk(h_with([2.25, 4.0, 3.0, 2.0, 0.0, -1.0], d), W, None, 3)
    assert gap2["margin"][0] == 0.25


def test_stall_free_masked_cut_gap():
    # unmasked top-2 {0, 1} with gaps of 2; among the available {2, 3, 5} the cut
    # between 4 and 3.75 is 0.25: the smaller one decides
    E, d = 6, 8
    z = [8.0, 6.0, 4.0, 3.75, 0.0, -2.0]
    avail = np.array([0, 0, 1, 1, 0, 1], bool)
    g = gating.gate_topk(h_with(z, d), identity_router(E, d), None, 2, gating.STALL_FREE,
                         avail)
    assert list(g["route_idx"][0]) == [0, 1]
    assert list(g["exec_idx"][0]) == [2, 3]
    assert g["margin"][0] == 0.25
    exact = gating.gate_topk(h_with(z, d), identity_router(E, d), None, 2)
    assert exact["margin"][0] == 2.0


def test_gate_margin_is_the_distance_to_a_changed_decision():
    # no perturbation of the logits by less than half the margin each changes the
    # ordered sets; moving the closest deciding pair together by just over half the
    # margin each does
    rng = np.random.default_rng(9)
    E, d = 10, 16
    W = identity_router(E, d)
    for trial in range(200):
        k = int(rng.integers(1, E))
        z = rng.standard_normal(E).astype(np.float32)
        mode = int(rng.integers(0, 2))
        avail = rng.random(E) < 0.6
        g = gating.gate_topk(h_with(z, d), W, None, k, mode, avail)
        margin = g["margin"][0]
        zz = z.astype(np.float64)
        for _ in range(5):
            dz = rng.uniform(-0.499, 0.499, E) * margin
            p = gating.gate_topk(h_with(zz + dz, d, np.float64), W, None, k, mode, avail)
            assert np.array_equal(p["route_idx"], g["route_idx"]), trial
            assert np.array_equal(p["exec_idx"], g["exec_idx"]), trial
        changed = False
        order = sorted(range(E), key=lambda e: (-zz[e], e))
        pairs = list(zip(order, order[1:]))
        if mode == gating.STALL_FREE:
            av = [e for e in order if avail[e]]
            pairs += list(zip(av, av[1:]))
        for hi, lo in pairs:
            if abs((zz[hi] - zz[lo]) - margin) > 1e-12:
                continue
            dz = np.zeros(E)
            dz[hi] -= 0.5 * margin * (1 + 1e-6) + 1e-12
            dz[lo] += 0.5 * margin * (1 + 1e-6) + 1e-12
            p = gating.gate_topk(h_with(zz + dz, d, np.float64), W, None, k, mode, avail)
            changed |= not (np.array_equal(p["route_idx"], g["route_idx"]) and
                            np.array_equal(p["exec_idx"], g["exec_idx"]))
        assert changed, trial

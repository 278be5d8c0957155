"""GPU parity of each entry point against the oracle, through the C ABI.

Inputs come from the seeded generators; the oracle computes the expected values on
the CPU in float64.  Index sets must match exactly except at near ties (counted);
FFN outputs within the tolerance stated in tests/parity.py.
"""
import os

import numpy as np
import pytest

from oracle import ffn as offn
from oracle import gating, routing
from oracle.residency import Residency
from paper_2608_11688_amd import configs, inputs, native
from tests.ffn_plans import PLAN_CASES
from tests.parity import TieLedger, ffn_close

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    native.lib()
    return t


def shape(name, cfg_id, d, E, k, I=64, C=None, k_max=None, bias=False):
    return configs.MoEConfig(name, cfg_id, L=1, d=d, E=E, k=k, I=I, C=C or E,
                             k_max=k_max or E, tau=0.9, steps=64, bias_skew=bias)


def dev(torch, a, dtype=None):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).cuda()


def tokens(cfg, n, which=0):
    h_pre, h_post = inputs.hidden_states(cfg, 0, 1, n)
    return (h_pre if which == 0 else h_post)[:, 0, :]


# --------------------------------------------------------------------------- route
def gpu_route(torch, h, wpf, bias, k, k_max, policy, tau, sd=0, cdf=(None, None),
              out_host=False):
    B, d = h.shape
    E = wpf.shape[0]
    kw = dict(pin_memory=True) if out_host else dict(device="cuda")
    pf_idx = torch.full((B, k_max), -7, dtype=torch.int32, **kw)
    pf_count = torch.full((B,), -7, dtype=torch.int32, **kw)
    prob = torch.full((B, E), -1.0, dtype=torch.float32, device="cuda")
    cw = None if cdf[0] is None else dev(torch, np.asarray(cdf[0], np.float32))
    ct = None if cdf[1] is None else dev(torch, np.asarray(cdf[1], np.float32))
    native.apex_prefetch_route(dev(torch, h), dev(torch, wpf),
                               None if bias is None else dev(torch, bias), B, d, E, k, k_max,
                               policy, tau, sd, cw, ct, pf_idx, pf_count, prob)
    torch.cuda.synchronize()
    return pf_idx.cpu().numpy(), pf_count.cpu().numpy(), prob.cpu().numpy()


def check_route(torch, cfg, h, policy, tau, sd=0, cdf=(None, None), k_max=None, ledger=None):
    k_max = cfg.k_max if k_max is None else k_max
    _, wpf, bias = inputs.router_weights(cfg, 0)
    tau32 = float(np.float32(tau))
    idx, cnt, prob = gpu_route(torch, h, wpf, bias, cfg.k, k_max, policy, tau32, sd, cdf)
    ref = routing.prefetch_route(h, wpf, bias, cfg.k, k_max, policy, tau32, sd, *cdf)
    ledger = ledger or TieLedger()
    ledger.compare_rows(cnt[:, None], ref["pf_count"][:, None], ref["margin"], "pf_count")
    ledger.compare_rows(idx, ref["pf_idx"], ref["margin"], "pf_idx")
    assert np.abs(prob - ref["prob"]).max() < 2e-6
    return ledger


@pytest.mark.parametrize("name", list(configs.CONFIGS))
def test_route_configs_all_policies(torch, name):
    cfg = configs.CONFIGS[name]
    h = tokens(cfg, 64)
    ledger = TieLedger()
    check_route(torch, cfg, h, native.SEL_CUMPROB, cfg.tau, ledger=ledger)
    check_route(torch, cfg, h, native.SEL_ORDINAL_CDF, cfg.tau, cdf=inputs.cdf_params(cfg, 0),
                ledger=ledger)
    check_route(torch, cfg, h, native.SEL_STATIC, 0.0, sd=2, ledger=ledger)
    check_route(torch, cfg, h, native.SEL_STATIC, 0.0, sd=0, ledger=ledger)
    check_route(torch, cfg, h, native.SEL_NONE, 0.0, ledger=ledger)
    print(name, ledger)


def test_route_tau_sweep_granite3b(torch):
    cfg = configs.GRANITE_3B
    h = tokens(cfg, 256)
    ledger = TieLedger()
    for tau in cfg.taus:
        check_route(torch, cfg, h, native.SEL_CUMPROB, tau, ledger=ledger)
    print(ledger)


@pytest.mark.parametrize("d,E,k,k_max,tau", [
    (8, 64, 1, 64, 1.0),       # smallest d, all 64 experts, tau unreachable -> whole list
    (520, 64, 8, 16, 0.0),     # ragged d (not a multiple of 512), tau = 0 -> m = k
    (1032, 1, 1, 1, 0.9),      # single expert
    (4096, 33, 5, 33, 0.97),
    (8192, 8, 2, 4, 0.9),      # largest supported d (LDS holds 32 KB of hidden state)
])
def test_route_edge_shapes(torch, d, E, k, k_max, tau):
    cfg = shape(f"edge{d}", 200 + E, d, E, k, k_max=k_max, bias=True)
    h = tokens(cfg, 17)
    ledger = check_route(torch, cfg, h, native.SEL_CUMPROB, tau)
    check_route(torch, cfg, h, native.SEL_ORDINAL_CDF, tau, cdf=inputs.cdf_params(cfg, 0),
                ledger=ledger)
    if tau >= 1.0:
        idx, cnt, _ = gpu_route(torch, h, inputs.router_weights(cfg, 0)[1], None, k, k_max,
                                native.SEL_CUMPROB, 1.0)
        assert (cnt == min(E, k_max)).all()


def test_route_writes_pinned_host_memory(torch):
    cfg = configs.GRANITE_1B
    h = tokens(cfg, 8)
    _, wpf, bias = inputs.router_weights(cfg, 0)
    a = gpu_route(torch, h, wpf, bias, cfg.k, cfg.k_max, native.SEL_CUMPROB, 0.9)
    b = gpu_route(torch, h, wpf, bias, cfg.k, cfg.k_max, native.SEL_CUMPROB, 0.9, out_host=True)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


# --------------------------------------------------------------------------- gate
def gpu_gate(torch, h, wg, bias, k, mode, avail=None, stride=0):
    B, d = h.shape
    E = wg.shape[0]
    outs = [torch.full((B, k), -7, dtype=torch.int32, device="cuda"),
            torch.full((B, k), -7.0, dtype=torch.float32, device="cuda"),
            torch.full((B, k), -7, dtype=torch.int32, device="cuda"),
            torch.full((B, k), -7.0, dtype=torch.float32, device="cuda"),
            torch.full((B, E), -7.0, dtype=torch.float32, device="cuda")]
    av = None if avail is None else dev(torch, avail.astype(np.uint8))
    native.apex_gate_topk(dev(torch, h), dev(torch, wg), None if bias is None else dev(torch, bias),
                          B, d, E, k, mode, av, stride, *outs)
    torch.cuda.synchronize()
    return [o.cpu().numpy() for o in outs]


def check_gate(torch, cfg, h, mode, avail=None, stride=0, ledger=None):
    wg, _, bias = inputs.router_weights(cfg, 0)
    ri, rg, xi, xg, prob = gpu_gate(torch, h, wg, bias, cfg.k, mode, avail, stride)
    if avail is not None and stride:
        B, E = h.shape[0], cfg.E
        mask = avail.reshape(-1)[:B * stride].reshape(B, stride)[:, :E].astype(bool)
    else:
        mask = None if avail is None else avail[:cfg.E].astype(bool)
    ref = gating.gate_topk(h, wg, bias, cfg.k, mode, mask)
    ledger = ledger or TieLedger()
    ledger.compare_rows(ri, ref["route_idx"], ref["margin"], "route_idx")
    ledger.compare_rows(xi, ref["exec_idx"], ref["margin"], "exec_idx")
    same = np.array([np.array_equal(xi[b], ref["exec_idx"][b]) for b in range(len(xi))])
    assert np.abs(xg[same] - ref["exec_gate"][same]).max(initial=0) < 2e-6
    assert np.abs(prob - ref["prob"]).max() < 2e-6
    assert np.allclose(xg.sum(1)[(xi >= 0).any(1)], 1.0, atol=1e-5)
    return ledger


@pytest.mark.parametrize("name", list(configs.CONFIGS))
def test_gate_configs_both_modes(torch, name):
    cfg = configs.CONFIGS[name]
    h = tokens(cfg, 64, which=1)
    rng = np.random.default_rng(cfg.cfg_id)
    ledger = check_gate(torch, cfg, h, native.MODE_EXACT)
    # stall-free with everything available equals exact
    a = gpu_gate(torch, h, *inputs.router_weights(cfg, 0)[::2], cfg.k, native.MODE_EXACT)
    b = gpu_gate(torch, h, *inputs.router_weights(cfg, 0)[::2], cfg.k, native.MODE_STALL_FREE,
                 np.ones(cfg.E, np.uint8))
    for u, v in zip(a, b):
        assert np.array_equal(u, v)
    # a cache-sized shared mask, per-token masks, and a padded per-token stride
    shared = np.zeros(cfg.E, np.uint8)
    shared[rng.choice(cfg.E, cfg.C, replace=False)] = 1
    check_gate(torch, cfg, h, native.MODE_STALL_FREE, shared, 0, ledger)
    per = (rng.random((64, cfg.E)) < 0.5).astype(np.uint8)
    check_gate(torch, cfg, h, native.MODE_STALL_FREE, per.ravel(), cfg.E, ledger)
    padded = np.zeros((64, cfg.E + 5), np.uint8)
    padded[:, :cfg.E] = per
    check_gate(torch, cfg, h, native.MODE_STALL_FREE, padded.ravel(), cfg.E + 5, ledger)
    print(name, ledger)


def test_gate_fewer_available_than_k_and_none(torch):
    cfg = shape("gate_few", 301, 264, 16, 6, bias=True)
    h = tokens(cfg, 9, which=1)
    few = np.zeros(16, np.uint8)
    few[[3, 9, 11]] = 1
    check_gate(torch, cfg, h, native.MODE_STALL_FREE, few)
    wg, _, bias = inputs.router_weights(cfg, 0)
    _, _, xi, xg, _ = gpu_gate(torch, h, wg, bias, 6, native.MODE_STALL_FREE,
                               np.zeros(16, np.uint8))
    assert (xi == -1).all() and (xg == 0).all()


# --------------------------------------------------------------------------- FFN
class FfnCase:
    """A slot pool holding some of the experts, and a batch routed over all of them."""

    def __init__(self, torch, cfg, B, seed, resident_frac=1.0, n_slots_extra=0, weights="bf16"):
        rng = np.random.default_rng(seed)
        self.cfg, self.B, self.weights = cfg, B, weights
        E, k = cfg.E, cfg.k
        _, nbytes, pack, self.ffn = native.weight_format(weights)
        self.S = nbytes(cfg.d, cfg.I)
        self.x = rng.standard_normal((B, cfg.d)).astype(np.float32)
        self.exec_idx = np.stack([rng.choice(E, k, replace=False) for _ in range(B)]).astype(np.int32)
        if B > 1:
            self.exec_idx[rng.random((B, k)) < 0.1] = -1     # unused positions
        g = rng.random((B, k)) + 0.05
        self.gate = (g / g.sum(1, keepdims=True)).astype(np.float32)
        used = sorted(set(int(e) for e in self.exec_idx.ravel() if e >= 0))
        n_res = max(1, int(round(len(used) * resident_frac)))
        self.resident = sorted(rng.choice(used, n_res, replace=False).tolist())
        self.n_slots = len(self.resident) + n_slots_extra
        slot_ids = rng.permutation(self.n_slots)[:len(self.resident)]
        self.table = np.full(E, -1, np.int32)
        for e, s in zip(self.resident, slot_ids):
            self.table[e] = s
        self.bits = {}
        if weights != "bf16":
            pool = np.zeros(self.n_slots * self.S, np.uint8)
            piece = lambda s: pool[s * self.S:(s + 1) * self.S]
        else:
            pool = np.zeros(self.n_slots * self.S // 2, np.uint16)
            piece = lambda s: pool[s * self.S // 2:(s + 1) * self.S // 2]
        for e in self.resident:
            self.bits[e] = inputs.expert_weights(cfg, 0, e)
            pack(*self.bits[e], cfg.d, cfg.I, piece(int(self.table[e])))
        self.pool = dev(torch, pool)
        self.torch = torch

    def run(self, table=None, y0=None, accumulate=0):
        torch, cfg, B = self.torch, self.cfg, self.B
        table = self.table if table is None else table
        ws_bytes = native.apex_moe_ffn_workspace_bytes(B, cfg.d, cfg.I, cfg.k)
        ws = torch.full((ws_bytes,), 0xAB, dtype=torch.uint8, device="cuda")
        y = dev(torch, y0) if y0 is not None else torch.full((B, cfg.d), float("nan"),
                                                              device="cuda")
        self.ffn(dev(torch, self.x), B, cfg.d, cfg.I, cfg.E, cfg.k, dev(torch, self.exec_idx),
            dev(torch, self.gate), dev(torch, table), self.pool, self.n_slots, y, accumulate, ws,
            ws_bytes)
        torch.cuda.synchronize()
        return y.cpu().numpy()

    def oracle_rows(self, rows):
        """The oracle for a few tokens only (each output row depends on its token alone)."""
        skip = set(range(self.cfg.E)) - set(self.resident)
        return offn.moe_ffn(self.x[rows], self.exec_idx[rows],
                            self.gate[rows].astype(np.float64), lambda e: self.bits[e], skip=skip,
                            weights=self.weights)

    def oracle(self, only=None):
        keep = set(self.resident) if only is None else set(only)
        skip = set(range(self.cfg.E)) - keep
        return offn.moe_ffn(self.x, self.exec_idx, self.gate.astype(np.float64),
                            lambda e: self.bits[e], skip=skip, weights=self.weights)


FFN_SHAPES = [
    # (cfg, B)
    (shape("ffn_small", 400, 256, 8, 2, I=512), 1),
    (shape("ffn_ragged", 401, 520, 5, 3, I=136), 3),     # ragged d and I tails
    (shape("ffn_tiny_tiles", 402, 8, 4, 2, I=8), 2),     # one 16-byte chunk per row
    (shape("ffn_b8", 403, 1024, 32, 8, I=512), 8),
    (shape("ffn_wide_k", 404, 264, 64, 16, I=72), 64),   # B*k = 1024 pairs (the maximum)
    # one token with rows of 513..4096 values: the up projection splits each row over a
    # workgroup's lanes (one 16-byte chunk per lane, idle lanes past the row's end)
    (shape("ffn_split_d520", 420, 520, 5, 3, I=72), 1),      # 65 chunks on 128 lanes
    (shape("ffn_split_d1032", 421, 1032, 6, 2, I=96), 1),    # 129 chunks on 256 lanes
    (shape("ffn_split_d1800", 408, 1800, 6, 3, I=136), 1),   # 225 chunks on 256 lanes
    (shape("ffn_split_d2056", 409, 2056, 4, 2, I=40), 1),    # 257 chunks on 512 lanes
    (shape("ffn_split_two_rows", 418, 2304, 3, 2, I=8200), 1),  # I*k > 16384: 2 rows
]


@pytest.mark.parametrize("cfg,B", FFN_SHAPES, ids=[c.name for c, _ in FFN_SHAPES])
def test_ffn_parity_shapes(torch, cfg, B):
    case = FfnCase(torch, cfg, B, seed=cfg.cfg_id)
    y = case.run()
    print(cfg.name, ffn_close(y, case.oracle(), cfg.name))


@pytest.mark.parametrize("name,B", [("granite-1b-a400m", 1), ("granite-3b-a800m", 1),
                                    ("granite-3b-a800m", 8), ("olmoe-1b-7b", 1),
                                    ("olmoe-1b-7b", 16), ("olmoe-1b-7b", 64),
                                    ("deepseek-16b", 1), ("phi-7b", 1), ("tiny", 1)])
def test_ffn_parity_workload_shapes(torch, name, B):
    cfg = configs.CONFIGS[name]
    case = FfnCase(torch, cfg, B, seed=cfg.cfg_id * 10 + B)
    y = case.run()
    print(name, B, ffn_close(y, case.oracle(), f"{name} B{B}"))


MFMA_SHAPES = [
    # batched path (>= 2 tokens; the shapes above with B > 1 take it too): matrix-core
    # grouped GEMMs with one, two or four 16-token tiles per pass
    (shape("mfma_ragged", 410, 264, 12, 3, I=200), 40),   # d % 32 != 0, I % 16 != 0
    (shape("mfma_b48", 411, 512, 6, 2, I=256), 48),       # four token tiles per pass
    (shape("mfma_b16", 412, 1024, 32, 8, I=512), 16),     # one tile per pass
    (shape("mfma_b2", 415, 1024, 32, 8, I=512), 2),       # smallest batch on this path
    # four experts with ragged K tails on both sides (every split plan is run by
    # test_ffn_every_plan_matches_oracle)
    (shape("mfma_split_a", 416, 776, 4, 2, I=1000), 4),
    (shape("mfma_split_b", 417, 1000, 4, 2, I=776), 5),
]


@pytest.mark.parametrize("cfg,B", MFMA_SHAPES, ids=[c.name for c, _ in MFMA_SHAPES])
def test_ffn_mfma_parity(torch, cfg, B):
    case = FfnCase(torch, cfg, B, seed=cfg.cfg_id)
    y = case.run()
    print(cfg.name, B, ffn_close(y, case.oracle(), cfg.name))


@pytest.mark.parametrize("weights,B,d,I,E,plan", PLAN_CASES,
                         ids=[f"{w}-B{b}-d{d}-I{i}-{'x'.join(map(str, p))}"
                              for w, b, d, i, _, p in PLAN_CASES])
def test_ffn_every_plan_matches_oracle(torch, weights, B, d, I, E, plan):
    cfg = shape(f"plan_{weights}_{B}_{d}_{I}", 460 + PLAN_CASES.index(
        (weights, B, d, I, E, plan)), d, E, 2, I=I)
    case = FfnCase(torch, cfg, B, seed=cfg.cfg_id, weights=weights)
    assert native.apex_moe_ffn_plan(B, d, I, E, 2, case.n_slots, weights) == plan
    y = case.run()
    print(cfg.name, plan, ffn_close(y, case.oracle(), f"{cfg.name} {plan}"))
    # no atomics and a fixed order of the split sums: a second call (fresh workspace
    # garbage, NaN-filled output) gives the same bits
    y2 = case.run()
    assert np.array_equal(y.view(np.uint32), y2.view(np.uint32)), f"{cfg.name} {plan}"


def test_ffn_mfma_skewed_expert_takes_every_token(torch):
    # expert 0 is in every token's set: 128 tokens on one expert = several passes of
    # four 16-token tiles; the others are spread out
    cfg = shape("mfma_skew", 413, 256, 16, 8, I=128)
    case = FfnCase(torch, cfg, 128, seed=5)
    rng = np.random.default_rng(6)
    for b in range(128):
        others = rng.choice(np.arange(1, 16), cfg.k - 1, replace=False)
        case.exec_idx[b] = np.concatenate([[0], others]).astype(np.int32)
    assert all(case.table[e] >= 0 for e in range(16))   # 128 random tokens used all 16
    y = case.run()
    print("skew", ffn_close(y, case.oracle(), "skewed"))


def test_ffn_mfma_two_passes_equal_one(torch):
    cfg = shape("mfma_pass", 414, 392, 12, 4, I=200)
    case = FfnCase(torch, cfg, 24, seed=17, n_slots_extra=2)
    full = case.oracle()
    res = case.resident
    first, second = res[: len(res) // 2], res[len(res) // 2:]
    t1 = case.table.copy()
    t1[second] = -1
    t2 = case.table.copy()
    t2[first] = -1
    y1 = case.run(t1)
    ffn_close(y1, case.oracle(only=first), "mfma pass 1")
    y2 = case.run(t2, y0=y1, accumulate=1)
    ffn_close(y2, full, "mfma pass 1 + pass 2")


def test_ffn_parity_mixtral_batch1(torch):
    cfg = configs.MIXTRAL
    case = FfnCase(torch, cfg, 1, seed=44)
    y = case.run()
    print("mixtral", ffn_close(y, case.oracle(), "mixtral B1"))


@pytest.mark.parametrize("B", [8, 32])
def test_ffn_parity_mixtral_batched_sampled_tokens(torch, B):
    # the bench's launch configuration at full size: 4 of the 8 experts resident, so the
    # down projection splits K four ways (and the gate/up projection two ways at B = 8);
    # the oracle checks three of the tokens, one at a time, and a permuted batch the rest
    cfg = configs.MIXTRAL
    case = FfnCase(torch, cfg, B, seed=45 + B, resident_frac=0.5)
    y = case.run()
    rows = [0, B // 2, B - 1]
    want = case.oracle_rows(rows)
    for i, r in enumerate(rows):
        print("mixtral", B, r, ffn_close(y[r:r + 1], want[i:i + 1], f"mixtral B{B} token {r}"))
    # every other token: a token's output depends on its own row alone, in a fixed order
    # of operations, so the same batch in another token order gives the same rows, bit
    # for bit (the plan depends on the sizes only); the three checked tokens move to other
    # positions, tiles and split partials
    perm = np.random.default_rng(B).permutation(B)
    case.x, case.exec_idx, case.gate = case.x[perm], case.exec_idx[perm], case.gate[perm]
    y_perm = case.run()
    assert np.array_equal(y_perm, y[perm])


FP8_SHAPES = [
    # E4M3 experts (apex_moe_ffn_fp8): d and I multiples of 16
    (configs.GRANITE_1B, 1), (configs.GRANITE_3B, 1), (configs.OLMOE, 1), (configs.TINY, 1),
    (configs.GRANITE_3B, 8), (configs.OLMOE, 16),
    (shape("fp8_b48", 430, 512, 6, 2, I=256), 48),         # four token tiles per pass
    (shape("fp8_split_a", 431, 784, 4, 2, I=1008), 4),     # few experts, ragged K tails
    (shape("fp8_split_b", 432, 1008, 4, 2, I=784), 5),
    (shape("fp8_small", 433, 16, 3, 2, I=48), 3),          # one 16-byte chunk per row
    # one token, rows of 1025..4096 values: the up projection splits each row over a
    # workgroup (one 16-code chunk per lane, 1, 2 or 4 row pairs per workgroup)
    (configs.PHI_7B, 1), (configs.DEEPSEEK_16B, 1),
    (shape("fp8_b1_split_a", 436, 1040, 6, 3, I=112), 1),  # 65 chunks on 128 lanes
    (shape("fp8_b1_split_b", 437, 2064, 4, 2, I=1104), 1),  # 129 chunks on 256 lanes
    (shape("fp8_b1_split_c", 438, 2080, 3, 2, I=8224), 1),  # I*k > 16384: 4 row pairs
]


@pytest.mark.parametrize("cfg,B", FP8_SHAPES, ids=[f"{c.name}-B{b}" for c, b in FP8_SHAPES])
def test_ffn_fp8_parity(torch, cfg, B):
    case = FfnCase(torch, cfg, B, seed=cfg.cfg_id * 7 + B, weights="fp8")
    y = case.run()
    print(cfg.name, B, ffn_close(y, case.oracle(), f"{cfg.name} B{B} fp8"))


def test_ffn_fp8_mixtral_batch1_and_two_passes(torch):
    # d = 4096 takes the wide batch-1 kernels; a second pass adds the other experts
    cfg = configs.MIXTRAL
    case = FfnCase(torch, cfg, 1, seed=50, weights="fp8")
    print("mixtral fp8", ffn_close(case.run(), case.oracle(), "mixtral B1 fp8"))
    cfg = shape("fp8_pass", 434, 512, 12, 4, I=256)
    case = FfnCase(torch, cfg, 20, seed=51, n_slots_extra=2, weights="fp8")
    res = case.resident
    first, second = res[: len(res) // 2], res[len(res) // 2:]
    t1, t2 = case.table.copy(), case.table.copy()
    t1[second] = -1
    t2[first] = -1
    y1 = case.run(t1)
    ffn_close(y1, case.oracle(only=first), "fp8 pass 1")
    ffn_close(case.run(t2, y0=y1, accumulate=1), case.oracle(), "fp8 pass 1 + pass 2")


MXFP4_SHAPES = [
    # MXFP4 experts (apex_moe_ffn_mxfp4): d and I multiples of 32
    (configs.GRANITE_1B, 1), (configs.GRANITE_3B, 1), (configs.OLMOE, 1), (configs.TINY, 1),
    (configs.PHI_7B, 1), (configs.DEEPSEEK_16B, 1),         # d = 4096; I = 1472
    (configs.GRANITE_3B, 8), (configs.OLMOE, 16),
    (shape("fp4_b48", 440, 512, 6, 2, I=256), 48),          # four token tiles per pass
    (shape("fp4_split_a", 441, 800, 4, 2, I=992), 4),       # few experts; ragged last K block
    (shape("fp4_split_b", 442, 992, 4, 2, I=800), 5),
    (shape("fp4_small", 443, 32, 3, 2, I=64), 3),           # one block per row
    # one token, rows of 1025..4096 values: split rows, one 16-code unit per lane
    (shape("fp4_b1_split_a", 445, 1056, 6, 3, I=96), 1),    # 66 units on 128 lanes
    (shape("fp4_b1_split_b", 446, 2080, 3, 2, I=8224), 1),  # I*k > 16384: 4 row pairs
]


@pytest.mark.parametrize("cfg,B", MXFP4_SHAPES, ids=[f"{c.name}-B{b}" for c, b in MXFP4_SHAPES])
def test_ffn_mxfp4_parity(torch, cfg, B):
    case = FfnCase(torch, cfg, B, seed=cfg.cfg_id * 11 + B, weights="mxfp4")
    y = case.run()
    print(cfg.name, B, ffn_close(y, case.oracle(), f"{cfg.name} B{B} mxfp4"))


def test_ffn_mxfp4_mixtral_batch1_and_two_passes(torch):
    cfg = configs.MIXTRAL
    case = FfnCase(torch, cfg, 1, seed=52, weights="mxfp4")
    print("mixtral mxfp4", ffn_close(case.run(), case.oracle(), "mixtral B1 mxfp4"))
    cfg = shape("fp4_pass", 444, 512, 12, 4, I=256)
    case = FfnCase(torch, cfg, 20, seed=53, n_slots_extra=2, weights="mxfp4")
    res = case.resident
    first, second = res[: len(res) // 2], res[len(res) // 2:]
    t1, t2 = case.table.copy(), case.table.copy()
    t1[second] = -1
    t2[first] = -1
    y1 = case.run(t1)
    ffn_close(y1, case.oracle(only=first), "mxfp4 pass 1")
    ffn_close(case.run(t2, y0=y1, accumulate=1), case.oracle(), "mxfp4 pass 1 + pass 2")


FP32_SHAPES = [
    # 32-bit experts (apex_moe_ffn_fp32, batch 1 only): d and I multiples of 4; the up
    # projection's workgroup covers the row one 16-byte chunk (4 values) per lane
    (configs.GRANITE_1B, 1), (configs.GRANITE_3B, 1), (configs.OLMOE, 1), (configs.TINY, 1),
    (configs.PHI_7B, 1), (configs.DEEPSEEK_16B, 1),
    (shape("fp32_d260", 510, 260, 5, 3, I=76), 1),        # 65 chunks on 128 lanes
    (shape("fp32_d1028", 511, 1028, 4, 2, I=44), 1),      # 257 chunks on 512 lanes
    (shape("fp32_d4100", 512, 4100, 4, 2, I=36), 1),      # beyond 4096: a row pair per wavefront
    (shape("fp32_two_rows", 513, 520, 3, 2, I=8200), 1),  # I*k > 16384: two row pairs
]


@pytest.mark.parametrize("cfg,B", FP32_SHAPES, ids=[f"{c.name}-B{b}" for c, b in FP32_SHAPES])
def test_ffn_fp32_parity(torch, cfg, B):
    case = FfnCase(torch, cfg, B, seed=cfg.cfg_id * 13 + B, weights="fp32")
    y = case.run()
    print(cfg.name, B, ffn_close(y, case.oracle(), f"{cfg.name} B{B} fp32"))


def test_ffn_fp32_mixtral_batch1_two_passes_and_repeat(torch):
    # the Mixtral shape (704 MB experts), then two passes, absent experts and a repeated
    # call at a small shape
    case = FfnCase(torch, configs.MIXTRAL, 1, seed=52, weights="fp32")
    print("mixtral fp32", ffn_close(case.run(), case.oracle(), "mixtral B1 fp32"))
    cfg = shape("fp32_pass", 514, 1028, 6, 3, I=76)
    case = FfnCase(torch, cfg, 1, seed=53, n_slots_extra=2, weights="fp32")
    res = case.resident
    t1, t2 = case.table.copy(), case.table.copy()
    t1[res[1:]] = -1
    t2[res[:1]] = -1
    y1 = case.run(t1)
    ffn_close(y1, case.oracle(only=res[:1]), "fp32 pass 1")
    ffn_close(case.run(t2, y0=y1, accumulate=1), case.oracle(), "fp32 pass 1 + pass 2")
    none = np.full(cfg.E, -1, np.int32)
    assert np.array_equal(case.run(none, y0=y1, accumulate=1), y1)
    assert (case.run(none) == 0).all()
    assert np.array_equal(case.run(), case.run())


def test_ffn_mxfp4_rejects_partial_blocks(torch):
    A = 4096
    with pytest.raises(native.ApexError):
        native.apex_moe_ffn_mxfp4(A, 1, 48, 64, 4, 1, A, A, A, A, 1, A, 0, A, 1 << 20)
    with pytest.raises(native.ApexError):
        native.apex_moe_ffn_mxfp4(A, 1, 64, 48, 4, 1, A, A, A, A, 1, A, 0, A, 1 << 20)


def test_ffn_two_passes_equal_one(torch):
    cfg = shape("ffn_pass", 405, 392, 12, 4, I=200)
    case = FfnCase(torch, cfg, 5, seed=7, n_slots_extra=3)
    full = case.oracle()
    res = case.resident
    first, second = res[: len(res) // 2], res[len(res) // 2:]
    t1 = case.table.copy()
    t1[second] = -1
    t2 = case.table.copy()
    t2[first] = -1
    y1 = case.run(t1)
    ffn_close(y1, case.oracle(only=first), "pass 1")
    y2 = case.run(t2, y0=y1, accumulate=1)
    ffn_close(y2, full, "pass 1 + pass 2")
    # nothing resident: accumulate leaves y unchanged, overwrite gives zeros
    none = np.full(cfg.E, -1, np.int32)
    assert np.array_equal(case.run(none, y0=y1, accumulate=1), y1)
    assert (case.run(none) == 0).all()


@pytest.mark.parametrize("d,I", [(520, 72), (1800, 136), (2056, 40), (2056, 4104)])
def test_ffn_batch1_split_rows_two_passes_and_repeat(torch, d, I):
    """One token over the split-row up projection: two passes (the second accumulating)
    equal one, absent experts leave y alone, and a repeated call is bitwise equal.  Past
    2048 output rows the down projection takes two rows per wavefront over short dot
    products (3 x 40 values) and four over long ones (3 x 4104, a ragged chunk count)."""
    cfg = shape(f"ffn_split_pass_{d}", 419, d, 6, 3, I=I)
    case = FfnCase(torch, cfg, 1, seed=d, n_slots_extra=2)
    full = case.oracle()
    res = case.resident
    first, second = res[:1], res[1:]
    t1 = case.table.copy()
    t1[second] = -1
    t2 = case.table.copy()
    t2[first] = -1
    y1 = case.run(t1)
    ffn_close(y1, case.oracle(only=first), "pass 1")
    y2 = case.run(t2, y0=y1, accumulate=1)
    ffn_close(y2, full, "pass 1 + pass 2")
    none = np.full(cfg.E, -1, np.int32)
    assert np.array_equal(case.run(none, y0=y1, accumulate=1), y1)
    assert (case.run(none) == 0).all()
    assert np.array_equal(case.run(), case.run())


def test_ffn_slots_beyond_pool_are_skipped(torch):
    cfg = shape("ffn_bound", 406, 128, 6, 2, I=64)
    case = FfnCase(torch, cfg, 4, seed=9)
    bad = case.table.copy()
    victim = case.resident[0]
    bad[victim] = case.n_slots + 5          # out of the pool: treated as absent
    y = case.run(bad)
    ffn_close(y, case.oracle(only=case.resident[1:]), "out-of-pool slot")


def test_ffn_is_deterministic(torch):
    cfg = shape("ffn_det", 407, 1024, 16, 4, I=256)
    case = FfnCase(torch, cfg, 8, seed=11)
    a, b = case.run(), case.run()
    assert np.array_equal(a, b)


# --------------------------------------------------------------------------- copies
def test_expert_prefetch_and_miss_fetch(torch):
    cfg = shape("pf", 500, 64, 8, 2, I=32, C=4, k_max=4)
    E, C, S = cfg.E, cfg.C, native.apex_expert_bytes(cfg.d, cfg.I)
    rng = np.random.default_rng(5)
    host = torch.empty(E * S // 2, dtype=torch.int16, pin_memory=True)
    host.copy_(torch.from_numpy(rng.integers(-30000, 30000, E * S // 2).astype(np.int16)))
    slots = torch.zeros(C * S // 2, dtype=torch.int16, device="cuda")
    slots.copy_(host[:C * S // 2])
    eos = np.arange(C, dtype=np.int32)
    lu = np.full(E, -1, np.int64)
    slot_dev = dev(torch, np.array([s if s < C else -1 for s in range(E)], np.int32))
    avail_dev = torch.zeros(E, dtype=torch.uint8, device="cuda")
    side = torch.cuda.Stream()
    cs, ss = torch.cuda.current_stream().cuda_stream, side.cuda_stream
    ready = native.apex_event_create(False)
    done = native.apex_event_create(False)
    ref = Residency(E, C)
    B = 2
    for t in range(25):
        pf_idx = np.full((B, cfg.k_max), -1, np.int32)
        pf_cnt = np.zeros(B, np.int32)
        lists = []
        for b in range(B):
            m = int(rng.integers(cfg.k, cfg.k_max + 1))
            pf_idx[b, :m] = rng.choice(E, m, replace=False)
            pf_cnt[b] = m
            lists.append(list(pf_idx[b, :m]))
        copied = np.zeros(C, np.int32)
        n = native.apex_expert_prefetch(host, slots, E, C, S, pf_idx, pf_cnt, B, cfg.k_max, t,
                                        eos, lu, slot_dev, avail_dev, ss, cs, done, ready, copied)
        want = ref.plan(lists, t)
        assert [int(e) for e in copied[:n]] == [e for e, _ in want]
        native.apex_stream_wait_event(cs, ready)
        native.apex_event_record(done, cs)
        torch.cuda.synchronize()
        hs, ds = host.view(E, -1), slots.view(C, -1).cpu()
        for s in range(C):
            assert torch.equal(ds[s], hs[int(eos[s])]), (t, s)
        table = np.full(E, -1, np.int32)
        table[eos] = np.arange(C)
        assert np.array_equal(slot_dev.cpu().numpy(), table)
        assert np.array_equal(avail_dev.cpu().numpy(), (table >= 0).astype(np.uint8))
    # miss correction: routed experts outside the resident set go to scratch, in id order
    scratch = torch.zeros(E * S // 2, dtype=torch.int16, device="cuda")
    miss_tab = torch.full((E,), -9, dtype=torch.int32, device="cuda")
    route = np.stack([rng.choice(E, cfg.k, replace=False) for _ in range(3)]).astype(np.int32)
    missing = np.zeros(E, np.int32)
    n = native.apex_expert_fetch_misses(host, scratch, E, E, C, S, route, 3, cfg.k, eos,
                                        miss_tab, ss, cs, None, ready, missing)
    expect = sorted(set(route.ravel().tolist()) - set(eos.tolist()))
    assert list(missing[:n]) == expect
    native.apex_stream_wait_event(cs, ready)
    torch.cuda.synchronize()
    hs, sc = host.view(E, -1), scratch.view(E, -1).cpu()
    for i, e in enumerate(expect):
        assert torch.equal(sc[i], hs[e])
    mt = np.full(E, -1, np.int32)
    mt[expect] = np.arange(len(expect))
    assert np.array_equal(miss_tab.cpu().numpy(), mt)
    native.apex_event_destroy(ready)
    native.apex_event_destroy(done)


def test_expert_copies_span_strides_and_refuse_pageable_memory(torch):
    # experts of 1.63 MB: 400 chunks of 4 KB each, the last one ragged, so every copy
    # workgroup moves many chunks across expert boundaries
    d, I, E, C = 1032, 264, 6, 3
    S = native.apex_expert_bytes(d, I)
    assert (S // 16) % 256 != 0 and S // 4096 > 24
    rng = np.random.default_rng(21)
    host = torch.empty(E * S // 2, dtype=torch.int16, pin_memory=True)
    host.copy_(torch.from_numpy(rng.integers(-30000, 30000, E * S // 2).astype(np.int16)))
    slots = torch.zeros(C * S // 2, dtype=torch.int16, device="cuda")
    eos = np.full(C, -1, np.int32)
    lu = np.full(E, -1, np.int64)
    slot_dev = torch.full((E,), -1, dtype=torch.int32, device="cuda")
    side = torch.cuda.Stream()
    cs, ss = torch.cuda.current_stream().cuda_stream, side.cuda_stream
    ready = native.apex_event_create(False)
    pf_idx = np.array([[4, 1, 5, -1]], np.int32)
    pf_cnt = np.array([3], np.int32)
    # pageable memory (which a kernel cannot read) is refused before any table changes or
    # anything is enqueued
    for bad in (np.zeros(E * S // 2, np.int16),):
        with pytest.raises(native.ApexError, match="pinned"):
            native.apex_expert_prefetch(bad, slots, E, C, S, pf_idx, pf_cnt, 1, 4, 0, eos, lu,
                                        slot_dev, None, ss, cs, None, ready)
        with pytest.raises(native.ApexError, match="pinned"):
            native.apex_expert_fetch_misses(bad, slots, C, E, C, S, np.array([[0, 2]], np.int32),
                                            1, 2, eos, slot_dev, ss, cs, None, ready)
        assert (eos == -1).all() and (lu == -1).all()
    n = native.apex_expert_prefetch(host, slots, E, C, S, pf_idx, pf_cnt, 1, 4, 0, eos, lu,
                                    slot_dev, None, ss, cs, None, ready)
    assert n == 3
    native.apex_stream_wait_event(cs, ready)
    torch.cuda.synchronize()
    hs, ds = host.view(E, -1), slots.view(C, -1).cpu()
    assert sorted(eos.tolist()) == [1, 4, 5]
    for s in range(C):
        assert torch.equal(ds[s], hs[int(eos[s])]), s
    # misses: experts 0 and 2 into a scratch pool of 2
    scratch = torch.zeros(2 * S // 2, dtype=torch.int16, device="cuda")
    miss_tab = torch.full((E,), -9, dtype=torch.int32, device="cuda")
    n = native.apex_expert_fetch_misses(host, scratch, 2, E, C, S, np.array([[2, 5, 0]], np.int32),
                                        1, 3, eos, miss_tab, ss, cs, None, ready)
    assert n == 2
    native.apex_stream_wait_event(cs, ready)
    torch.cuda.synchronize()
    sc = scratch.view(2, -1).cpu()
    assert torch.equal(sc[0], hs[0]) and torch.equal(sc[1], hs[2])
    native.apex_event_destroy(ready)


def test_expert_copies_of_large_experts(torch):
    # experts of 48 MB and a ragged 4 KB chunk at the end of each: the copy kernel's wide
    # grid for experts of 32 MB and more, for the prefetch and for the miss fetch, every
    # byte compared
    E, C = 3, 2
    S = (48 << 20) + 1040
    assert S >= (32 << 20) and S % 16 == 0 and (S // 16) % 256 != 0
    host = torch.randint(-2 ** 15, 2 ** 15 - 1, (E * S // 2,), dtype=torch.int16,
                         generator=torch.Generator().manual_seed(31)).pin_memory()
    slots = torch.zeros(C * S // 2, dtype=torch.int16, device="cuda")
    eos = np.full(C, -1, np.int32)
    lu = np.full(E, -1, np.int64)
    slot_dev = torch.full((E,), -1, dtype=torch.int32, device="cuda")
    side = torch.cuda.Stream()
    cs, ss = torch.cuda.current_stream().cuda_stream, side.cuda_stream
    ready = native.apex_event_create(False)
    n = native.apex_expert_prefetch(host, slots, E, C, S, np.array([[2, 0]], np.int32),
                                    np.array([2], np.int32), 1, 2, 0, eos, lu, slot_dev, None,
                                    ss, cs, None, ready)
    assert n == 2 and sorted(eos.tolist()) == [0, 2]
    native.apex_stream_wait_event(cs, ready)
    torch.cuda.synchronize()
    hs, ds = host.view(E, -1), slots.view(C, -1).cpu()
    for s in range(C):
        assert torch.equal(ds[s], hs[int(eos[s])]), s
    assert slot_dev.cpu().numpy()[1] == -1
    scratch = torch.zeros(S // 2, dtype=torch.int16, device="cuda")
    miss_tab = torch.full((E,), -9, dtype=torch.int32, device="cuda")
    n = native.apex_expert_fetch_misses(host, scratch, 1, E, C, S, np.array([[1, 2]], np.int32),
                                        1, 2, eos, miss_tab, ss, cs, None, ready)
    assert n == 1
    native.apex_stream_wait_event(cs, ready)
    torch.cuda.synchronize()
    assert torch.equal(scratch.cpu(), hs[1])
    assert miss_tab.cpu().numpy().tolist() == [-1, 0, -1]
    native.apex_event_destroy(ready)


def test_spin_and_copy_kernel(torch):
    s = torch.cuda.current_stream().cuda_stream
    a, b = native.apex_event_create(True), native.apex_event_create(True)
    native.apex_event_record(a, s)
    native.apex_spin_us(300.0, s)
    native.apex_event_record(b, s)
    native.apex_event_synchronize(b)
    ms = native.apex_event_elapsed_ms(a, b)
    assert 0.29 <= ms < 5.0, ms
    src = torch.randint(-2 ** 31, 2 ** 31 - 1, (1 << 22,), dtype=torch.int32, device="cuda")
    dst = torch.zeros_like(src)
    native.apex_copy_kernel(dst, src, src.numel() * 4, s)
    torch.cuda.synchronize()
    assert torch.equal(src, dst)
    native.apex_event_destroy(a)
    native.apex_event_destroy(b)


def test_read_kernel_reads_every_chunk(torch):
    # the fold of all words equals the XOR of the buffer: every 16-byte chunk was read
    s = torch.cuda.current_stream().cuda_stream
    for n_words in (4, 4 * 1000 + 4, 1 << 22):           # tails shorter than one stride
        src = torch.randint(-2 ** 31, 2 ** 31 - 1, (n_words,), dtype=torch.int32, device="cuda")
        words = native.apex_read_kernel_sink_words(n_words * 4)
        sink = torch.full((words,), 0, dtype=torch.int32, device="cuda")
        native.apex_read_kernel(src, n_words * 4, sink, s)
        torch.cuda.synchronize()
        want = np.bitwise_xor.reduce(src.cpu().numpy().view(np.uint32))
        got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
        assert got == want, n_words
    with pytest.raises(native.ApexError):
        native.apex_read_kernel(src, 12, sink, s)


def test_readme_example_runs(torch):
    """The Python example of README.md, run as written."""
    import re
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    text = open(os.path.join(root, "README.md")).read()
    code = re.search(r"<!-- example: moe_ffn -->\s*```python\n(.*?)```", text, re.S).group(1)
    exec(compile(code, "README.md example", "exec"), {})


GRAPH_CASES = [(configs.GRANITE_1B, 1, "bf16"), (configs.MIXTRAL, 1, "bf16"),
               (configs.GRANITE_3B, 8, "bf16"), (configs.OLMOE, 16, "fp8"),
               (configs.OLMOE, 1, "mxfp4"), (configs.GRANITE_1B, 1, "fp32")]


@pytest.mark.parametrize("cfg,B,weights", GRAPH_CASES,
                         ids=[f"{c.name}-B{b}-{w}" for c, b, w in GRAPH_CASES])
def test_ffn_replayed_from_a_captured_graph_matches_eager(torch, cfg, B, weights):
    """The FFN entry points allocate nothing and set no memory inside a call, so a caller can
    capture them in a HIP graph: every replay, with new activations copied in, eager calls
    and synchronisations between the replays, equals the eager call on the same inputs bit
    for bit (the workspace entry point and the one that allocates nothing)."""
    case = FfnCase(torch, cfg, B, seed=cfg.cfg_id * 7 + B, weights=weights)
    d, I, E, k = cfg.d, cfg.I, cfg.E, cfg.k
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    x, idx, gate, table = dev(case.x), dev(case.exec_idx), dev(case.gate), dev(case.table)
    ws_bytes = native.apex_moe_ffn_workspace_bytes(B, d, I, k)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    calls = {
        "workspace": lambda out, s: case.ffn(x, B, d, I, E, k, idx, gate, table, case.pool,
                                             case.n_slots, out, 0, ws, ws_bytes, s),
        "noalloc": lambda out, s: native.apex_moe_ffn_noalloc(
            x, B, d, I, E, k, idx, gate, table, case.pool, case.n_slots, weights, out, 0, s),
    }
    rng = np.random.default_rng(cfg.cfg_id)
    for name, call in calls.items():
        y = torch.zeros((B, d), device="cuda")
        y_eager = torch.zeros_like(y)
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            call(y, side.cuda_stream)          # first call outside the capture
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=side):
            call(y, side.cuda_stream)
        torch.cuda.synchronize()
        for r in range(3):
            x.copy_(dev(rng.standard_normal((B, d)).astype(np.float32)))
            y.fill_(float("nan"))
            graph.replay()
            torch.cuda.synchronize()
            call(y_eager, torch.cuda.current_stream().cuda_stream)
            torch.cuda.synchronize()
            assert torch.equal(y, y_eager), (name, r)
            assert torch.isfinite(y).all(), (name, r)
        del graph


@pytest.mark.parametrize("cfg,B", [(configs.GRANITE_1B, 1), (configs.OLMOE, 4)],
                         ids=["granite-1b-a400m-B1", "olmoe-1b-7b-B4"])
def test_router_gate_ffn_chain_replayed_from_a_captured_graph(torch, cfg, B):
    """The device side of a layer-step with every expert resident (prefetch router, gate
    top-k, expert FFN reading the gate's executed sets from device memory) captured as one
    HIP graph: each replay, with new hidden states copied in and eager work between the
    replays, gives the eager chain's sets and outputs bit for bit."""
    d, I, E, k = cfg.d, cfg.I, cfg.E, cfg.k
    S = native.apex_expert_bytes(d, I)
    host = np.empty(E * S // 2, np.uint16)
    for e in range(E):
        w1, w3, w2 = inputs.expert_weights(cfg, 0, e)
        native.apex_pack_expert(w1, w3, w2, d, I, host[e * S // 2:])
    pool = dev(torch, host.view(np.int16))
    table = dev(torch, np.arange(E, dtype=np.int32))
    wg, wpf, bias = inputs.router_weights(cfg, 0)
    wg, wpf = dev(torch, wg.view(np.int16)), dev(torch, wpf.view(np.int16))
    bias = None if bias is None else dev(torch, bias.astype(np.float32))
    h_pre, h_post = inputs.hidden_states(cfg, 0, B, 4)
    x_pre, x_post = dev(torch, h_pre[0]), dev(torch, h_post[0])
    ws_bytes = native.apex_moe_ffn_workspace_bytes(B, d, I, k)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    i32 = dict(dtype=torch.int32, device="cuda")
    f32 = dict(dtype=torch.float32, device="cuda")

    def buffers():
        return dict(pf_idx=torch.empty((B, cfg.k_max), **i32), pf_count=torch.empty(B, **i32),
                    route_idx=torch.empty((B, k), **i32), route_gate=torch.empty((B, k), **f32),
                    exec_idx=torch.empty((B, k), **i32), exec_gate=torch.empty((B, k), **f32),
                    y=torch.empty((B, d), **f32))

    def chain(o, s):
        native.apex_prefetch_route(x_pre, wpf, bias, B, d, E, k, cfg.k_max,
                                   native.SEL_CUMPROB, cfg.tau, 0, None, None, o["pf_idx"],
                                   o["pf_count"], None, s)
        native.apex_gate_topk(x_post, wg, bias, B, d, E, k, native.MODE_EXACT, None, 0,
                              o["route_idx"], o["route_gate"], o["exec_idx"], o["exec_gate"],
                              None, s)
        native.apex_moe_ffn(x_post, B, d, I, E, k, o["exec_idx"], o["exec_gate"], table, pool,
                            E, o["y"], 0, ws, ws_bytes, s)

    graph_out, eager_out = buffers(), buffers()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        chain(graph_out, side.cuda_stream)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        chain(graph_out, side.cuda_stream)
    torch.cuda.synchronize()
    for t in range(1, 4):
        x_pre.copy_(dev(torch, h_pre[t]))
        x_post.copy_(dev(torch, h_post[t]))
        for v in graph_out.values():
            v.fill_(-7)
        graph.replay()
        torch.cuda.synchronize()
        chain(eager_out, torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        for name in graph_out:
            assert torch.equal(graph_out[name], eager_out[name]), (name, t)
        assert (graph_out["exec_idx"] >= 0).all()
    del graph

"""End-to-end decode parity: the runner's per-layer results against the oracle.

Teacher-forced where the result depends on history: the oracle's cache replay is fed
the GPU's prefetched sets (identical to the oracle's except at counted near ties), and
the oracle FFN is evaluated on the GPU's executed sets and gates, which are checked
against the oracle's own separately.

The driver's counters (overlap, full coverage, cache hits, delta_hat, copies, misses)
are checked against the oracle's metric definitions (Sec. V-C overlap accuracy; Eq. 2
full coverage; Eq. 9 delta_hat) on the oracle's own sets: exactly, except that each
(token, layer) row where a near tie let the GPU's sets differ may move each sum by at
most one.
"""
import numpy as np
import pytest

from oracle import decode as odecode
from oracle import ffn as offn
from oracle import gating, metrics, routing
from oracle.residency import Residency
from paper_2608_11688_amd import configs, inputs, native
from tests.parity import TIE, TieLedger, ffn_close


class Counters:
    """The driver's apex_decode_stats, accumulated from the oracle's metric functions."""

    FIELDS = ("tokens", "layer_steps", "copies", "misses", "coverage_count", "delta_hat_sum",
              "overlap_sum", "hit_sum")

    def __init__(self):
        self.v = dict.fromkeys(self.FIELDS, 0)
        self.v["overlap_sum"] = self.v["hit_sum"] = 0.0
        self.loose_rows = 0        # rows whose sets may differ from the GPU's (near ties)

    def add_layer_step(self, k, pf_lists, route_idx, resident, copies, misses):
        for b, pf in enumerate(pf_lists):
            routed = [int(e) for e in route_idx[b]]
            self.v["overlap_sum"] += metrics.overlap(routed, pf, k)
            self.v["coverage_count"] += int(metrics.full_coverage(routed, pf))
            self.v["hit_sum"] += len(set(routed) & set(resident)) / k
            self.v["delta_hat_sum"] += max(len(pf) - k, 0)
            self.v["tokens"] += 1
        self.v["layer_steps"] += 1
        self.v["copies"] += copies
        self.v["misses"] += misses

    def check(self, stats, what=""):
        got = {f: getattr(stats, f) for f in self.FIELDS}
        slack = self.loose_rows
        for f in self.FIELDS:
            tol = slack + (1e-9 * max(1, self.v["tokens"]) if f.endswith("_sum") else 0)
            assert abs(got[f] - self.v[f]) <= tol, (what, f, got[f], self.v[f], slack)
        return got

pytestmark = pytest.mark.gpu


def check_decode(cfg, batch, mode, steps, layers, policy=native.SEL_CUMPROB, tau=None,
                 ffn_every=1, cdf=None, weights="bf16", window="spin", ffn_at=None):
    """cdf: {layer: (w, theta)} for the ORDINAL policy; seeded random models if None.
    ffn_at: the (step, layer) pairs whose FFN output is checked, instead of every
    ffn_every-th one."""
    from paper_2608_11688_amd.runtime import DecodeRunner
    tau = cfg.tau if tau is None else tau
    tau32 = float(np.float32(tau))
    runner = DecodeRunner(cfg, batch=batch, mode=mode, tau=tau32, policy=policy, steps=steps,
                          layers=layers, t_attn_us=2.0, record=True, cdf=cdf, weights=weights,
                          window=window, ctx=128)
    ledger = TieLedger()
    oracle_counts = Counters()
    res = {l: Residency(cfg.E, cfg.C) for l in layers}
    routers = {l: inputs.router_weights(cfg, l) for l in layers}
    hs = {l: inputs.hidden_states(cfg, l, batch, steps) for l in layers}
    cdfs = cdf if cdf is not None else {l: inputs.cdf_params(cfg, l) for l in layers}
    stats = dict(copies=0, misses=0, ffn_checked=0, worst_l1=0.0, covered=0, tokens=0)
    bits_cache = {}

    def expert_bits(l, e):
        if (l, e) not in bits_cache:
            bits_cache[(l, e)] = inputs.expert_weights(cfg, l, e)
        return bits_cache[(l, e)]
    try:
        for t in range(steps):
            logs = runner.step()
            for l in layers:
                log = logs[l]
                wg, wpf, bias = routers[l]
                h_pre, h_post = hs[l][0][t], hs[l][1][t]
                cw, ct = cdfs[l] if policy == native.SEL_ORDINAL_CDF else (None, None)
                r = routing.prefetch_route(h_pre, wpf, bias, cfg.k, cfg.k_max, policy, tau32, 0,
                                           cw, ct)
                ledger.compare_rows(log.pf_count[:, None], r["pf_count"][:, None], r["margin"],
                                    f"pf_count t{t} l{l}")
                ledger.compare_rows(log.pf_idx, r["pf_idx"], r["margin"], f"pf_idx t{t} l{l}")
                lists = [list(log.pf_idx[b, :log.pf_count[b]]) for b in range(batch)]
                copies = res[l].plan(lists, t)
                R = res[l].resident()
                assert sorted(R) == log.resident, (t, l)
                assert len(copies) == log.copies, (t, l)
                avail = np.array([e in R for e in range(cfg.E)])
                g = gating.gate_topk(h_post, wg, bias, cfg.k, mode, avail)
                ledger.compare_rows(log.route_idx, g["route_idx"], g["margin"], f"route t{t} l{l}")
                ledger.compare_rows(log.exec_idx, g["exec_idx"], g["margin"], f"exec t{t} l{l}")
                for b in range(batch):
                    stats["covered"] += set(log.route_idx[b]) <= set(lists[b])
                stats["tokens"] += batch
                if mode == native.MODE_EXACT:
                    want = sorted(set(int(e) for e in log.route_idx.ravel()) - R)
                    assert log.missing == want, (t, l, log.missing, want)
                    stats["misses"] += len(want)
                else:
                    assert set(int(e) for e in log.exec_idx.ravel() if e >= 0) <= R
                stats["copies"] += log.copies
                # the metrics on the oracle's own sets (the cache replay is teacher-forced)
                o_lists = [list(r["pf_idx"][b, :r["pf_count"][b]]) for b in range(batch)]
                o_miss = set(int(e) for e in g["route_idx"].ravel()) - R
                oracle_counts.add_layer_step(
                    cfg.k, o_lists, g["route_idx"], R, len(copies),
                    len(o_miss) if mode == native.MODE_EXACT else 0)
                oracle_counts.loose_rows += sum(
                    int(not (np.array_equal(log.pf_idx[b], r["pf_idx"][b]) and
                             np.array_equal(log.route_idx[b], g["route_idx"][b])))
                    for b in range(batch))
                if ((t, l) in ffn_at if ffn_at is not None
                        else (t * len(layers) + layers.index(l)) % ffn_every == 0):
                    bits = lambda e, l=l: expert_bits(l, e)
                    y_ref = offn.moe_ffn(h_post, log.exec_idx, log.exec_gate.astype(np.float64),
                                         bits, weights=weights)
                    if cfg.shared:
                        sbits = lambda s, l=l: inputs.shared_expert_weights(cfg, l, s)
                        y_ref = y_ref + odecode.shared_ffn(h_post, cfg.shared, sbits, weights)
                    _, l1 = ffn_close(log.y, y_ref, f"y t{t} l{l}")
                    stats["worst_l1"] = max(stats["worst_l1"], l1)
                    stats["ffn_checked"] += 1
        runner.finish()
        stats["counters"] = oracle_counts.check(runner.stats, f"{cfg.name} B{batch} mode {mode}")
    finally:
        runner.close()
    print(cfg.name, batch, mode, ledger, stats)
    return stats


def oracle_counters(cfg, batch, mode, steps, layers, policy, tau, empty=None):
    """Counters of the oracle's own decode replay (no teacher forcing) and the number of
    (token, layer) rows where a near tie could let the GPU decide differently.

    empty: {layer: experts} whose slots start empty instead of holding them; the first
    step after which each layer holds all E experts is left in ``full_at``."""
    from oracle import decode as odec
    c = Counters()
    states = odec.make_states(cfg, layers, policy=policy)
    for l, experts in (empty or {}).items():
        eos = states[l].res.expert_of_slot
        for e in experts:
            eos[eos.index(e)] = -1
    c.full_at = {}
    for t, l, out in odec.run(cfg, batch, steps, mode=mode, tau=tau, layers=layers,
                              run_ffn=False, policy=policy, states=states):
        if len(out["resident"]) == cfg.E:
            c.full_at.setdefault(l, t)
        pf = [list(out["route"]["pf_idx"][b, :out["route"]["pf_count"][b]])
              for b in range(batch)]
        c.add_layer_step(cfg.k, pf, out["gate"]["route_idx"], out["resident"],
                         len(out["copies"]), len(out["misses"]))
        near = (out["route"]["margin"] < TIE) | (out["gate"]["margin"] < TIE)
        c.loose_rows += int(near.sum())
    return c


@pytest.mark.parametrize("mode", [native.MODE_EXACT, native.MODE_STALL_FREE])
def test_decode_tiny_all_steps(mode):
    cfg = configs.TINY
    st = check_decode(cfg, 1, mode, cfg.steps, [0])
    assert st["copies"] > 0


@pytest.mark.parametrize("mode", [native.MODE_EXACT, native.MODE_STALL_FREE])
def test_decode_no_prefetch_baseline(mode):
    # nothing is prefetched: the cache keeps its initial experts, exact mode loads every
    # other routed expert after the gate, stall-free mode runs on the initial experts
    cfg = configs.GRANITE_1B
    st = check_decode(cfg, 1, mode, 6, [0, 13], policy=native.SEL_NONE)
    assert st["copies"] == 0 and st["covered"] == 0
    if mode == native.MODE_EXACT:
        assert st["misses"] > 0


def test_decode_granite1b_exact():
    cfg = configs.GRANITE_1B
    st = check_decode(cfg, 1, native.MODE_EXACT, 4, list(range(cfg.L)), ffn_every=3)
    assert st["copies"] > 0


def test_decode_mixtral_shape_exact_with_a_miss():
    # 352 MB experts through the whole path: the copy kernel's wide grid for the prefetch
    # (a copy at every step of these layers) and for the miss fetch (layer 2 misses
    # expert 7 at step 4), the second FFN pass over the scratch pool
    cfg = configs.MIXTRAL
    st = check_decode(cfg, 1, native.MODE_EXACT, 5, [2, 5], ffn_at={(4, 2), (1, 5)})
    assert st["copies"] > 0 and st["misses"] >= 1 and st["ffn_checked"] == 2


def test_decode_granite3b_batch8_stall_free_ordinal():
    cfg = configs.GRANITE_3B
    check_decode(cfg, 8, native.MODE_STALL_FREE, 3, [0, 17, 31],
                 policy=native.SEL_ORDINAL_CDF)


def test_decode_olmoe_batch16_exact():
    cfg = configs.OLMOE
    check_decode(cfg, 16, native.MODE_EXACT, 3, [0, 9], ffn_every=2)


def test_decode_granite1b_ordinal_fitted_model():
    # per-layer models fitted on held-out tokens (training stage on the GPU kernels), then
    # decoding with them; the oracle replays the same fitted parameters
    from paper_2608_11688_amd import cdf_fit
    cfg = configs.GRANITE_1B
    layers = [0, 11, 23]
    params, report = cdf_fit.fit_model(cfg, tokens=512, layers=layers)
    st = check_decode(cfg, 1, native.MODE_EXACT, 8, layers, policy=native.SEL_ORDINAL_CDF,
                      tau=0.9, cdf=params)
    print(report, st)
    # calibrated at tau = 0.9 on held-out tokens: most of these tokens are fully covered
    assert st["covered"] >= 0.6 * st["tokens"]


def test_decode_every_expert_resident():
    # C = E: the cache holds every expert from the start, so nothing is ever copied or
    # missed, and stall-free mode executes exactly the routed sets
    cfg = configs.MoEConfig("all_resident", 420, L=2, d=256, E=8, k=2, I=128, C=8, k_max=8,
                            tau=0.9, steps=12)
    for mode in (native.MODE_EXACT, native.MODE_STALL_FREE):
        st = check_decode(cfg, 2, mode, 12, [0, 1])
        assert st["copies"] == 0 and st["misses"] == 0


def test_decode_every_expert_routed():
    # k = E: every token routes to every expert; the prefetched set is the whole list
    # (m is clamped to k = k_max = E), so every token is fully covered
    cfg = configs.MoEConfig("all_routed", 421, L=1, d=264, E=4, k=4, I=136, C=4, k_max=4,
                            tau=0.5, steps=10)
    for mode in (native.MODE_EXACT, native.MODE_STALL_FREE):
        st = check_decode(cfg, 3, mode, 10, [0])
        assert st["covered"] == st["tokens"] and st["copies"] == 0


@pytest.mark.parametrize("mode", [native.MODE_EXACT, native.MODE_STALL_FREE])
def test_decode_granite1b_fp8_experts(mode):
    # E4M3 experts through prefetch, miss correction and both FFN passes
    cfg = configs.GRANITE_1B
    st = check_decode(cfg, 1, mode, 4, [0, 7, 23], weights="fp8")
    assert st["copies"] > 0


def test_decode_olmoe_batch16_fp8_experts():
    cfg = configs.OLMOE
    check_decode(cfg, 16, native.MODE_EXACT, 2, [3], ffn_every=1, weights="fp8")


def test_decode_with_attention_window():
    # the window is the layers' real decode attention: the MoE path is unchanged, and every
    # step's attention output matches the oracle's block on the same caches
    from oracle import attention as oatt
    from paper_2608_11688_amd.runtime import DecodeRunner
    cfg = configs.GRANITE_1B
    check_decode(cfg, 1, native.MODE_EXACT, 3, [0, 11], window="attention")
    layers, steps, ctx, B = [2, 17], 3, 200, 2
    H, G, hd = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    runner = DecodeRunner(cfg, batch=B, mode=native.MODE_STALL_FREE, steps=steps, layers=layers,
                          record=True, window="attention", ctx=ctx)
    try:
        caches = {l: tuple(runner.bufs[l][n].cpu().numpy().view(np.uint16)
                           for n in ("k_cache", "v_cache")) for l in layers}
        weights = {l: inputs.attention_weights(cfg, l) for l in layers}
        hs = {l: inputs.hidden_states(cfg, l, B, steps)[0] for l in layers}
        worst = 0.0
        for t in range(steps):
            runner.step()
            for l in layers:
                got = runner.bufs[l]["attn_out"].cpu().numpy().astype(np.float64)
                ref = oatt.attention_block(hs[l][t], *weights[l], *caches[l], H, G, hd, ctx)["o"]
                err = np.abs(got - ref).max() / np.abs(ref).max()
                assert err <= 1e-4, (t, l, err)
                worst = max(worst, err)
        print("attention window worst rel err", worst)
    finally:
        runner.close()


@pytest.mark.parametrize("batch,mode", [(1, native.MODE_EXACT), (16, native.MODE_STALL_FREE)])
def test_decode_deepseek_shape_with_shared_experts(batch, mode):
    # 64 routed experts (k = 6) plus two shared experts that every token runs with weight 1,
    # before the routed experts' copies land; batch 16 takes the grouped path for both
    cfg = configs.DEEPSEEK_16B
    st = check_decode(cfg, batch, mode, 3, [0, 25])
    assert st["ffn_checked"] > 0


SMALL_SHARED = configs.MoEConfig("small_shared", 421, L=2, d=512, E=16, k=4, I=256, C=8,
                                k_max=8, tau=0.9, steps=8, shared=2)


@pytest.mark.parametrize("mode", [native.MODE_EXACT, native.MODE_STALL_FREE])
def test_decode_small_experts_with_shared_experts(mode):
    # experts of 0.79 MB (short copies) with two shared experts, which run on the side
    # stream while a layer-step's copies are in flight and are waited for with an event;
    # parity with records, then the unrecorded timeline against the recorded one
    cfg = SMALL_SHARED
    st = check_decode(cfg, 1, mode, cfg.steps, [0, 1])
    assert st["copies"] > 0 and st["ffn_checked"] > 0
    (y_free, c_free, _, _), (y_rec, c_rec, _, _) = run_unrecorded_and_recorded(cfg, 1, mode,
                                                                          cfg.steps, [0, 1])
    assert c_free == c_rec
    assert np.abs(y_free - y_rec).max() <= 1e-5 * np.abs(y_rec).max()


def empty_slots(runner, empty):
    """Empties, before the first step, the slots of the given {layer: experts}: the host
    table, the device table and the availability mask the driver reads."""
    torch = runner.torch
    for l, experts in empty.items():
        b = runner.bufs[l]
        for e in experts:
            b["eos"][int(np.flatnonzero(b["eos"] == e)[0])] = -1
        table = np.full(runner.cfg.E, -1, np.int32)
        for s, e in enumerate(b["eos"]):
            if e >= 0:
                table[e] = s
        b["slot_dev"].copy_(torch.from_numpy(table))
        b["avail_dev"].copy_(torch.from_numpy((table >= 0).astype(np.uint8)))
    torch.cuda.synchronize()


def run_unrecorded_and_recorded(cfg, batch, mode, steps, layers, policy=native.SEL_CUMPROB,
                                empty=None, window="spin"):
    """Final outputs and counters of the same decode without and with per-layer records
    (empty: {layer: experts} whose slots start empty)."""
    from paper_2608_11688_amd.runtime import DecodeRunner
    out = []
    for record in (False, True):
        runner = DecodeRunner(cfg, batch=batch, mode=mode, tau=float(np.float32(cfg.tau)),
                              policy=policy, steps=steps, layers=layers, t_attn_us=2.0,
                              record=record, window=window, ctx=256)
        try:
            if empty:
                empty_slots(runner, empty)
            for _ in range(steps):
                runner.step()
            runner.finish()
            s = runner.stats
            counts = tuple(getattr(s, f) for f in Counters.FIELDS)
            lu = {l: runner.bufs[l]["last_used"].copy() for l in runner.layers}
            out.append((runner.y.cpu().numpy().copy(), counts, s, lu))
        finally:
            runner.close()
    return out


@pytest.mark.parametrize("cfg_name,batch,mode,layers,policy", [
    ("GRANITE_1B", 1, native.MODE_EXACT, None, native.SEL_CUMPROB),
    ("GRANITE_1B", 1, native.MODE_STALL_FREE, None, native.SEL_CUMPROB),
    ("OLMOE", 16, native.MODE_EXACT, [0, 5, 9, 15], native.SEL_CUMPROB),
    ("DEEPSEEK_16B", 1, native.MODE_EXACT, [0, 12, 25], native.SEL_CUMPROB),
    # no router: in stall-free mode nothing orders the gate before the counters are
    # folded except the poll of the stream it ran on
    ("GRANITE_1B", 1, native.MODE_STALL_FREE, None, native.SEL_NONE),
    ("OLMOE", 16, native.MODE_EXACT, [2, 11], native.SEL_NONE),
], ids=["g1-exact", "g1-stall-free", "olmoe-b16-exact", "deepseek-exact", "g1-none-stall-free",
        "olmoe-b16-none-exact"])
def test_decode_without_records_matches_recorded(cfg_name, batch, mode, layers, policy):
    # The parity tests above record every layer, which synchronizes the host with the
    # device after each one; the timed path does not, and there the copies, the window,
    # the gate and the FFN overlap across the two streams.  Same inputs, same state: the
    # counters must agree exactly and the last step's outputs to rounding.  The counters
    # of the timed path must also equal the oracle's own replay: these inputs have no
    # near tie, so the oracle's decisions are the GPU's.
    cfg = getattr(configs, cfg_name)
    layers = list(range(cfg.L)) if layers is None else layers
    steps = 6
    (y_free, c_free, s_free, _), (y_rec, c_rec, _, _) = run_unrecorded_and_recorded(
        cfg, batch, mode, steps, layers, policy)
    assert c_free == c_rec
    if policy == native.SEL_NONE:
        assert c_free[2] == 0 and s_free.overlap_sum == 0 and s_free.delta_hat_sum == 0
    else:
        assert c_free[2] > 0                    # copies happened
    scale = np.abs(y_rec).max()
    assert scale > 0
    assert np.abs(y_free - y_rec).max() <= 1e-5 * scale
    ref = oracle_counters(cfg, batch, mode, steps, layers, policy, float(np.float32(cfg.tau)))
    assert ref.loose_rows == 0
    print(cfg_name, ref.check(s_free, "unrecorded vs oracle"))


@pytest.mark.parametrize("batch,mode", [(1, native.MODE_EXACT), (8, native.MODE_STALL_FREE)])
def test_decode_phi_shape(batch, mode):
    cfg = configs.PHI_7B
    st = check_decode(cfg, batch, mode, 3, [0, 31])
    assert st["ffn_checked"] > 0


def test_decode_deepseek_shape_fp8_shared_experts():
    # the shared pool is packed in the layer's weight format as well
    check_decode(configs.DEEPSEEK_16B, 1, native.MODE_EXACT, 2, [7], weights="fp8")


def test_decode_granite1b_mxfp4_experts():
    # 4-bit experts through the whole decode path: packing, prefetch copies, misses, FFN
    cfg = configs.GRANITE_1B
    st = check_decode(cfg, 1, native.MODE_EXACT, 4, [0, 23], weights="mxfp4")
    assert st["copies"] > 0


def test_decode_deepseek_shape_mxfp4_batch16():
    check_decode(configs.DEEPSEEK_16B, 16, native.MODE_STALL_FREE, 2, [4], weights="mxfp4")


def test_decode_granite1b_fp32_experts():
    # 32-bit experts through the whole decode path: twice the bytes of every copy
    cfg = configs.GRANITE_1B
    st = check_decode(cfg, 1, native.MODE_EXACT, 4, [0, 23], weights="fp32")
    assert st["copies"] > 0


def test_decode_create_rejects_bad_configurations():
    # validation happens before anything is allocated or enqueued
    from paper_2608_11688_amd.runtime import DecodeRunner
    import dataclasses
    cfg = configs.MoEConfig("val", 450, L=1, d=256, E=8, k=2, I=96, C=4, k_max=4, tau=0.9,
                            steps=2)
    # MXFP4 needs d and I multiples of 32 (I = 96 is; 80 is not)
    bad_i = dataclasses.replace(cfg, I=80)
    with pytest.raises(native.ApexError):
        DecodeRunner(bad_i, batch=1, steps=1, weights="mxfp4")
    # 32-bit experts run at batch 1 only
    with pytest.raises(native.ApexError) as ei:
        DecodeRunner(cfg, batch=2, steps=1, weights="fp32")
    assert ei.value.status == native.APEX_E_UNSUPPORTED
    # shared experts need an intermediate size that fits the weight format
    bad_shared = dataclasses.replace(cfg, shared=1, I_shared=40)
    with pytest.raises(native.ApexError):
        DecodeRunner(bad_shared, batch=1, steps=1, weights="fp8")
    # more pinned host experts than the runner holds: refused before anything is drawn
    with pytest.raises(ValueError, match="pinned host memory"):
        DecodeRunner(configs.MIXTRAL, batch=1, steps=1, weights="fp32")
    # a good configuration still builds and steps
    r = DecodeRunner(dataclasses.replace(cfg, shared=1, I_shared=64), batch=1, steps=1,
                     weights="mxfp4")
    try:
        r.step()
        r.finish()
    finally:
        r.close()


@pytest.mark.parametrize("cfg,batch,mode,layers,weights", [
    (configs.GRANITE_1B, 1, native.MODE_EXACT, [0, 23], "bf16"),
    (configs.GRANITE_3B, 1, native.MODE_STALL_FREE, [7], "bf16"),
    (configs.OLMOE, 1, native.MODE_EXACT, [4], "bf16"),
    (configs.GRANITE_3B, 8, native.MODE_EXACT, [30], "bf16"),
    (configs.DEEPSEEK_16B, 1, native.MODE_STALL_FREE, [12], "bf16"),
    (configs.PHI_7B, 1, native.MODE_EXACT, [3], "fp8"),
    (configs.GRANITE_1B, 1, native.MODE_EXACT, [9], "mxfp4"),
], ids=["granite-1b-a400m-exact", "granite-3b-a800m-stall-free", "olmoe-1b-7b-exact",
        "granite-3b-a800m-B8-exact", "deepseek-16b-shared-stall-free", "phi-7b-fp8-exact",
        "granite-1b-a400m-mxfp4-exact"])
def test_decode_every_step_of_the_workload(cfg, batch, mode, layers, weights):
    """Every decode step of the workload (256) on some of its layers: after hundreds of
    cache plans (eviction by last use, ties between equal last uses; at batch 8 the union
    of the tokens' sets) the resident sets, the prefetched, routed and executed sets, the
    misses and the driver's counters still match the oracle's replay; the FFN output
    (with DeepSeek's shared experts, and over E4M3 or MXFP4 slots) is checked every 64th
    layer-step."""
    st = check_decode(cfg, batch, mode, cfg.steps, layers, ffn_every=64, weights=weights)
    assert st["copies"] > 0 and st["ffn_checked"] >= 4


def test_decode_mixtral_shape_first_16_steps():
    """Steps 0-15 of a Mixtral-shaped layer: a 352 MB expert copied at most steps, the
    sets and cache state against the oracle at every step, the FFN output at the last."""
    cfg = configs.MIXTRAL
    st = check_decode(cfg, 1, native.MODE_EXACT, 16, [6], ffn_at={(15, 6)})
    assert st["copies"] > 0 and st["ffn_checked"] == 1


@pytest.mark.parametrize("cfg_name,batch,mode,layers,policy,window", [
    ("GRANITE_1B", 1, native.MODE_EXACT, None, native.SEL_CUMPROB, "spin"),
    ("GRANITE_1B", 1, native.MODE_STALL_FREE, [0, 7, 23], native.SEL_ORDINAL_CDF, "spin"),
    ("GRANITE_1B", 1, native.MODE_EXACT, [3, 4], native.SEL_NONE, "spin"),
    ("DEEPSEEK_16B", 2, native.MODE_EXACT, [0, 12], native.SEL_CUMPROB, "spin"),
    ("OLMOE", 4, native.MODE_STALL_FREE, [1, 9], native.SEL_CUMPROB, "attention"),
], ids=["g1-exact", "g1-stall-free-ordinal", "g1-none", "deepseek-b2-shared",
        "olmoe-b4-attention"])
def test_decode_with_every_expert_resident_skips_the_host_waits(cfg_name, batch, mode, layers,
                                                                policy, window):
    """Every expert resident (C = E): the timed path queues router, window (the spin, or
    the layer's decode attention), gate, shared experts and FFN without waiting for the
    host and folds the statistics later; the recorded path takes the general route.
    Counters, outputs and the host's last-use table agree, and the counters equal the
    oracle's replay."""
    import dataclasses
    base = getattr(configs, cfg_name)
    cfg = dataclasses.replace(base, C=base.E)
    layers = list(range(cfg.L)) if layers is None else layers
    steps = 6
    (y_free, c_free, s_free, lu_free), (y_rec, c_rec, _, lu_rec) = run_unrecorded_and_recorded(
        cfg, batch, mode, steps, layers, policy, window=window)
    assert c_free == c_rec
    assert s_free.copies == 0 and s_free.misses == 0
    for l in layers:
        assert np.array_equal(lu_free[l], lu_rec[l]), l
    scale = np.abs(y_rec).max()
    assert scale > 0
    assert np.abs(y_free - y_rec).max() <= 1e-5 * scale
    if policy != native.SEL_ORDINAL_CDF:      # the oracle replay draws its own CDF models
        ref = oracle_counters(cfg, batch, mode, steps, layers, policy,
                              float(np.float32(cfg.tau)))
        ref.check(s_free, "unrecorded, every expert resident, vs oracle")


@pytest.mark.parametrize("cfg_name,batch,mode,empty", [
    ("TINY", 1, native.MODE_EXACT, {0: [4, 0]}),
    ("TINY", 1, native.MODE_STALL_FREE, {0: [4, 0]}),
    ("GRANITE_1B", 1, native.MODE_EXACT, {1: [30, 14, 29, 11], 5: [3, 19, 30]}),
    ("GRANITE_1B", 1, native.MODE_STALL_FREE, {1: [30, 14, 29, 11], 5: [3, 19, 30]}),
], ids=["tiny-exact", "tiny-stall-free", "g1-exact", "g1-stall-free"])
def test_decode_fills_empty_slots_then_skips_the_host_waits(cfg_name, batch, mode, empty):
    """C = E with some slots empty at the start: the layers take the general route, whose
    cache plan fills the empty slots as the experts enter prefetched sets, then the route
    without host waits, each layer from its own step on.  Against the recorded run (always
    the general route) and the oracle's replay from the same initial cache."""
    import dataclasses
    base = getattr(configs, cfg_name)
    cfg = dataclasses.replace(base, C=base.E)
    layers = sorted(empty)
    steps = 12
    tau = float(np.float32(cfg.tau))
    ref = oracle_counters(cfg, batch, mode, steps, layers, native.SEL_CUMPROB, tau, empty)
    assert ref.loose_rows == 0
    # every layer switches routes with steps to spare
    assert all(0 < ref.full_at.get(l, steps) < steps - 2 for l in layers), ref.full_at
    (y_free, c_free, s_free, lu_free), (y_rec, c_rec, _, lu_rec) = run_unrecorded_and_recorded(
        cfg, batch, mode, steps, layers, native.SEL_CUMPROB, empty)
    assert c_free == c_rec
    assert s_free.copies == sum(len(v) for v in empty.values())
    for l in layers:
        assert np.array_equal(lu_free[l], lu_rec[l]), l
    scale = np.abs(y_rec).max()
    assert scale > 0
    assert np.abs(y_free - y_rec).max() <= 1e-5 * scale
    print(cfg_name, ref.full_at, ref.check(s_free, "unrecorded, slots filled, vs oracle"))

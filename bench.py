#!/usr/bin/env python3
"""Benchmark of the MoE-decode hot path on one MI355X.

One step = one decode token (batch B) through every MoE layer of the workload:
prefetch router + adaptive K_p, cache plan + host-to-HBM expert copies (a copy kernel
on the compute stream, which the attention window and the gate run beside on the side
stream), the attention window (a spin of --t-attn-us, or with --window attention the
layer's real decode attention), gate top-k (correctness-preserving mode by default),
expert FFN over the HBM slots, miss correction (its copies on the side stream).  Inputs
(hidden states, routers, the HBM slot pools and the pinned host copy of every expert) are
resident before timing.

Prints one JSON line.  ``value`` is microseconds per token per MoE layer of the decode
timeline with the attention window subtracted (the spin's length, or the attention
block's measured device time): the MoE path's own cost including exposed stall; lower
is better.  The same timeline with every expert resident in HBM (no copies, no misses)
is timed after it; the difference is the exposed stall.

    python bench.py [--steps K] [--warmup W] [--config mixtral-8x7b] [--batch 1]
                    [--mode exact|stall_free] [--policy cumprob|ordinal|static|none]
                    [--static-delta D] [--tau T] [--weights bf16|fp8|mxfp4|fp32]
                    [--window spin|attention] [--t-attn-us 10] [--ctx 1024]
                    [--no-compute-only] [--no-cpu-baseline]

The default workload is the largest that fits one GPU: eight Mixtral-8x7B-shaped MoE
layers (d 4096, 8 experts of intermediate size 14336, top-2, 4 experts resident per
layer), batch 1, bf16 experts, correctness-preserving mode.

With --policy ordinal, every layer's coverage model is first fitted on held-out tokens
(the method's training stage, outside the timed region).
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import gc
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
# PCIe 5.0 x16, one direction: 32 GT/s x 16 lanes with 128b/130b encoding
PCIE_PEAK_GBPS = 32.0 * 16 * 128 / 130 / 8
# the kernels of one FFN call, per weight format, at batch 1 and at batch >= 2
FFN_KERNELS = {
    ("bf16", True): "apex_moe_ffn (up_sk or up_b1, then down_b1)",
    ("fp8", True): "apex_moe_ffn_fp8 (up_sk_e4m3 or up_b1_e4m3, then down_b1_e4m3)",
    ("mxfp4", True): "apex_moe_ffn_mxfp4 (up_sk_mxfp4 or up_b1_mxfp4, then down_b1_mxfp4 or "
                     "down_rows_mxfp4)",
    ("fp32", True): "apex_moe_ffn_fp32 (up_sk_f32 or up_b1_f32, then down_f32)",
    ("bf16", False): "apex_moe_ffn (up_gemm + down_gemm + combine_pairs)",
    ("fp8", False): "apex_moe_ffn_fp8 (up_gemm + down_gemm + combine_pairs, E4M3 tiles)",
    ("mxfp4", False): "apex_moe_ffn_mxfp4 (up_gemm + down_gemm + combine_pairs, MXFP4 tiles)",
}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=128)
    p.add_argument("--warmup", type=int, default=8)
    p.add_argument("--config", default="mixtral-8x7b")
    p.add_argument("--batch", type=int, default=1)
    p.add_argument("--mode", default="exact", choices=["exact", "stall_free"])
    p.add_argument("--tau", type=float, default=None)
    p.add_argument("--policy", default="cumprob",
                   choices=["cumprob", "ordinal", "static", "none"])
    p.add_argument("--static-delta", type=int, default=0)
    p.add_argument("--weights", default="bf16", choices=["bf16", "fp8", "mxfp4", "fp32"],
                   help="expert weight format (fp8: E4M3 with fp32 row scales; mxfp4: E2M1 "
                        "with a power-of-two scale per block of 32; fp32: the bf16 experts "
                        "stored as fp32, batch 1 only)")
    p.add_argument("--cdf-tokens", type=int, default=1024,
                   help="held-out tokens per layer for the ordinal-model fit")
    p.add_argument("--t-attn-us", type=float, default=10.0,
                   help="length of the spin that stands in for attention (--window spin)")
    p.add_argument("--window", default="spin", choices=["spin", "attention"],
                   help="attention window: a spin of --t-attn-us, or the layers' real decode "
                        "attention over --ctx cached positions")
    p.add_argument("--ctx", type=int, default=1024)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-compute-only", action="store_true",
                   help="skip the all-resident run that the exposed stall is measured against")
    p.add_argument("--cpu-budget-s", type=float, default=15.0)
    p.add_argument("--cpu-1thread-budget-s", type=float, default=6.0,
                   help="seconds of the oracle under one BLAS thread (0: skip)")
    return p.parse_args()


def pinned_h2d_peak(torch, nbytes=1 << 30, reps=3):
    src = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    dst = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst.copy_(src, non_blocking=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        dst.copy_(src, non_blocking=True)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / reps
    del src, dst
    return nbytes / dt / 1e9


def expert_copy_leg(torch, native, expert_bytes, E, link_peak, reps=5):
    """Times the prefetch's copy kernel (apex_expert_prefetch) on a plan of n experts of
    the workload (3, or 1 when three would pass 256 MB), event pair on the copy stream
    around the call (the slot-table publish goes to another stream), against the same
    bytes moved by one DMA-engine copy per expert and against the link's pinned peak.  A
    spin kernel holds the stream while the host plans and enqueues, so the pair brackets
    device time only.
    """
    n = 3 if 3 * expert_bytes <= (256 << 20) else 1
    n = min(n, E)
    host = torch.empty(n * expert_bytes, dtype=torch.uint8, pin_memory=True)
    pool = torch.empty(n * expert_bytes, dtype=torch.uint8, device="cuda")
    slot_dev = torch.full((n,), -1, dtype=torch.int32, device="cuda")
    cs, ts = torch.cuda.Stream(), torch.cuda.Stream()
    pf_idx = np.arange(n, dtype=np.int32)[None, :]
    pf_cnt = np.array([n], np.int32)

    def timed(body):
        out = []
        for _ in range(reps + 1):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            native.apex_spin_us(100.0, cs.cuda_stream)
            e0.record(cs)
            body()
            e1.record(cs)
            e1.synchronize()
            out.append(e0.elapsed_time(e1) * 1e3)
        return float(np.median(out[1:]))

    def kernel():
        eos = np.full(n, -1, np.int32)
        lu = np.full(n, -1, np.int64)
        got = native.apex_expert_prefetch(host, pool, n, n, expert_bytes, pf_idx, pf_cnt, 1, n,
                                          0, eos, lu, slot_dev, None, cs.cuda_stream,
                                          ts.cuda_stream, None, None)
        assert got == n

    def dma():
        with torch.cuda.stream(cs):
            for i in range(n):
                a, b = i * expert_bytes, (i + 1) * expert_bytes
                pool[a:b].copy_(host[a:b], non_blocking=True)

    us_kernel, us_dma = timed(kernel), timed(dma)
    torch.cuda.synchronize()
    del host, pool
    gbps = n * expert_bytes / (us_kernel * 1e-6) / 1e9
    return {"kernel": "expert_copy_kernel", "experts": n, "bytes": n * expert_bytes,
            "us": round(us_kernel, 2), "GBps": round(gbps, 2),
            "dma_per_expert_us": round(us_dma, 2),
            "link_peak_GBps": round(link_peak, 2),
            "frac_of_link_peak": round(gbps / link_peak, 4),
            "published_link_GBps": round(PCIE_PEAK_GBPS, 2),
            "frac_of_published_link": round(gbps / PCIE_PEAK_GBPS, 4)}


def ffn_roofline_leg(torch, native, runner, reps=8, seed=123):
    """Times apex_moe_ffn in the decode timeline's launch configuration.

    Every layer's slot pool is used in turn (together far larger than the 256 MB
    Infinity Cache, so weights stream from HBM); each launch executes k resident
    experts per token.  A spin kernel holds the stream while the host enqueues, then
    one event pair brackets the whole queued batch, so the average per launch is device
    time only (both kernels of a call and the gap between them).
    Returns (mean ms per launch, algorithmic bytes per launch, launches).
    """
    cfg, B, k = runner.cfg, runner.B, runner.cfg.k
    rng = np.random.default_rng(seed)
    cs = runner.cs
    plan = []
    for l in runner.layers:
        b = runner.bufs[l]
        table = b["slot_dev"].cpu().numpy()
        resident = np.flatnonzero(table >= 0)
        idx = np.stack([rng.choice(resident, k, replace=False) for _ in range(B)]).astype(np.int32)
        g = rng.random((B, k)) + 0.1
        gate = (g / g.sum(1, keepdims=True)).astype(np.float32)
        n_exp = len(set(idx.ravel().tolist()))
        plan.append((b, torch.from_numpy(idx).cuda(), torch.from_numpy(gate).cuda(), n_exp))
    n = reps * len(plan)
    y = torch.empty((B, cfg.d), dtype=torch.float32, device="cuda")
    e0, e1 = native.apex_event_create(True), native.apex_event_create(True)
    torch.cuda.synchronize()
    ffn = runner.moe_ffn
    native.apex_spin_us(min(5000.0 + 50.0 * n, 1e6), cs)
    native.apex_event_record(e0, cs)
    for i in range(n):
        b, idx, gate, _ = plan[i % len(plan)]
        ffn(b["h_post"][0], B, cfg.d, cfg.I, cfg.E, k, idx, gate, b["slot_dev"], b["slots"],
            cfg.C, y, 0, runner.ws, runner.ws_bytes, cs)
    native.apex_event_record(e1, cs)
    native.apex_event_synchronize(e1)
    ms = native.apex_event_elapsed_ms(e0, e1) / n
    native.apex_event_destroy(e0)
    native.apex_event_destroy(e1)
    nbytes = float(np.mean([plan[i % len(plan)][3] * runner.S + 2 * B * cfg.d * 4
                            for i in range(n)]))
    return ms, nbytes, n


def router_leg(torch, native, runner, reps=8):
    """Device time of the prefetch router (apex_prefetch_route with the bench's policy) on
    every layer's weights in turn, queued behind a spin kernel, one event pair around
    them.  Returns us per call."""
    cfg, B = runner.cfg, runner.B
    pf_idx = torch.empty((B, cfg.k_max), dtype=torch.int32, device="cuda")
    pf_count = torch.empty((B,), dtype=torch.int32, device="cuda")
    n = reps * len(runner.layers)
    e0, e1 = native.apex_event_create(True), native.apex_event_create(True)
    torch.cuda.synchronize()
    native.apex_spin_us(min(2000.0 + 20.0 * n, 1e6), runner.cs)
    native.apex_event_record(e0, runner.cs)
    for i in range(n):
        b = runner.bufs[runner.layers[i % len(runner.layers)]]
        native.apex_prefetch_route(b["h_pre"][0], b["wpf"], b["bias"], B, cfg.d, cfg.E, cfg.k,
                                   cfg.k_max, runner.policy, runner.tau, runner.static_delta,
                                   b["cdf_w"], b["cdf_theta"], pf_idx, pf_count, None,
                                   runner.cs)
    native.apex_event_record(e1, runner.cs)
    native.apex_event_synchronize(e1)
    us = native.apex_event_elapsed_ms(e0, e1) * 1e3 / n
    native.apex_event_destroy(e0)
    native.apex_event_destroy(e1)
    return us


def stream_floor_leg(torch, native, cs, nbytes, n=192, buf_bytes=1 << 30):
    """Device time of a plain read of the FFN call's weight bytes, split into two
    launches as the FFN splits them (W1/W3 rows, then W2 rows): the fastest any kernel
    can bring those bytes in at that size on this GPU.  Each launch reads fresh memory
    (a buffer of 1 GB, or twice the larger launch's bytes, far larger than the 256 MB
    Infinity Cache).  Returns mean us per call."""
    parts = [int(nbytes * 2 / 3) // 256 * 256, int(nbytes / 3) // 256 * 256]
    buf_bytes = max(buf_bytes, 2 * max(parts))   # every read stays inside the buffer
    buf = torch.empty(buf_bytes, dtype=torch.uint8, device="cuda")
    sink = torch.empty(native.apex_read_kernel_sink_words(max(parts)), dtype=torch.int32,
                       device="cuda")
    base, off = buf.data_ptr(), 0
    e0, e1 = native.apex_event_create(True), native.apex_event_create(True)
    torch.cuda.synchronize()
    native.apex_spin_us(min(5000.0 + 30.0 * n, 1e6), cs)
    native.apex_event_record(e0, cs)
    for _ in range(n):
        for part in parts:
            if off + part > buf_bytes:
                off = 0
            native.apex_read_kernel(base + off, part, sink, cs)
            off += part
    native.apex_event_record(e1, cs)
    native.apex_event_synchronize(e1)
    us = native.apex_event_elapsed_ms(e0, e1) * 1e3 / n
    native.apex_event_destroy(e0)
    native.apex_event_destroy(e1)
    del buf, sink
    return us


def attention_leg(torch, native, runner, reps=8):
    """Device time of one layer's decode attention (apex_attention_decode) in the decode
    launch configuration: calls cycling over the layers, queued behind a spin kernel,
    one event pair around the batch.  Returns mean microseconds per call."""
    cfg, B = runner.cfg, runner.B
    H, G, hd = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    ws_bytes = native.apex_attention_workspace_bytes(B, H, G, hd, runner.ctx + 1)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    cs = runner.cs
    n = reps * len(runner.layers)
    e0, e1 = native.apex_event_create(True), native.apex_event_create(True)
    torch.cuda.synchronize()
    native.apex_spin_us(min(5000.0 + 30.0 * n, 1e6), cs)
    native.apex_event_record(e0, cs)
    for i in range(n):
        b = runner.bufs[runner.layers[i % len(runner.layers)]]
        native.apex_attention_decode(b["h_pre"][0], b["w_qkv"], b["w_o"], B, cfg.d, H, G, hd,
                                     b["k_cache"], b["v_cache"], runner.ctx + 1, runner.ctx,
                                     b["attn_out"], ws, ws_bytes, cs)
    native.apex_event_record(e1, cs)
    native.apex_event_synchronize(e1)
    us = native.apex_event_elapsed_ms(e0, e1) * 1e3 / n
    native.apex_event_destroy(e0)
    native.apex_event_destroy(e1)
    return us


def copy_calibration(torch, native, cs, nbytes=256 << 20, reps=5):
    """A plain streaming copy of known size (apex_copy_kernel): measured HBM copy rate,
    and the reference dispatch for scaling the FETCH_SIZE / WRITE_SIZE counters."""
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    native.apex_copy_kernel(dst, src, nbytes, cs)
    e0, e1 = native.apex_event_create(True), native.apex_event_create(True)
    native.apex_event_record(e0, cs)
    for _ in range(reps):
        native.apex_copy_kernel(dst, src, nbytes, cs)
    native.apex_event_record(e1, cs)
    native.apex_event_synchronize(e1)
    ms = native.apex_event_elapsed_ms(e0, e1) / reps
    native.apex_event_destroy(e0)
    native.apex_event_destroy(e1)
    del src, dst
    return dict(bytes_read=nbytes, bytes_written=nbytes, us=round(ms * 1e3, 2),
                GBps_read_plus_write=round(2 * nbytes / (ms * 1e-3) / 1e9, 1))


def measured_traffic(cfg, batch, weights="bf16"):
    """HBM bytes per apex_moe_ffn call from the committed FETCH_SIZE / WRITE_SIZE records,
    or None when no record is for this workload and batch, or the source of the kernels
    it covers or the compiler flags they are built with have changed since the counters
    were taken."""
    import hashlib
    from paper_2608_11688_amd import build as _build
    path = os.path.join(ROOT, "profiles", "moe_ffn_traffic.json")
    try:
        records = json.load(open(path))["records"]
    except (OSError, KeyError, ValueError):
        return None
    for rec in records:
        if (rec.get("workload") != cfg.name or rec.get("batch") != batch or
                rec.get("weights", "bf16") != weights):
            continue
        try:
            src = open(os.path.join(ROOT, rec["kernel_source"]), "rb").read()
        except (OSError, KeyError):
            return None
        if hashlib.sha256(src).hexdigest() != rec.get("kernel_source_sha256"):
            return None
        if rec.get("hipcc_flags") != list(_build.HIPCC_FLAGS):
            return None
        return rec.get("traffic_bytes_per_call")
    return None


def time_steps(torch, runner, steps, warmup):
    """Runs warmup untimed steps, then times `steps` decode steps; ms per step.  The
    metrics of the warm-up steps alone (cold cache first) are kept in
    runner.warmup_summary; the runner's own metrics then cover the timed steps only."""
    for _ in range(warmup):
        runner.step()
    runner.finish()
    runner.warmup_summary = runner.summary() if warmup else None
    runner.reset_metrics()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        runner.step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    runner.finish()
    return (t1 - t0) * 1e3 / steps


def compute_only_leg(torch, args, cfg, make_runner, host_runner):
    """The same decode with every expert resident in HBM (C = E): the same kernels, no
    copies and no misses, over the pinned experts of `host_runner` (which stays open).
    Returns ms per step."""
    import dataclasses
    runner = make_runner(dataclasses.replace(cfg, C=cfg.E, k_max=min(cfg.k_max, cfg.E)),
                         host_experts_from=host_runner)
    try:
        return time_steps(torch, runner, args.steps, args.warmup)
    finally:
        runner.close()


def selection_stats(ranked, routed, pf_sel, pf_count, k):
    """Prefetch accounting of one layer, per token, from the router's whole ranking
    `ranked` [n, N] (best first), the routed set `routed` [n, k], the policy's selection
    `pf_sel` [n, >= max m] (ranked order, -1 after position m) and its size `pf_count`
    [n]: delta* (Eq. 3), delta_hat = max(m - k, 0) (Eq. 9; 0 when nothing is fetched),
    the overlap |K_r & K_p| / k and full coverage K_r subset of K_p (Eq. 2)."""
    ranked = np.asarray(ranked, np.int64)
    routed = np.asarray(routed, np.int64)
    pf_sel = np.asarray(pf_sel, np.int64)
    m = np.asarray(pf_count, np.int64)
    n, N = ranked.shape
    rows = np.arange(n)[:, None]
    pos = np.empty((n, N), np.int64)
    pos[rows, ranked] = np.arange(N)[None, :]
    dstar = np.maximum(pos[rows, routed].max(axis=1) + 1 - k, 0)
    slot = np.arange(pf_sel.shape[1])[None, :]
    sel = np.where(slot < m[:, None], pf_sel, -1)
    hit = (routed[:, :, None] == sel[:, None, :]).any(axis=2)
    return dict(delta_star=dstar, delta_hat=np.maximum(m - k, 0), m=m,
                overlap=hit.sum(axis=1) / k, coverage=hit.all(axis=1))


def per_layer_leg(cfg, policy, tau, static_delta, cdf, tokens=256, seed=2, streams=64):
    """Prefetch quality of every layer on `tokens` held-out tokens (hidden-state streams of
    their own seed: disjoint from the timed decode's and from the ordinal fit's), from the
    router and gate kernels: the router once with the whole ranking (static budget N - k,
    k_max = N) and once with the bench's policy, then the exact gate top-k.  Returns the
    per-layer means of delta*, delta_hat, overlap and coverage, the delta* histogram over
    every layer (index delta* = 0 .. N - k) and the histogram of the prefetched-set size
    m = k + delta_hat (index m = 0 .. k_max; m = 0 only with no prefetch)."""
    import torch
    from paper_2608_11688_amd import inputs, native
    E, k, d = cfg.E, cfg.k, cfg.d
    dev = torch.device("cuda")
    stream = torch.cuda.current_stream().cuda_stream
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    steps = -(-tokens // streams)
    rows = dict(delta_star=[], delta_hat=[], recall=[], full_coverage=[])
    dstar_all, m_all = [], []
    for l in range(cfg.L):
        h_pre, h_post = inputs.hidden_states(cfg, l, streams, steps, seed)
        h_pre, h_post = h_pre.reshape(-1, d)[:tokens], h_post.reshape(-1, d)[:tokens]
        wg, wpf, bias = inputs.router_weights(cfg, l, 0)
        b = None if bias is None else t(bias.astype(np.float32))
        hp, wp = t(h_pre), t(wpf.view(np.int16))
        cdf_w = cdf_theta = None
        if policy == native.SEL_ORDINAL_CDF:
            w, theta = (inputs.cdf_params(cfg, l, 0) if cdf is None
                        else cdf[l] if isinstance(cdf, dict) else cdf)
            cdf_w, cdf_theta = t(np.asarray(w, np.float32)), t(np.asarray(theta, np.float32))
        full = torch.empty((tokens, E), dtype=torch.int32, device=dev)
        sel = torch.empty((tokens, cfg.k_max), dtype=torch.int32, device=dev)
        cnt_full = torch.empty((tokens,), dtype=torch.int32, device=dev)
        cnt = torch.empty_like(cnt_full)
        prob = torch.empty((tokens, E), dtype=torch.float32, device=dev)
        native.apex_prefetch_route(hp, wp, b, tokens, d, E, k, E, native.SEL_STATIC, 0.0,
                                   E - k, None, None, full, cnt_full, prob, stream)
        native.apex_prefetch_route(hp, wp, b, tokens, d, E, k, cfg.k_max, policy, tau,
                                   static_delta, cdf_w, cdf_theta, sel, cnt, prob, stream)
        route_idx = torch.empty((tokens, k), dtype=torch.int32, device=dev)
        route_gate = torch.empty((tokens, k), dtype=torch.float32, device=dev)
        exec_idx, exec_gate = torch.empty_like(route_idx), torch.empty_like(route_gate)
        native.apex_gate_topk(t(h_post), t(wg.view(np.int16)), b, tokens, d, E, k,
                              native.MODE_EXACT, None, 0, route_idx, route_gate, exec_idx,
                              exec_gate, None, stream)
        torch.cuda.synchronize()
        st = selection_stats(full.cpu().numpy(), route_idx.cpu().numpy(), sel.cpu().numpy(),
                             cnt.cpu().numpy(), k)
        rows["delta_star"].append(round(float(st["delta_star"].mean()), 3))
        rows["delta_hat"].append(round(float(st["delta_hat"].mean()), 3))
        rows["recall"].append(round(float(st["overlap"].mean()), 4))
        rows["full_coverage"].append(round(float(st["coverage"].mean()), 4))
        dstar_all.append(st["delta_star"])
        m_all.append(st["m"])
    dstar_all, m_all = np.concatenate(dstar_all), np.concatenate(m_all)
    summary = dict(mean=round(float(dstar_all.mean()), 4),
                   p90=int(np.percentile(dstar_all, 90)), tokens=int(dstar_all.size),
                   layers=cfg.L)
    return summary, dict(tokens_per_layer=tokens, **rows,
                         delta_star_hist=np.bincount(dstar_all, minlength=E - k + 1).tolist(),
                         prefetch_size_hist=np.bincount(m_all,
                                                        minlength=cfg.k_max + 1).tolist())


def oracle_sample(cfg, batch, weights, policy, cdf, preload_bytes=8e9, threads=16):
    """The oracle's inputs for the CPU baseline, drawn before any timing, as the GPU leg's
    are: the first layers of the workload (as many as keep the drawn bf16 experts under
    `preload_bytes`, at most 4), their routers and every expert's weights, and the hidden
    states of the first steps (16 for experts of 64 MB and more, else 64)."""
    from oracle import decode
    from paper_2608_11688_amd import inputs
    S = 6 * cfg.d * cfg.I
    n_layers = max(1, min(cfg.L, 4, int(preload_bytes // (cfg.E * S))))
    layers = list(range(n_layers))
    steps = 16 if S >= (64 << 20) else 64
    states = decode.make_states(cfg, layers, policy=policy, cdf=cdf, weights=weights)
    with cf.ThreadPoolExecutor(threads) as pool:
        list(pool.map(lambda le: states[le[0]].expert_bits(le[1]),
                      [(l, e) for l in layers for e in range(cfg.E)]))
    hidden = {l: inputs.hidden_states(cfg, l, batch, steps) for l in layers}
    return dict(layers=layers, steps=steps, states=states, hidden=hidden)


def cpu_baseline(cfg, batch, mode, tau, budget_s, sample, policy=0, static_delta=0, cdf=None,
                 weights="bf16", threads_limit=None):
    """The oracle, as it stands, on the first layer-steps of the same workload, over the
    inputs of `sample` (oracle_sample: drawn beforehand, so the timed region holds the
    oracle's own arithmetic only); with threads_limit, under that many BLAS threads.  Also
    counts the near ties the oracle finds in the sample (decision margins below 1e-5 at the
    gate's top-k cut and at the prefetch selection's cut), the points where a GPU set may
    differ legitimately."""
    from oracle import decode
    import contextlib
    try:
        import threadpoolctl
        limit = (threadpoolctl.threadpool_limits(threads_limit) if threads_limit
                 else contextlib.nullcontext())
    except Exception:
        threadpoolctl, limit = None, contextlib.nullcontext()
    layers, steps = sample["layers"], sample["steps"]
    # fresh caches for every timed run, the drawn weights shared
    states = decode.make_states(cfg, layers, policy=policy, cdf=cdf, weights=weights,
                                bits_from=sample["states"])
    n, elapsed, gate_ties, cut_ties, rows, t_last = 0, 0.0, 0, 0, 0, 0
    with limit:
        threads = 1
        if threadpoolctl is not None:
            threads = max((i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()),
                          default=1)
        gen = decode.run(cfg, batch, steps, mode=mode, tau=tau, layers=layers, policy=policy,
                         static_delta=static_delta, cdf=cdf, weights=weights, states=states,
                         hidden=sample["hidden"])
        it = iter(gen)
        t0 = time.perf_counter()
        for t, l, out in it:
            n += 1
            t_last = t
            gate_ties += int((out["gate"]["margin"] < 1e-5).sum())
            cut_ties += int((out["route"]["margin"] < 1e-5).sum())
            rows += len(out["gate"]["margin"])
            elapsed = time.perf_counter() - t0
            if elapsed > budget_s:
                break
    base = dict(value=elapsed * 1e6 / (n * batch), unit="us/token/layer", cores=int(threads),
                kind="oracle",
                sample=f"{cfg.name} batch {batch} {['exact', 'stall_free'][mode]} mode, first {n} "
                       f"layer-steps (steps 0-{t_last} of layers {layers[0]}-{layers[-1]}), fp64 "
                       f"NumPy; hidden states, routers and expert weights drawn before timing")
    ties = dict(token_layers=rows, gate_cut=gate_ties, prefetch_cut=cut_ties, margin_below=1e-5,
                sample=f"the oracle's {n} layer-steps above")
    return base, ties


def release(torch):
    """Waits for the device and returns every cached block, so that nothing this process
    allocated on the GPU or in pinned memory is left for interpreter and library teardown."""
    torch.cuda.synchronize()
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    try:
        torch._C._host_emptyCache()
    except Exception:
        pass


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              f"(the hot path runs on one GPU; sharding it across GPUs is not built)",
              file=sys.stderr)
        return 2
    import torch
    from paper_2608_11688_amd import configs, native
    from paper_2608_11688_amd.runtime import DecodeRunner, EXACT, STALL_FREE

    cfg = configs.get(args.config)
    mode = EXACT if args.mode == "exact" else STALL_FREE
    tau = cfg.tau if args.tau is None else args.tau
    policy = {"cumprob": native.SEL_CUMPROB, "ordinal": native.SEL_ORDINAL_CDF,
              "static": native.SEL_STATIC, "none": native.SEL_NONE}[args.policy]
    cdf, cdf_report = None, None
    if policy == native.SEL_ORDINAL_CDF:
        from paper_2608_11688_amd import cdf_fit
        cdf, cdf_report = cdf_fit.fit_model(cfg, tokens=args.cdf_tokens)
    total = args.warmup + args.steps

    def make_runner(c, **kw):
        return DecodeRunner(c, batch=args.batch, mode=mode, tau=tau, steps=max(total, 1),
                            t_attn_us=args.t_attn_us, policy=policy,
                            static_delta=args.static_delta, cdf=cdf, weights=args.weights,
                            window=args.window, ctx=args.ctx, **kw)

    try:
        runner = make_runner(cfg)
    except ValueError as e:       # a workload the runner refuses, before anything is drawn
        print(f"bench.py: {e}", file=sys.stderr)
        return 2
    h2d_peak = pinned_h2d_peak(torch)
    ms_per_step = time_steps(torch, runner, args.steps, args.warmup)
    leg_ms, leg_bytes, leg_n = ffn_roofline_leg(torch, native, runner)
    router_us = None if policy == native.SEL_NONE else router_leg(torch, native, runner)
    floor_us = stream_floor_leg(torch, native, runner.cs, leg_bytes)
    calib = copy_calibration(torch, native, runner.cs)

    L, B = len(runner.layers), args.batch
    us_layer_step = ms_per_step * 1e3 / L
    attn_us = attention_leg(torch, native, runner) if args.window == "attention" else None
    window_us = attn_us if attn_us is not None else args.t_attn_us
    value = (us_layer_step - window_us) / B
    S = runner.S
    achieved = leg_bytes / (leg_ms * 1e-3) / 1e9
    s = runner.summary()
    warm = runner.warmup_summary
    copied_bytes_per_step = s["copies_per_layer_step"] * L * S
    # exposed stall: this timeline against the same one with every expert resident
    value_resident = stall = None
    if not args.no_compute_only:
        ms_res = compute_only_leg(torch, args, cfg, make_runner, runner)
        value_resident = (ms_res * 1e3 / L - window_us) / B
        stall = value - value_resident
    runner.close()
    del runner
    copy_leg = expert_copy_leg(torch, native, S, cfg.E, h2d_peak)
    dstar, per_layer = per_layer_leg(cfg, policy, tau, args.static_delta, cdf)
    release(torch)
    out = {
        "metric": "MoE-layer decode us/token + expert-weight HBM GB/s; prefetch recall vs oracle",
        "value": round(value, 3),
        "unit": "us/token/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"fp8": "fp8-e4m3", "mxfp4": "mxfp4", "bf16": "bf16",
                  "fp32": "fp32"}[args.weights],
        "arithmetic": {"fp8": "fp8 e4m3 weights with fp32 row scales, fp32 accumulate",
                       "mxfp4": "mxfp4 (e2m1, e8m0 block scales) weights, fp32 accumulate",
                       "bf16": "bf16 weights, fp32 accumulate",
                       "fp32": "fp32 weights, fp32 accumulate"}[args.weights],
        "data": "synthetic (seeded AR(1) hidden states, N(0,0.02) bf16 experts)",
        "config": {"workload": cfg.name, "layers": L, "d": cfg.d, "E": cfg.E, "k": cfg.k,
                   "I": cfg.I, "C": cfg.C, "k_max": cfg.k_max, "tau": tau, "batch": B,
                   "mode": args.mode, "policy": args.policy, "weights": args.weights,
                   "window": args.window},
        "us_per_layer_step_incl_attn_window": round(us_layer_step, 3),
        "attn_window_us": round(window_us, 3),
        "ffn_us": round(leg_ms * 1e3, 3),
        "ffn_hbm_GBps": round(achieved, 1),
        "recall": round(s["recall"], 5),
        "full_coverage": round(s["full_coverage"], 5),
        "mean_delta_hat": None if args.policy == "none" else round(s["mean_delta_hat"], 4),
        "cache_hit_rate": round(s["hit_rate"], 5),
        "mean_delta_star": dstar["mean"],
        "delta_star": dstar,
        "per_layer": per_layer,
        "router": None if router_us is None else {
            "us_per_call": round(router_us, 3),
            "share_of_layer_step": round(router_us / us_layer_step, 5),
            "share_of_compute_only_layer_step": (
                None if value_resident is None
                else round(router_us / (value_resident * B + window_us), 5)),
            # the paper's overhead count per layer: the router's d x E weights plus 2E
            "extra_params_per_layer": cfg.d * cfg.E + 2 * cfg.E},
        "copies_per_layer_step": round(s["copies_per_layer_step"], 4),
        "copied_MB_per_layer_step": round(s["copies_per_layer_step"] * S / 1e6, 3),
        "misses_per_layer_step": round(s["misses_per_layer_step"], 4),
        "warmup_cold_cache": None if warm is None else {
            "steps": args.warmup, "recall": round(warm["recall"], 5),
            "full_coverage": round(warm["full_coverage"], 5),
            "cache_hit_rate": round(warm["hit_rate"], 5),
            "copies_per_layer_step": round(warm["copies_per_layer_step"], 4),
            "misses_per_layer_step": round(warm["misses_per_layer_step"], 4)},
        "compute_only_us_per_token_layer": (None if value_resident is None
                                            else round(value_resident, 3)),
        "exposed_stall_us_per_token_layer": None if stall is None else round(stall, 3),
        "h2d_GBps_over_step": round(copied_bytes_per_step / (ms_per_step * 1e-3) / 1e9, 2),
        "h2d_pinned_peak_GBps": round(h2d_peak, 2),
        "copy_leg": copy_leg,
        "hbm_copy_kernel": calib,
        "roofline": {"bound": "hbm", "kernel": FFN_KERNELS[(args.weights, B == 1)],
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": measured_traffic(cfg, B, args.weights),
                     "bytes_per_launch": leg_bytes, "launches": leg_n,
                     # the same bytes read by a plain two-launch read stream
                     "read_stream_us": round(floor_us, 3),
                     "frac_of_read_stream": round(floor_us / (leg_ms * 1e3), 4)},
    }
    if args.policy == "static":
        out["config"]["static_delta"] = args.static_delta
    if args.window == "attention":
        out["config"].update(ctx=args.ctx, heads=cfg.n_heads, kv_heads=cfg.n_kv_heads)
    else:
        out["config"]["t_attn_us"] = args.t_attn_us
    if cdf_report is not None:
        out["ordinal_fit"] = cdf_report
    if not args.no_cpu_baseline:
        sample = oracle_sample(cfg, B, args.weights, policy, cdf)
        out["cpu_baseline"], out["oracle_near_ties"] = cpu_baseline(
            cfg, B, mode, tau, args.cpu_budget_s, sample, policy, args.static_delta, cdf,
            args.weights)
        if args.cpu_1thread_budget_s > 0:
            out["cpu_baseline_1thread"], _ = cpu_baseline(
                cfg, B, mode, tau, args.cpu_1thread_budget_s, sample, policy, args.static_delta,
                cdf, args.weights, threads_limit=1)
        del sample
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())

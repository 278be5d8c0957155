"""Decode runner: one MoE-decode step per call, every layer through the C ABI.

Per layer and step (Sec. IV-A two-stage runtime; Sec. IV-E execution modes):

  compute: apex_prefetch_route(h_pre) -> K_p written straight to pinned host memory
           record route_done; apex_spin_us(t_attn) (the attention window)
  host:    wait route_done; apex_expert_prefetch: plan + H2D copies on the side stream
           (they overlap the attention window), publish the slot table on compute
  compute: apex_gate_topk(h_post) -> K_r to pinned host memory, executed set on device
           wait ready (copies landed); apex_moe_ffn pass 1 over the resident experts
  exact mode only -
  host:    wait gate_done; apex_expert_fetch_misses: copies of K_r minus resident into
           the miss scratch on the side stream while pass 1 runs
  compute: wait ready_miss; apex_moe_ffn pass 2 (accumulate) over the scratch pool
  compute: record readers_done (the next copy into this layer's slots waits for it)

PyTorch only provides device/pinned memory and the streams; every step above is a
call into the library.
"""
from __future__ import annotations

import concurrent.futures as cf
import time
from dataclasses import dataclass, field

import numpy as np

from . import configs, inputs, native

EXACT, STALL_FREE = native.MODE_EXACT, native.MODE_STALL_FREE


def _torch():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("the decode runner needs a GPU")
    return torch


@dataclass
class LayerBuffers:
    wg: object
    wpf: object
    bias: object
    host_experts: object       # pinned int16 [E * S_e / 2]
    slots: object              # device int16 [C * S_e / 2]
    slot_dev: object           # device int32 [E]
    avail_dev: object          # device uint8 [E]
    expert_of_slot: np.ndarray
    last_used: np.ndarray
    h_pre: object              # device fp32 [steps, B, d]
    h_post: object
    ready: int = 0
    readers_done: int = 0
    cdf_w: object = None
    cdf_theta: object = None


@dataclass
class StepLog:
    pf_idx: np.ndarray
    pf_count: np.ndarray
    route_idx: np.ndarray
    route_gate: np.ndarray
    exec_idx: np.ndarray
    exec_gate: np.ndarray
    resident: list
    copies: int
    missing: list
    y: np.ndarray = None


class DecodeRunner:
    def __init__(self, cfg: configs.MoEConfig, batch=1, mode=EXACT, tau=None,
                 policy=native.SEL_CUMPROB, static_delta=0, seed=0, steps=None, t_attn_us=10.0,
                 layers=None, n_scratch=None, record=False, cdf=None, time_ffn=False,
                 gen_threads=16):
        torch = _torch()
        self.torch = torch
        self.cfg, self.B, self.mode = cfg, batch, mode
        self.tau = cfg.tau if tau is None else tau
        self.policy, self.static_delta, self.seed = policy, static_delta, seed
        self.steps = cfg.steps if steps is None else steps
        self.t_attn_us = t_attn_us
        self.layers = list(range(cfg.L)) if layers is None else list(layers)
        self.record, self.time_ffn = record, time_ffn
        self.dev = torch.device("cuda")
        self.compute = torch.cuda.current_stream()
        self.side = torch.cuda.Stream()
        self.cs, self.ss = self.compute.cuda_stream, self.side.cuda_stream
        self.S = native.apex_expert_bytes(cfg.d, cfg.I)
        E, B, k = cfg.E, batch, cfg.k
        self.n_scratch = min(E, B * k) if n_scratch is None else n_scratch

        self.L = {}
        with cf.ThreadPoolExecutor(gen_threads) as pool:
            for l in self.layers:
                self.L[l] = self._make_layer(l, pool, cdf)
        torch.cuda.synchronize()

        i32 = dict(dtype=torch.int32)
        self.pf_idx_h = torch.empty((B, cfg.k_max), pin_memory=True, **i32)
        self.pf_count_h = torch.empty(B, pin_memory=True, **i32)
        self.route_idx_h = torch.empty((B, k), pin_memory=True, **i32)
        self.route_gate_h = torch.empty((B, k), dtype=torch.float32, pin_memory=True)
        self.exec_idx = torch.empty((B, k), device=self.dev, **i32)
        self.exec_gate = torch.empty((B, k), dtype=torch.float32, device=self.dev)
        self.y = torch.empty((B, cfg.d), dtype=torch.float32, device=self.dev)
        self.ws_bytes = native.apex_moe_ffn_workspace_bytes(B, k, cfg.I)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.dev)
        self.scratch = torch.empty(max(1, self.n_scratch) * self.S // 2, dtype=torch.int16,
                                   device=self.dev)
        self.miss_table = torch.full((E,), -1, device=self.dev, **i32)
        self.ev_route = native.apex_event_create(False)
        self.ev_gate = native.apex_event_create(False)
        self.ready_miss = native.apex_event_create(False)
        self.scratch_free = native.apex_event_create(False)
        native.apex_event_record(self.scratch_free, self.cs)
        self.ev_pool, self.ffn_pending = [], []
        if time_ffn and mode == STALL_FREE and batch > 1:
            self.exec_ring = torch.empty((self.steps * len(self.layers), B, k), pin_memory=True,
                                         **i32)
        self.ring_pos = 0
        self.copied = np.zeros(max(cfg.C, 1), np.int32)
        self.missing = np.zeros(E, np.int32)
        self.t = 0
        self.reset_metrics()

    # ------------------------------------------------------------------ setup
    def _make_layer(self, l, pool, cdf):
        torch, cfg = self.torch, self.cfg
        wg, wpf, bias = inputs.router_weights(cfg, l, self.seed)
        to_dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(self.dev)
        S2 = self.S // 2
        host = torch.empty(cfg.E * S2, dtype=torch.int16, pin_memory=True)
        hp = host.data_ptr()

        def fill(e):
            w1, w3, w2 = inputs.expert_weights(cfg, l, e, self.seed)
            native.apex_pack_expert(w1, w3, w2, cfg.d, cfg.I, hp + e * self.S)

        list(pool.map(fill, range(cfg.E)))
        slots = torch.empty(cfg.C * S2, dtype=torch.int16, device=self.dev)
        n0 = min(cfg.C, cfg.E)
        slots[:n0 * S2].copy_(host[:n0 * S2])
        eos = np.array([s if s < cfg.E else -1 for s in range(cfg.C)], np.int32)
        table = np.full(cfg.E, -1, np.int32)
        for s, e in enumerate(eos):
            if e >= 0:
                table[e] = s
        h_pre, h_post = inputs.hidden_states(cfg, l, self.B, self.steps, self.seed)
        lb = LayerBuffers(
            wg=to_dev(wg.view(np.int16)), wpf=to_dev(wpf.view(np.int16)),
            bias=None if bias is None else to_dev(bias), host_experts=host, slots=slots,
            slot_dev=to_dev(table), avail_dev=to_dev((table >= 0).astype(np.uint8)),
            expert_of_slot=eos, last_used=np.full(cfg.E, -1, np.int64),
            h_pre=to_dev(h_pre), h_post=to_dev(h_post))
        lb.ready = native.apex_event_create(False)
        lb.readers_done = native.apex_event_create(False)
        if self.policy == native.SEL_ORDINAL_CDF:
            w, theta = cdf if cdf is not None else inputs.cdf_params(cfg, l, self.seed)
            lb.cdf_w, lb.cdf_theta = to_dev(np.asarray(w, np.float32)), to_dev(
                np.asarray(theta, np.float32))
        return lb

    def reset_metrics(self):
        self.m = dict(layer_steps=0, tokens=0, overlap=0.0, coverage=0, copies=0, misses=0,
                      delta_hat=0, ffn_ms=0.0, ffn_calls=0, ffn_experts=0, hits=0.0)

    # ------------------------------------------------------------------ step
    def layer_step(self, l, t):
        cfg, B, k = self.cfg, self.B, self.cfg.k
        lb = self.L[l]
        cs, ss = self.cs, self.ss
        native.apex_prefetch_route(
            lb.h_pre[t], lb.wpf, lb.bias, B, cfg.d, cfg.E, k, cfg.k_max, self.policy, self.tau,
            self.static_delta, lb.cdf_w, lb.cdf_theta, self.pf_idx_h, self.pf_count_h, None, cs)
        native.apex_event_record(self.ev_route, cs)
        native.apex_spin_us(self.t_attn_us, cs)
        native.apex_event_synchronize(self.ev_route)
        n_copy = native.apex_expert_prefetch(
            lb.host_experts, lb.slots, cfg.E, cfg.C, self.S, self.pf_idx_h, self.pf_count_h, B,
            cfg.k_max, t, lb.expert_of_slot, lb.last_used, lb.slot_dev, lb.avail_dev, ss, cs,
            lb.readers_done, lb.ready, self.copied)
        native.apex_gate_topk(
            lb.h_post[t], lb.wg, lb.bias, B, cfg.d, cfg.E, k, self.mode, lb.avail_dev, 0,
            self.route_idx_h, self.route_gate_h, self.exec_idx, self.exec_gate, None, cs)
        native.apex_event_record(self.ev_gate, cs)
        native.apex_stream_wait_event(cs, lb.ready)
        if self.time_ffn:
            evs = self.ev_pool.pop() if self.ev_pool else (native.apex_event_create(True),
                                                            native.apex_event_create(True))
            native.apex_event_record(evs[0], cs)
        native.apex_moe_ffn(lb.h_post[t], B, cfg.d, cfg.I, cfg.E, k, self.exec_idx,
                            self.exec_gate, lb.slot_dev, lb.slots, cfg.C, self.y, 0, self.ws,
                            self.ws_bytes, cs)
        if self.time_ffn:
            native.apex_event_record(evs[1], cs)
            ring = None
            if self.mode == STALL_FREE and B > 1:
                ring = self.exec_ring[self.ring_pos % self.exec_ring.shape[0]]
                ring.copy_(self.exec_idx, non_blocking=True)
                self.ring_pos += 1
        n_miss = 0
        native.apex_event_synchronize(self.ev_gate)
        pf_idx = self.pf_idx_h.numpy().copy()
        pf_count = self.pf_count_h.numpy().copy()
        route_idx = self.route_idx_h.numpy().copy()
        if self.mode == EXACT:
            n_miss = native.apex_expert_fetch_misses(
                lb.host_experts, self.scratch, self.n_scratch, cfg.E, cfg.C, self.S, route_idx, B,
                k, lb.expert_of_slot, self.miss_table, ss, cs, self.scratch_free, self.ready_miss,
                self.missing)
            if n_miss:
                native.apex_stream_wait_event(cs, self.ready_miss)
                native.apex_moe_ffn(lb.h_post[t], B, cfg.d, cfg.I, cfg.E, k, self.exec_idx,
                                    self.exec_gate, self.miss_table, self.scratch,
                                    self.n_scratch, self.y, 1, self.ws, self.ws_bytes, cs)
                native.apex_event_record(self.scratch_free, cs)
        native.apex_event_record(lb.readers_done, cs)
        if self.time_ffn:
            resident = set(int(e) for e in lb.expert_of_slot if e >= 0)
            if self.mode == EXACT:
                n_exp = len(set(int(e) for e in route_idx.ravel()) & resident)
            elif B == 1:
                n_exp = min(k, len(resident))
            else:
                n_exp = None                      # read from the ring after the sync
            self.ffn_pending.append((evs, n_exp, ring))
        self._account(pf_idx, pf_count, route_idx, n_copy, n_miss, lb)
        if self.record:
            return self._log(l, pf_idx, pf_count, route_idx, n_copy, n_miss, lb)
        return None

    def step(self):
        """One decode step through every layer; returns the per-layer logs if recording."""
        t = self.t
        logs = {}
        for l in self.layers:
            r = self.layer_step(l, t)
            if self.record:
                logs[l] = r
        self.t += 1
        return logs

    # ------------------------------------------------------------------ bookkeeping
    def _account(self, pf_idx, pf_count, route_idx, n_copy, n_miss, lb):
        cfg, m = self.cfg, self.m
        resident = set(int(e) for e in lb.expert_of_slot if e >= 0)
        for b in range(self.B):
            K_p = set(int(e) for e in pf_idx[b, :pf_count[b]])
            K_r = set(int(e) for e in route_idx[b])
            m["overlap"] += len(K_r & K_p) / cfg.k
            m["coverage"] += int(K_r <= K_p)
            m["delta_hat"] += int(pf_count[b]) - cfg.k
            m["hits"] += len(K_r & resident) / cfg.k
        m["tokens"] += self.B
        m["layer_steps"] += 1
        m["copies"] += n_copy
        m["misses"] += n_miss

    def drain_ffn_times(self):
        """[(ms, distinct experts read)] of every timed pass-1 FFN call since the last drain."""
        self.torch.cuda.synchronize()
        out = []
        for evs, n_exp, ring in self.ffn_pending:
            if n_exp is None:
                n_exp = len(set(int(e) for e in ring.numpy().ravel() if e >= 0))
            out.append((native.apex_event_elapsed_ms(evs[0], evs[1]), n_exp))
            self.ev_pool.append(evs)
        self.ffn_pending = []
        return out

    def _log(self, l, pf_idx, pf_count, route_idx, n_copy, n_miss, lb):
        torch = self.torch
        torch.cuda.synchronize()
        return StepLog(
            pf_idx=pf_idx, pf_count=pf_count, route_idx=route_idx,
            route_gate=self.route_gate_h.numpy().copy(),
            exec_idx=self.exec_idx.cpu().numpy(), exec_gate=self.exec_gate.cpu().numpy(),
            resident=sorted(int(e) for e in lb.expert_of_slot if e >= 0), copies=n_copy,
            missing=[int(e) for e in self.missing[:n_miss]], y=self.y.cpu().numpy())

    def summary(self):
        m = self.m
        tok = max(m["tokens"], 1)
        ls = max(m["layer_steps"], 1)
        return dict(recall=m["overlap"] / tok, full_coverage=m["coverage"] / tok,
                    mean_delta_hat=m["delta_hat"] / tok, hit_rate=m["hits"] / tok,
                    copies_per_layer_step=m["copies"] / ls, misses_per_layer_step=m["misses"] / ls,
                    expert_bytes=self.S)

    def close(self):
        self.drain_ffn_times()
        for ev in (self.ev_route, self.ev_gate, self.ready_miss, self.scratch_free):
            native.apex_event_destroy(ev)
        for evs in self.ev_pool:
            for ev in evs:
                native.apex_event_destroy(ev)
        self.ev_pool = []
        for lb in self.L.values():
            native.apex_event_destroy(lb.ready)
            native.apex_event_destroy(lb.readers_done)
        self.L = {}

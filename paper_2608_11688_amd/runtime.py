"""Decode runner: buffers for a workload plus the native decode driver.

The per-layer sequence of a decode step (prefetch router, cache plan and expert
copies on a side stream, attention-window stand-in, gate, expert FFN, miss correction)
runs inside the library's decode driver (apex_decode_step), which calls the same
entry points the tests exercise one by one.  This module only allocates the device
and pinned buffers with PyTorch, fills them from the seeded generators, and marshals
pointers.
"""
from __future__ import annotations

import concurrent.futures as cf
import ctypes as C
from dataclasses import dataclass

import numpy as np

from . import configs, inputs, native

EXACT, STALL_FREE = native.MODE_EXACT, native.MODE_STALL_FREE


def _torch():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("the decode runner needs a GPU")
    return torch


MAX_PINNED_EXPERT_BYTES = 32 << 30


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
                 layers=None, n_scratch=None, record=False, cdf=None, gen_threads=16,
                 weights="bf16", window="spin", ctx=1024, host_experts_from=None):
        """host_experts_from: another runner of the same workload, layers and weight
        format whose pinned host experts this one uses instead of drawing and pinning its
        own (the other runner must stay open while this one runs)."""
        torch = _torch()
        self.torch = torch
        self.cfg, self.B, self.mode = cfg, batch, mode
        self.tau = cfg.tau if tau is None else tau
        self.policy, self.static_delta, self.seed = policy, static_delta, seed
        self.steps = cfg.steps if steps is None else steps
        self.t_attn_us = t_attn_us
        self.layers = list(range(cfg.L)) if layers is None else list(layers)
        self.record = record
        self.dev = torch.device("cuda")
        self.compute = torch.cuda.current_stream()
        self.side = torch.cuda.Stream()
        self.cs, self.ss = self.compute.cuda_stream, self.side.cuda_stream
        self._wcode, self._wbytes, self._wpack, self.moe_ffn = native.weight_format(weights)
        self.weights = weights
        if window not in ("spin", "attention"):
            raise ValueError(f"window must be 'spin' or 'attention', not {window!r}")
        self.window, self.ctx = window, ctx
        self.S = self.expert_bytes(cfg.I)
        E, B, k = cfg.E, batch, cfg.k
        self.n_scratch = min(E, B * k) if n_scratch is None else n_scratch
        L = len(self.layers)

        # every layer's experts are held in pinned host memory at once; a Mixtral-shaped
        # stack with fp32 experts (8 x 8 experts of 705 MB, 45 GB) ended in a host
        # segmentation fault before its first output, cause not established, so the
        # runner stays within what has run
        pinned = L * E * self.S
        if host_experts_from is None and pinned > MAX_PINNED_EXPERT_BYTES:
            raise ValueError(f"{L} layers of {E} {weights} experts need {pinned / 1e9:.1f} GB "
                             f"of pinned host memory; the runner holds at most "
                             f"{MAX_PINNED_EXPERT_BYTES / 2**30:.0f} GiB")
        if host_experts_from is not None:
            o = host_experts_from
            if (o.cfg.d, o.cfg.I, o.cfg.E, o.weights, o.seed) != (cfg.d, cfg.I, cfg.E, weights,
                                                                   seed) or \
                    not set(self.layers) <= set(o.bufs):
                raise ValueError("host_experts_from: another workload, format or layer set")
        self.bufs = {}
        with cf.ThreadPoolExecutor(gen_threads) as pool:
            for l in self.layers:
                shared = None if host_experts_from is None else host_experts_from.bufs[l]["host"]
                self.bufs[l] = self._make_layer(l, pool, cdf, shared)
        i32 = dict(dtype=torch.int32, device=self.dev)
        self.exec_idx = torch.empty((B, k), **i32)
        self.exec_gate = torch.empty((B, k), dtype=torch.float32, device=self.dev)
        self.y = torch.zeros((L, B, cfg.d), dtype=torch.float32, device=self.dev)
        self.ws_bytes = native.apex_moe_ffn_workspace_bytes(B, cfg.d, cfg.I, k)
        if cfg.shared:
            self.ws_bytes = max(self.ws_bytes, native.apex_moe_ffn_workspace_bytes(
                B, cfg.d, cfg.shared_I, cfg.shared))
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.dev)
        self.scratch = torch.empty(max(1, self.n_scratch) * self.S // 2, dtype=torch.int16,
                                   device=self.dev)
        self.miss_table = torch.full((E,), -1, **i32)
        torch.cuda.synchronize()

        dcfg = native.DecodeConfig(L=L, B=B, d=cfg.d, E=E, k=k, I=cfg.I, C=cfg.C,
                                   k_max=cfg.k_max, policy=policy, tau=self.tau,
                                   static_delta=static_delta, mode=mode, t_attn_us=t_attn_us,
                                   n_scratch=self.n_scratch,
                                   weights=self._wcode,
                                   attn_heads=cfg.n_heads if window == "attention" else 0,
                                   attn_kv_heads=cfg.n_kv_heads, attn_ctx=ctx,
                                   n_shared=cfg.shared, I_shared=cfg.shared_I)
        descs = []
        for l in self.layers:
            b = self.bufs[l]
            p = lambda t: None if t is None else native.ptr(t)
            descs.append(native.DecodeLayer(
                w_pf=p(b["wpf"]), w_g=p(b["wg"]), b_pf=p(b["bias"]), b_g=p(b["bias"]),
                cdf_w=p(b["cdf_w"]), cdf_theta=p(b["cdf_theta"]),
                host_experts=p(b["host"]), slots=p(b["slots"]),
                slot_of_expert_dev=p(b["slot_dev"]), avail_dev=p(b["avail_dev"]),
                expert_of_slot=b["eos"].ctypes.data, last_used=b["last_used"].ctypes.data,
                w_qkv=p(b.get("w_qkv")), w_o=p(b.get("w_o")), k_cache=p(b.get("k_cache")),
                v_cache=p(b.get("v_cache")), attn_out=p(b.get("attn_out")),
                shared_slots=p(b.get("shared_slots"))))
        self.dec, self._descs = native.apex_decode_create(
            dcfg, descs, self.scratch, self.miss_table, self.exec_idx, self.exec_gate, self.ws,
            self.ws_bytes, self.cs, self.ss)
        PtrArr = C.c_void_p * L
        row = B * cfg.d * 4
        self._h_pre = [PtrArr(*[self.bufs[l]["h_pre"].data_ptr() + t * row for l in self.layers])
                       for t in range(self.steps)]
        self._h_post = [PtrArr(*[self.bufs[l]["h_post"].data_ptr() + t * row
                                 for l in self.layers]) for t in range(self.steps)]
        self._y = PtrArr(*[self.y[i].data_ptr() for i in range(L)])
        self.stats = native.DecodeStats()
        if record:
            self._rec_arrays = dict(
                pf_idx=np.zeros((L, B, cfg.k_max), np.int32), pf_count=np.zeros((L, B), np.int32),
                route_idx=np.zeros((L, B, k), np.int32), route_gate=np.zeros((L, B, k), np.float32),
                exec_idx=np.zeros((L, B, k), np.int32), exec_gate=np.zeros((L, B, k), np.float32),
                resident=np.zeros((L, cfg.C), np.int32), n_copies=np.zeros(L, np.int32),
                missing=np.zeros((L, E), np.int32), n_missing=np.zeros(L, np.int32))
            self._rec = native.DecodeRecord(**{k_: a.ctypes.data
                                               for k_, a in self._rec_arrays.items()})
        self.t = 0

    # ------------------------------------------------------------------ setup
    def expert_bytes(self, I):
        """Bytes of one packed expert of intermediate size I in this runner's format."""
        return self._wbytes(self.cfg.d, I)

    def pack(self, w1, w3, w2, d, I, out):
        self._wpack(w1, w3, w2, d, I, out)

    def _make_layer(self, l, pool, cdf, host=None):
        torch, cfg = self.torch, self.cfg
        wg, wpf, bias = inputs.router_weights(cfg, l, self.seed)
        to_dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(self.dev)
        S2 = self.S // 2
        if host is None:
            host = torch.empty(cfg.E * S2, dtype=torch.int16, pin_memory=True)
            hp = host.data_ptr()

            def fill(e):
                w1, w3, w2 = inputs.expert_weights(cfg, l, e, self.seed)
                self.pack(w1, w3, w2, cfg.d, cfg.I, hp + e * self.S)

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
        out = dict(wg=to_dev(wg.view(np.int16)), wpf=to_dev(wpf.view(np.int16)),
                   bias=None if bias is None else to_dev(bias), host=host, slots=slots,
                   slot_dev=to_dev(table), avail_dev=to_dev((table >= 0).astype(np.uint8)),
                   eos=eos, last_used=np.full(cfg.E, -1, np.int64), h_pre=to_dev(h_pre),
                   h_post=to_dev(h_post), cdf_w=None, cdf_theta=None)
        if cfg.shared:
            # the shared experts: resident for the driver's life, never prefetched
            S_sh = self.expert_bytes(cfg.shared_I)
            sh = np.empty(cfg.shared * S_sh, np.uint8)
            for s_ in range(cfg.shared):
                w1, w3, w2 = inputs.shared_expert_weights(cfg, l, s_, self.seed)
                self.pack(w1, w3, w2, cfg.d, cfg.shared_I, sh[s_ * S_sh:].ctypes.data)
            out["shared_slots"] = to_dev(sh)
        if self.window == "attention":
            w_qkv, w_o = inputs.attention_weights(cfg, l, self.seed)
            out["w_qkv"] = to_dev(w_qkv.view(np.int16))
            out["w_o"] = to_dev(w_o.view(np.int16))
            out["k_cache"], out["v_cache"] = inputs.kv_cache_device(
                torch, cfg, l, self.B, self.ctx + 1, self.seed, self.dev)
            out["attn_out"] = torch.zeros((self.B, cfg.d), dtype=torch.float32, device=self.dev)
        if self.policy == native.SEL_ORDINAL_CDF:
            if cdf is None:
                w, theta = inputs.cdf_params(cfg, l, self.seed)
            elif isinstance(cdf, dict):
                w, theta = cdf[l]          # one fitted model per layer
            else:
                w, theta = cdf             # one model for every layer
            out["cdf_w"] = to_dev(np.asarray(w, np.float32))
            out["cdf_theta"] = to_dev(np.asarray(theta, np.float32))
        return out

    # ------------------------------------------------------------------ step
    def step(self):
        """One decode step through every layer; with record=True returns per-layer logs."""
        t = self.t
        if t >= self.steps:
            raise IndexError(f"the runner holds hidden states for {self.steps} steps")
        native.apex_decode_step(self.dec, t, self._h_pre[t], self._h_post[t], self._y,
                                self.stats, self._rec if self.record else None)
        self.t += 1
        if not self.record:
            return None
        a = self._rec_arrays
        ys = self.y.cpu().numpy()
        logs = {}
        for i, l in enumerate(self.layers):
            logs[l] = StepLog(
                pf_idx=a["pf_idx"][i].copy(), pf_count=a["pf_count"][i].copy(),
                route_idx=a["route_idx"][i].copy(), route_gate=a["route_gate"][i].copy(),
                exec_idx=a["exec_idx"][i].copy(), exec_gate=a["exec_gate"][i].copy(),
                resident=sorted(int(e) for e in a["resident"][i] if e >= 0),
                copies=int(a["n_copies"][i]),
                missing=[int(e) for e in a["missing"][i][:a["n_missing"][i]]], y=ys[i].copy())
        return logs

    def finish(self):
        native.apex_decode_finish(self.dec, self.stats)

    def reset_metrics(self):
        self.finish()
        self.stats = native.DecodeStats()

    def summary(self):
        s = self.stats
        tok = max(s.tokens, 1)
        ls = max(s.layer_steps, 1)
        return dict(recall=s.overlap_sum / tok, full_coverage=s.coverage_count / tok,
                    mean_delta_hat=s.delta_hat_sum / tok, hit_rate=s.hit_sum / tok,
                    copies_per_layer_step=s.copies / ls, misses_per_layer_step=s.misses / ls,
                    expert_bytes=self.S, tokens=int(s.tokens), layer_steps=int(s.layer_steps))

    def close(self):
        """Destroys the driver (which first waits for both streams) and drops every
        device and pinned buffer and the side stream this runner holds."""
        if getattr(self, "dec", None):
            native.apex_decode_destroy(self.dec)
            self.dec = None
        self.bufs = {}
        for name in ("exec_idx", "exec_gate", "y", "ws", "scratch", "miss_table", "side"):
            setattr(self, name, None)

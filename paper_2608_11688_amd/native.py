"""ctypes binding of the C ABI in include/apex.h (argument marshalling only).

Functions carry the C names.  Pointer arguments accept either an int address, a
torch tensor (its ``data_ptr()``), a numpy array (its buffer address) or None (NULL).
Streams are ``hipStream_t`` addresses (torch: ``stream.cuda_stream``) or None.
A non-OK status raises ``ApexError`` carrying the library's message.

The library is loaded on first use; if it has not been built this raises
``ApexLibraryMissing`` - there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os
import re

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
HEADER = os.path.join(ROOT, "include", "apex.h")
LIB_PATH = os.path.join(PKG, "libapex.so")
PLAN_LIB_PATH = os.path.join(PKG, "libapex_plan.so")

APEX_OK, APEX_E_INVAL, APEX_E_UNSUPPORTED, APEX_E_HIP, APEX_E_CAPACITY = 0, -1, -2, -3, -4
SEL_CUMPROB, SEL_ORDINAL_CDF, SEL_STATIC, SEL_NONE = 0, 1, 2, 3
MODE_EXACT, MODE_STALL_FREE = 0, 1
WEIGHTS_BF16, WEIGHTS_FP8_E4M3, WEIGHTS_MXFP4, WEIGHTS_FP32 = 0, 1, 2, 3
ABI_VERSION = 4
MAX_EXPERTS = 64
MAX_PAIRS = 1024
NOALLOC_WORKSPACE_BYTES = 64 << 20


class ApexError(RuntimeError):
    def __init__(self, fn, status, message):
        super().__init__(f"{fn} returned {status}: {message}")
        self.fn, self.status, self.message = fn, status, message


class ApexLibraryMissing(ImportError):
    pass


P = C.c_void_p
I32, I64, F32, F64, SZ = C.c_int, C.c_int64, C.c_float, C.c_double, C.c_size_t


class DecodeConfig(C.Structure):
    _fields_ = [(n, C.c_int) for n in ("L", "B", "d", "E", "k", "I", "C", "k_max", "policy")] + [
        ("tau", C.c_float), ("static_delta", C.c_int), ("mode", C.c_int),
        ("t_attn_us", C.c_double), ("n_scratch", C.c_int), ("weights", C.c_int),
        ("attn_heads", C.c_int), ("attn_kv_heads", C.c_int), ("attn_ctx", C.c_int),
        ("n_shared", C.c_int), ("I_shared", C.c_int)]


class DecodeLayer(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in (
        "w_pf", "w_g", "b_pf", "b_g", "cdf_w", "cdf_theta", "host_experts", "slots",
        "slot_of_expert_dev", "avail_dev", "expert_of_slot", "last_used", "w_qkv", "w_o",
        "k_cache", "v_cache", "attn_out", "shared_slots")]


class DecodeStats(C.Structure):
    _fields_ = [("overlap_sum", C.c_double), ("hit_sum", C.c_double),
                ("coverage_count", C.c_int64), ("delta_hat_sum", C.c_int64),
                ("tokens", C.c_int64), ("layer_steps", C.c_int64), ("copies", C.c_int64),
                ("misses", C.c_int64)]


class DecodeRecord(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in (
        "pf_idx", "pf_count", "route_idx", "route_gate", "exec_idx", "exec_gate", "resident",
        "n_copies", "missing", "n_missing")]

# name -> (restype, argtypes)
SIGNATURES = {
    "apex_abi_version": (C.c_int, []),
    "apex_last_error": (C.c_char_p, []),
    "apex_prefetch_route": (I32, [P, P, P, I32, I32, I32, I32, I32, I32, F32, I32, P, P, P, P, P,
                                  P]),
    "apex_gate_topk": (I32, [P, P, P, I32, I32, I32, I32, I32, P, I32, P, P, P, P, P, P]),
    "apex_expert_bytes": (SZ, [I32, I32]),
    "apex_pack_expert": (I32, [P, P, P, I32, I32, P]),
    "apex_expert_bytes_fp8": (SZ, [I32, I32]),
    "apex_pack_expert_fp8": (I32, [P, P, P, I32, I32, P]),
    "apex_expert_bytes_mxfp4": (SZ, [I32, I32]),
    "apex_pack_expert_mxfp4": (I32, [P, P, P, I32, I32, P]),
    "apex_expert_bytes_fp32": (SZ, [I32, I32]),
    "apex_pack_expert_fp32": (I32, [P, P, P, I32, I32, P]),
    "apex_moe_ffn_workspace_bytes": (SZ, [I32, I32, I32, I32]),
    "apex_moe_ffn": (I32, [P, I32, I32, I32, I32, I32, P, P, P, P, I32, P, I32, P, SZ, P]),
    "apex_moe_ffn_fp8": (I32, [P, I32, I32, I32, I32, I32, P, P, P, P, I32, P, I32, P, SZ, P]),
    "apex_moe_ffn_mxfp4": (I32, [P, I32, I32, I32, I32, I32, P, P, P, P, I32, P, I32, P, SZ, P]),
    "apex_moe_ffn_fp32": (I32, [P, I32, I32, I32, I32, I32, P, P, P, P, I32, P, I32, P, SZ, P]),
    "apex_moe_ffn_plan": (I32, [I32, I32, I32, I32, I32, I32, I32, P]),
    "apex_moe_ffn_noalloc": (I32, [P, I32, I32, I32, I32, I32, P, P, P, P, I32, I32, P, I32, P]),
    "apex_attention_workspace_bytes": (SZ, [I32, I32, I32, I32, I32]),
    "apex_attention_decode": (I32, [P, P, P, I32, I32, I32, I32, I32, P, P, I32, I32, P, P, SZ,
                                    P]),
    "apex_plan_residency": (I32, [I32, I32, P, P, I32, I32, I64, P, P, P, P, P]),
    "apex_expert_prefetch": (I32, [P, P, I32, I32, SZ, P, P, I32, I32, I64, P, P, P, P, P, P, P,
                                   P, P, P]),
    "apex_expert_fetch_misses": (I32, [P, P, I32, I32, I32, SZ, P, I32, I32, P, P, P, P, P, P, P,
                                       P]),
    "apex_decode_create": (I32, [P, C.POINTER(DecodeConfig), P, P, P, P, P, P, SZ, P, P]),
    "apex_decode_step": (I32, [P, I64, P, P, P, P, P]),
    "apex_decode_finish": (I32, [P, P]),
    "apex_decode_destroy": (I32, [P]),
    "apex_spin_us": (I32, [F64, P]),
    "apex_event_create": (I32, [P, I32]),
    "apex_event_destroy": (I32, [P]),
    "apex_event_record": (I32, [P, P]),
    "apex_event_synchronize": (I32, [P]),
    "apex_event_elapsed_ms": (I32, [P, P, P]),
    "apex_stream_wait_event": (I32, [P, P]),
    "apex_stream_synchronize": (I32, [P]),
    "apex_copy_kernel": (I32, [P, P, SZ, P]),
    "apex_read_kernel_sink_words": (SZ, [SZ]),
    "apex_read_kernel": (I32, [P, SZ, P, P]),
}

HOST_ONLY = ("apex_abi_version", "apex_last_error", "apex_expert_bytes", "apex_pack_expert",
             "apex_expert_bytes_fp8", "apex_pack_expert_fp8", "apex_expert_bytes_mxfp4",
             "apex_pack_expert_mxfp4", "apex_expert_bytes_fp32", "apex_pack_expert_fp32",
             "apex_plan_residency")


def header_functions(path=HEADER):
    """Names of the functions include/apex.h declares."""
    text = open(path).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(apex_[a-z0-9_]+)\s*\(", text)))


def _load(path, names):
    if not os.path.exists(path):
        raise ApexLibraryMissing(
            f"{os.path.basename(path)} is not built; run `python -m paper_2608_11688_amd.build`")
    lib = C.CDLL(path)
    for name in names:
        res, args = SIGNATURES[name]
        f = getattr(lib, name)
        f.restype, f.argtypes = res, args
    return lib


_lib = None
_plan_lib = None


def lib():
    global _lib
    if _lib is None:
        _lib = _load(LIB_PATH, SIGNATURES)
    return _lib


def plan_lib():
    """Host-only library (no HIP runtime needed)."""
    global _plan_lib
    if _plan_lib is None:
        _plan_lib = _load(PLAN_LIB_PATH, HOST_ONLY)
    return _plan_lib


def ptr(a):
    if a is None:
        return None
    if isinstance(a, int):
        return a
    if hasattr(a, "data_ptr"):
        return a.data_ptr()
    if hasattr(a, "ctypes"):
        return a.ctypes.data
    if isinstance(a, C.c_void_p):
        return a.value
    raise TypeError(f"cannot take the address of {type(a)}")


def _check(L, fn, st):
    if st != APEX_OK:
        raise ApexError(fn, st, L.apex_last_error().decode(errors="replace"))


def _call(name, *args, L=None):
    L = L or lib()
    _check(L, name, getattr(L, name)(*args))


def abi_version(L=None):
    return (L or lib()).apex_abi_version()


def apex_prefetch_route(h_pre, w_pf, b_pf, B, d, E, k, k_max, policy, tau, static_delta,
                        cdf_w, cdf_theta, pf_idx, pf_count, pf_prob, stream=None):
    _call("apex_prefetch_route", ptr(h_pre), ptr(w_pf), ptr(b_pf), B, d, E, k, k_max, policy,
          float(tau), static_delta, ptr(cdf_w), ptr(cdf_theta), ptr(pf_idx), ptr(pf_count),
          ptr(pf_prob), stream)


def apex_gate_topk(h_post, w_g, b_g, B, d, E, k, mode, avail, avail_stride, route_idx,
                   route_gate, exec_idx, exec_gate, gate_prob, stream=None):
    _call("apex_gate_topk", ptr(h_post), ptr(w_g), ptr(b_g), B, d, E, k, mode, ptr(avail),
          avail_stride, ptr(route_idx), ptr(route_gate), ptr(exec_idx), ptr(exec_gate),
          ptr(gate_prob), stream)


def apex_expert_bytes(d, I, L=None):
    return (L or lib()).apex_expert_bytes(d, I)


def apex_pack_expert(w1, w3, w2, d, I, out, L=None):
    _call("apex_pack_expert", ptr(w1), ptr(w3), ptr(w2), d, I, ptr(out), L=L)


def apex_expert_bytes_fp8(d, I, L=None):
    return (L or lib()).apex_expert_bytes_fp8(d, I)


def apex_pack_expert_fp8(w1, w3, w2, d, I, out, L=None):
    _call("apex_pack_expert_fp8", ptr(w1), ptr(w3), ptr(w2), d, I, ptr(out), L=L)


def apex_expert_bytes_mxfp4(d, I, L=None):
    return (L or lib()).apex_expert_bytes_mxfp4(d, I)


def apex_pack_expert_mxfp4(w1, w3, w2, d, I, out, L=None):
    _call("apex_pack_expert_mxfp4", ptr(w1), ptr(w3), ptr(w2), d, I, ptr(out), L=L)


def apex_expert_bytes_fp32(d, I, L=None):
    return (L or lib()).apex_expert_bytes_fp32(d, I)


def apex_pack_expert_fp32(w1, w3, w2, d, I, out, L=None):
    _call("apex_pack_expert_fp32", ptr(w1), ptr(w3), ptr(w2), d, I, ptr(out), L=L)


def apex_moe_ffn_workspace_bytes(B, d, I, k):
    return lib().apex_moe_ffn_workspace_bytes(B, d, I, k)


def apex_moe_ffn_plan(B, d, I, E, k, n_slots, weights="bf16"):
    """(token tiles per pass, gate/up K splits, down K splits) of a grouped call."""
    plan = (C.c_int32 * 3)()
    code = WEIGHT_FORMATS[weights][0] if isinstance(weights, str) else int(weights)
    _call("apex_moe_ffn_plan", B, d, I, E, k, n_slots, code, C.addressof(plan))
    return tuple(plan)


def apex_moe_ffn(x, B, d, I, E, k, exec_idx, exec_gate, slot_of_expert, slots, n_slots, y,
                 accumulate, workspace, workspace_bytes, stream=None):
    _call("apex_moe_ffn", ptr(x), B, d, I, E, k, ptr(exec_idx), ptr(exec_gate),
          ptr(slot_of_expert), ptr(slots), n_slots, ptr(y), int(accumulate), ptr(workspace),
          workspace_bytes, stream)


def apex_moe_ffn_fp8(x, B, d, I, E, k, exec_idx, exec_gate, slot_of_expert, slots, n_slots, y,
                     accumulate, workspace, workspace_bytes, stream=None):
    _call("apex_moe_ffn_fp8", ptr(x), B, d, I, E, k, ptr(exec_idx), ptr(exec_gate),
          ptr(slot_of_expert), ptr(slots), n_slots, ptr(y), int(accumulate), ptr(workspace),
          workspace_bytes, stream)


def apex_moe_ffn_mxfp4(x, B, d, I, E, k, exec_idx, exec_gate, slot_of_expert, slots, n_slots,
                       y, accumulate, workspace, workspace_bytes, stream=None):
    _call("apex_moe_ffn_mxfp4", ptr(x), B, d, I, E, k, ptr(exec_idx), ptr(exec_gate),
          ptr(slot_of_expert), ptr(slots), n_slots, ptr(y), int(accumulate), ptr(workspace),
          workspace_bytes, stream)


def apex_moe_ffn_fp32(x, B, d, I, E, k, exec_idx, exec_gate, slot_of_expert, slots, n_slots,
                      y, accumulate, workspace, workspace_bytes, stream=None):
    _call("apex_moe_ffn_fp32", ptr(x), B, d, I, E, k, ptr(exec_idx), ptr(exec_gate),
          ptr(slot_of_expert), ptr(slots), n_slots, ptr(y), int(accumulate), ptr(workspace),
          workspace_bytes, stream)


def apex_moe_ffn_noalloc(x, B, d, I, E, k, exec_idx, exec_gate, slot_of_expert, slots, n_slots,
                         weights, y, accumulate, stream=None):
    """weights: an APEX_WEIGHTS_* code or a format name ("bf16", "fp8", "mxfp4", "fp32")."""
    code = WEIGHT_FORMATS[weights][0] if isinstance(weights, str) else int(weights)
    _call("apex_moe_ffn_noalloc", ptr(x), B, d, I, E, k, ptr(exec_idx), ptr(exec_gate),
          ptr(slot_of_expert), ptr(slots), n_slots, code, ptr(y), int(accumulate), stream)


# weight format name -> (decode-driver code, bytes of one packed expert, packer, FFN entry)
WEIGHT_FORMATS = {
    "bf16": (WEIGHTS_BF16, "apex_expert_bytes", "apex_pack_expert", "apex_moe_ffn"),
    "fp8": (WEIGHTS_FP8_E4M3, "apex_expert_bytes_fp8", "apex_pack_expert_fp8", "apex_moe_ffn_fp8"),
    "mxfp4": (WEIGHTS_MXFP4, "apex_expert_bytes_mxfp4", "apex_pack_expert_mxfp4",
              "apex_moe_ffn_mxfp4"),
    "fp32": (WEIGHTS_FP32, "apex_expert_bytes_fp32", "apex_pack_expert_fp32", "apex_moe_ffn_fp32"),
}


def weight_format(name):
    """(code, expert_bytes(d, I), pack(w1, w3, w2, d, I, out), moe_ffn(...)) of a format."""
    if name not in WEIGHT_FORMATS:
        raise ValueError(f"weights must be one of {sorted(WEIGHT_FORMATS)}, not {name!r}")
    code, nbytes, pack, ffn = WEIGHT_FORMATS[name]
    g = globals()
    return code, g[nbytes], g[pack], g[ffn]


def apex_attention_workspace_bytes(B, H, G, hd, ctx_max):
    return lib().apex_attention_workspace_bytes(B, H, G, hd, ctx_max)


def apex_attention_decode(h, w_qkv, w_o, B, d, H, G, hd, k_cache, v_cache, ctx_max, pos, o,
                          workspace, workspace_bytes, stream=None):
    _call("apex_attention_decode", ptr(h), ptr(w_qkv), ptr(w_o), B, d, H, G, hd, ptr(k_cache),
          ptr(v_cache), ctx_max, pos, ptr(o), ptr(workspace), workspace_bytes, stream)


def apex_plan_residency(E, Cslots, pf_idx, pf_count, B, k_max, step, expert_of_slot, last_used,
                        copy_expert, copy_slot, L=None):
    n = C.c_int(0)
    _call("apex_plan_residency", E, Cslots, ptr(pf_idx), ptr(pf_count), B, k_max, step,
          ptr(expert_of_slot), ptr(last_used), ptr(copy_expert), ptr(copy_slot), C.byref(n), L=L)
    return n.value


def apex_expert_prefetch(host_experts, slots, E, Cslots, expert_bytes, pf_idx, pf_count, B,
                         k_max, step, expert_of_slot, last_used, slot_of_expert_dev, avail_dev,
                         side, compute, readers_done, ready, copied_experts=None):
    n = C.c_int(0)
    _call("apex_expert_prefetch", ptr(host_experts), ptr(slots), E, Cslots, expert_bytes,
          ptr(pf_idx), ptr(pf_count), B, k_max, step, ptr(expert_of_slot), ptr(last_used),
          ptr(slot_of_expert_dev), ptr(avail_dev), side, compute, readers_done, ready,
          ptr(copied_experts), C.byref(n))
    return n.value


def apex_expert_fetch_misses(host_experts, scratch, n_scratch, E, Cslots, expert_bytes,
                             route_idx, B, k, expert_of_slot, miss_table_dev, side, compute,
                             scratch_free, ready, missing=None):
    n = C.c_int(0)
    _call("apex_expert_fetch_misses", ptr(host_experts), ptr(scratch), n_scratch, E, Cslots,
          expert_bytes, ptr(route_idx), B, k, ptr(expert_of_slot), ptr(miss_table_dev), side,
          compute, scratch_free, ready, ptr(missing), C.byref(n))
    return n.value


def apex_decode_create(cfg, layers, scratch, miss_table, exec_idx, exec_gate, workspace,
                       workspace_bytes, compute, side):
    out = C.c_void_p()
    arr = (DecodeLayer * len(layers))(*layers)
    _call("apex_decode_create", C.byref(out), C.byref(cfg), arr, ptr(scratch), ptr(miss_table),
          ptr(exec_idx), ptr(exec_gate), ptr(workspace), workspace_bytes, compute, side)
    return out.value, arr


def apex_decode_step(dec, step, h_pre_ptrs, h_post_ptrs, y_ptrs, stats=None, record=None):
    _call("apex_decode_step", dec, step, h_pre_ptrs, h_post_ptrs, y_ptrs,
          None if stats is None else C.byref(stats), None if record is None else C.byref(record))


def apex_decode_finish(dec, stats=None):
    _call("apex_decode_finish", dec, None if stats is None else C.byref(stats))


def apex_decode_destroy(dec):
    _call("apex_decode_destroy", dec)


def apex_spin_us(us, stream=None):
    _call("apex_spin_us", float(us), stream)


def apex_event_create(timing=True):
    ev = C.c_void_p()
    _call("apex_event_create", C.byref(ev), int(timing))
    return ev.value


def apex_event_destroy(ev):
    _call("apex_event_destroy", ev)


def apex_event_record(ev, stream=None):
    _call("apex_event_record", ev, stream)


def apex_event_synchronize(ev):
    _call("apex_event_synchronize", ev)


def apex_event_elapsed_ms(start, stop):
    ms = C.c_float(0.0)
    _call("apex_event_elapsed_ms", start, stop, C.byref(ms))
    return ms.value


def apex_stream_wait_event(stream, ev):
    _call("apex_stream_wait_event", stream, ev)


def apex_stream_synchronize(stream=None):
    _call("apex_stream_synchronize", stream)


def apex_copy_kernel(dst, src, nbytes, stream=None):
    _call("apex_copy_kernel", ptr(dst), ptr(src), nbytes, stream)


def apex_read_kernel_sink_words(nbytes):
    return lib().apex_read_kernel_sink_words(nbytes)


def apex_read_kernel(src, nbytes, sink, stream=None):
    _call("apex_read_kernel", ptr(src), nbytes, ptr(sink), stream)

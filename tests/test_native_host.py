"""Host-side checks of the C ABI (CPU only, no compute calls).

* both libraries load and export every function include/apex.h declares;
* the C++ cache plan equals the oracle's replay, slot for slot;
* apex_pack_expert writes the documented slot layout;
* invalid arguments are rejected before anything is enqueued (no HIP call is made on
  these paths, so they run without a GPU).
"""

import numpy as np
import pytest

from oracle.residency import Residency
from paper_2608_11688_amd import native


@pytest.fixture(scope="module")
def plan_lib():
    return native.plan_lib()


@pytest.fixture(scope="module")
def hip_lib():
    return native.lib()


def test_header_lists_the_hot_path_entry_points():
    names = native.header_functions()
    for n in ("apex_prefetch_route", "apex_gate_topk", "apex_moe_ffn", "apex_expert_prefetch"):
        assert n in names
    assert set(names) == set(native.SIGNATURES), set(names) ^ set(native.SIGNATURES)


def test_libraries_export_every_declared_symbol(hip_lib, plan_lib):
    for name in native.header_functions():
        assert hasattr(hip_lib, name), name
    for name in native.HOST_ONLY:
        assert hasattr(plan_lib, name), name
    assert native.abi_version(hip_lib) == native.ABI_VERSION
    assert native.abi_version(plan_lib) == native.ABI_VERSION


@pytest.mark.parametrize("E,Cs,B,k_max,steps", [(8, 4, 1, 4, 60), (32, 16, 1, 16, 80),
                                                 (40, 16, 8, 16, 60), (64, 24, 16, 16, 40),
                                                 (64, 64, 64, 64, 10), (5, 5, 3, 2, 30)])
def test_cpp_plan_matches_oracle_replay(plan_lib, E, Cs, B, k_max, steps):
    rng = np.random.default_rng(E * 1000 + Cs * 10 + B)
    ref = Residency(E, Cs)
    eos = np.array([s if s < E else -1 for s in range(Cs)], np.int32)
    lu = np.full(E, -1, np.int64)
    ce = np.zeros(Cs, np.int32)
    cs = np.zeros(Cs, np.int32)
    for t in range(steps):
        pf_idx = np.full((B, k_max), -1, np.int32)
        pf_count = np.zeros(B, np.int32)
        lists = []
        for b in range(B):
            m = int(rng.integers(1, k_max + 1))
            lst = rng.choice(E, size=m, replace=False).astype(np.int32)
            pf_idx[b, :m] = lst
            pf_count[b] = m
            lists.append(list(lst))
        want = ref.plan(lists, t)
        n = native.apex_plan_residency(E, Cs, pf_idx, pf_count, B, k_max, t, eos, lu, ce, cs,
                                       L=plan_lib)
        assert [(int(ce[i]), int(cs[i])) for i in range(n)] == want
        assert list(eos) == ref.expert_of_slot
        assert list(lu) == ref.last_used


def test_plan_rejects_bad_tables_without_touching_outputs(plan_lib):
    eos = np.array([0, 0], np.int32)           # expert 0 in two slots
    lu = np.full(4, -1, np.int64)
    ce = np.full(2, 77, np.int32)
    cs = np.full(2, 77, np.int32)
    pf = np.array([[1]], np.int32)
    cnt = np.array([1], np.int32)
    with pytest.raises(native.ApexError) as ei:
        native.apex_plan_residency(4, 2, pf, cnt, 1, 1, 0, eos, lu, ce, cs, L=plan_lib)
    assert ei.value.status == native.APEX_E_INVAL and "two slots" in ei.value.message
    assert (ce == 77).all() and (lu == -1).all()
    eos = np.array([0, 1], np.int32)
    with pytest.raises(native.ApexError):
        native.apex_plan_residency(4, 2, np.array([[9]], np.int32), cnt, 1, 1, 0, eos, lu, ce,
                                   cs, L=plan_lib)
    assert list(eos) == [0, 1]


def test_pack_expert_layout(plan_lib):
    d, I = 16, 24
    rng = np.random.default_rng(3)
    w1 = rng.integers(0, 65535, (I, d), dtype=np.uint16)
    w3 = rng.integers(0, 65535, (I, d), dtype=np.uint16)
    w2 = rng.integers(0, 65535, (d, I), dtype=np.uint16)
    nbytes = native.apex_expert_bytes(d, I, L=plan_lib)
    assert nbytes == 6 * d * I
    out = np.zeros(nbytes // 2, np.uint16)
    native.apex_pack_expert(w1, w3, w2, d, I, out, L=plan_lib)
    rows = out[:2 * I * d].reshape(I, 2 * d)
    assert np.array_equal(rows[:, :d], w1) and np.array_equal(rows[:, d:], w3)
    assert np.array_equal(out[2 * I * d:].reshape(d, I), w2)


def _expect(status, fn, *args):
    with pytest.raises(native.ApexError) as ei:
        fn(*args)
    assert ei.value.status == status, ei.value
    return ei.value.message


def test_entry_points_validate_before_enqueue(hip_lib):
    A = 4096   # a fake, aligned, never-dereferenced address
    # prefetch route
    _expect(native.APEX_E_UNSUPPORTED, native.apex_prefetch_route, A, A, None, 1, 64, 65, 2, 4,
            0, 0.9, 0, None, None, A, A, None)
    _expect(native.APEX_E_INVAL, native.apex_prefetch_route, A, A, None, 1, 64, 8, 9, 9, 0, 0.9,
            0, None, None, A, A, None)
    _expect(native.APEX_E_INVAL, native.apex_prefetch_route, A, A, None, 1, 60, 8, 2, 4, 0, 0.9,
            0, None, None, A, A, None)
    _expect(native.APEX_E_INVAL, native.apex_prefetch_route, A, A, None, 1, 64, 8, 2, 4, 0, 1.5,
            0, None, None, A, A, None)
    _expect(native.APEX_E_INVAL, native.apex_prefetch_route, A, A, None, 1, 64, 8, 2, 4, 1, 0.9,
            0, None, None, A, A, None)       # ordinal without parameters
    _expect(native.APEX_E_INVAL, native.apex_prefetch_route, A + 4, A, None, 1, 64, 8, 2, 4, 0,
            0.9, 0, None, None, A, A, None)  # misaligned
    _expect(native.APEX_E_INVAL, native.apex_prefetch_route, A, A, None, 1, 64, 8, 2, 4, 0, 0.9,
            0, None, None, None, A, None)    # NULL output
    # gate
    _expect(native.APEX_E_INVAL, native.apex_gate_topk, A, A, None, 1, 64, 8, 2, 1, None, 0, A, A,
            A, A, None)                      # stall-free without a mask
    _expect(native.APEX_E_INVAL, native.apex_gate_topk, A, A, None, 1, 64, 8, 2, 1, A, 3, A, A,
            A, A, None)                      # stride below E
    _expect(native.APEX_E_INVAL, native.apex_gate_topk, A, A, None, 1, 64, 8, 2, 7, A, 0, A, A,
            A, A, None)                      # unknown mode
    # ffn
    msg = _expect(native.APEX_E_UNSUPPORTED, native.apex_moe_ffn, A, 129, 64, 64, 8, 8, A, A, A,
                  A, 1, A, 0, A, 1 << 30)
    assert "B*k" in msg
    _expect(native.APEX_E_CAPACITY, native.apex_moe_ffn, A, 2, 64, 64, 8, 2, A, A, A, A, 1, A, 0,
            A, 16)
    _expect(native.APEX_E_INVAL, native.apex_moe_ffn, A, 2, 64, 60, 8, 2, A, A, A, A, 1, A, 0, A,
            1 << 20)
    # the entry point without a workspace: a shape whose workspace exceeds its fixed array,
    # or an unknown weight format, is refused before any device call
    need = native.apex_moe_ffn_workspace_bytes(64, 4096, 14336, 16)
    assert need > native.NOALLOC_WORKSPACE_BYTES
    msg = _expect(native.APEX_E_CAPACITY, native.apex_moe_ffn_noalloc, A, 64, 4096, 14336, 16,
                  16, A, A, A, A, 1, "bf16", A, 0)
    assert "workspace" in msg
    _expect(native.APEX_E_INVAL, native.apex_moe_ffn_noalloc, A, 2, 64, 64, 8, 2, A, A, A, A, 1,
            7, A, 0)
    # B = 0 is a no-op that needs no device
    native.apex_prefetch_route(None, None, None, 0, 64, 8, 2, 4, 0, 0.9, 0, None, None, None,
                               None, None)
    native.apex_moe_ffn(None, 0, 64, 64, 8, 2, None, None, None, None, 1, None, 0, None, 0)
    # misses beyond scratch capacity are refused before any copy is enqueued
    eos = np.array([0, 1], np.int32)
    route = np.array([[2, 3]], np.int32)
    msg = _expect(native.APEX_E_CAPACITY, native.apex_expert_fetch_misses, A, A, 1, 4, 2, 96,
                  route, 1, 2, eos, A, None, None, None, A)
    assert "scratch" in msg


def test_workspace_size():
    small = native.apex_moe_ffn_workspace_bytes(1, 1024, 512, 8)
    assert small >= 8 * 512 * 4 and small % 256 == 0
    big = native.apex_moe_ffn_workspace_bytes(64, 2048, 1024, 8)   # batched path
    # bf16 h and fp32 per-pair outputs for 512 pairs, bf16 activations
    assert big >= 512 * (1024 * 2 + 2048 * 4) + 64 * 2048 * 2 and big % 256 == 0


def test_pack_expert_mxfp4_matches_the_oracle_quantiser(plan_lib):
    # the packed nibbles and block scales equal the oracle's own MXFP4 quantisation, byte
    # for byte, in the documented layout
    from oracle import mxfp4
    from oracle.bf16 import bf16_to_f64
    d, I = 96, 64
    rng = np.random.default_rng(42)

    def bf16(a):
        return (np.asarray(a, np.float32).view(np.uint32) >> 16).astype(np.uint16)
    w1 = bf16(rng.standard_normal((I, d)) * 0.02)
    w3 = bf16(rng.standard_normal((I, d)) * 1e-30)      # tiny blocks: very small exponents
    w2 = bf16(rng.standard_normal((d, I)) * 0.02)
    w1[5, 32:64] = 0                                     # an all-zero block
    w3[2, 3] = bf16([-1.0])[0]                           # a negative peak
    w2[7, :32] = bf16(np.linspace(-6.0, 6.0, 32))        # ties and the saturated top
    nbytes = native.apex_expert_bytes_mxfp4(d, I, L=plan_lib)
    assert nbytes == 3 * d * I // 2 + 3 * d * I // 32
    out = np.zeros(nbytes, np.uint8)
    native.apex_pack_expert_mxfp4(w1, w3, w2, d, I, out, L=plan_lib)
    rows = out[:I * d].reshape(I, d)                    # [W1 codes | W3 codes] per row
    c2 = out[I * d:3 * I * d // 2].reshape(d, I // 2)
    sc = out[3 * I * d // 2:]
    s1, s3, s2 = (sc[:I * d // 32].reshape(I, d // 32),
                  sc[I * d // 32:2 * I * d // 32].reshape(I, d // 32),
                  sc[2 * I * d // 32:].reshape(d, I // 32))
    for mat, codes, scales in ((w1, rows[:, :d // 2], s1), (w3, rows[:, d // 2:], s3),
                               (w2, c2, s2)):
        want_codes, X = mxfp4.quantize_blocks(bf16_to_f64(mat))
        assert np.array_equal(scales, mxfp4.scale_bytes(X))
        assert np.array_equal(codes, mxfp4.pack_nibbles(want_codes))
    assert s1[5, 1] == 0 and not rows[5, 16:32].any()
    with pytest.raises(native.ApexError):
        native.apex_pack_expert_mxfp4(w1, w3, w2, 80, I, out, L=plan_lib)  # d not a multiple of 32


def test_pack_expert_fp8_matches_the_oracle_quantiser(plan_lib):
    # the packed codes and scales equal the oracle's own E4M3 quantisation, byte for byte
    from oracle import fp8
    from oracle.bf16 import bf16_to_f64
    d, I = 48, 32
    rng = np.random.default_rng(41)
    def bf16(a):
        return (np.asarray(a, np.float32).view(np.uint32) >> 16).astype(np.uint16)
    w1 = bf16(rng.standard_normal((I, d)) * 0.02)
    w3 = bf16(rng.standard_normal((I, d)) * 3e-4)       # values reach the subnormal codes
    w2 = bf16(rng.standard_normal((d, I)) * 0.02)
    w1[5] = 0                                            # an all-zero row
    w3[2, 3] = bf16([-1.0])[0]                           # a negative peak
    nbytes = native.apex_expert_bytes_fp8(d, I, L=plan_lib)
    assert nbytes == 3 * d * I + 4 * (2 * I + d)
    out = np.zeros(nbytes, np.uint8)
    native.apex_pack_expert_fp8(w1, w3, w2, d, I, out, L=plan_lib)
    rows = out[:2 * I * d].reshape(I, 2 * d)
    c2 = out[2 * I * d:3 * I * d].reshape(d, I)
    sc = out[3 * I * d:].view(np.float32)
    for mat, codes, scales in ((w1, rows[:, :d], sc[:I]), (w3, rows[:, d:], sc[I:2 * I]),
                               (w2, c2, sc[2 * I:])):
        want_codes, want_scales = fp8.quantize_rows(bf16_to_f64(mat))
        assert np.array_equal(scales, want_scales)
        assert np.array_equal(codes, want_codes)
    assert sc[5] == 0 and not rows[5, :d].any()
    with pytest.raises(native.ApexError):
        native.apex_pack_expert_fp8(w1, w3, w2, 44, I, out, L=plan_lib)   # d not a multiple of 8


def test_pack_expert_fp32_widens_bf16_exactly(plan_lib):
    # the 32-bit slot holds the bf16 weights widened to fp32, bit for bit, in the bf16
    # slot's order
    d, I = 12, 20
    rng = np.random.default_rng(43)
    def bf16(a):
        return (np.asarray(a, np.float32).view(np.uint32) >> 16).astype(np.uint16)
    w1, w3 = bf16(rng.standard_normal((I, d))), bf16(rng.standard_normal((I, d)) * 1e-3)
    w2 = bf16(rng.standard_normal((d, I)) * 40.0)
    nbytes = native.apex_expert_bytes_fp32(d, I, L=plan_lib)
    assert nbytes == 12 * d * I
    out = np.zeros(nbytes // 4, np.uint32)
    native.apex_pack_expert_fp32(w1, w3, w2, d, I, out, L=plan_lib)
    widen = lambda w: w.astype(np.uint32) << 16
    rows = out[:2 * I * d].reshape(I, 2 * d)
    assert np.array_equal(rows[:, :d], widen(w1)) and np.array_equal(rows[:, d:], widen(w3))
    assert np.array_equal(out[2 * I * d:].reshape(d, I), widen(w2))
    with pytest.raises(native.ApexError):
        native.apex_pack_expert_fp32(w1, w3, w2, 10, I, out, L=plan_lib)   # d not a multiple of 4


def test_fp32_experts_run_at_batch1_only(hip_lib):
    # refused before anything is enqueued: more than one token, a size off the 4-value
    # grid, and the grouped plan for 32-bit experts
    A = 4096
    msg = _expect(native.APEX_E_UNSUPPORTED, native.apex_moe_ffn_fp32, A, 2, 64, 64, 8, 2, A, A,
                  A, A, 1, A, 0, A, 1 << 30)
    assert "batch 1" in msg
    _expect(native.APEX_E_UNSUPPORTED, native.apex_moe_ffn_noalloc, A, 2, 64, 64, 8, 2, A, A, A,
            A, 1, "fp32", A, 0)
    _expect(native.APEX_E_INVAL, native.apex_moe_ffn_fp32, A, 1, 64, 62, 8, 2, A, A, A, A, 1, A,
            0, A, 1 << 30)
    assert native.apex_moe_ffn_plan(1, 64, 64, 8, 2, 8, weights="fp32") == (0, 0, 0)
    with pytest.raises(native.ApexError) as ei:
        native.apex_moe_ffn_plan(2, 64, 64, 8, 2, 8, weights="fp32")
    assert ei.value.status == native.APEX_E_UNSUPPORTED


def test_moe_ffn_plan():
    # batch 1 takes the batch-1 kernels; bad arguments are errors
    assert native.apex_moe_ffn_plan(1, 2048, 1024, 64, 8, 24) == (0, 0, 0)
    with pytest.raises(native.ApexError):
        native.apex_moe_ffn_plan(8, 2048, 1024, 64, 8, 24, weights=7)
    with pytest.raises(native.ApexError):
        native.apex_moe_ffn_plan(8, 2048, 1024, 4, 8, 4)          # k > E
    # every plan the GPU parity test relies on is still taken by its shape (all of the
    # shape's experts resident; k = 2)
    from tests.ffn_plans import PLAN_CASES
    seen = set()
    for weights, B, d, I, E, plan in PLAN_CASES:
        assert native.apex_moe_ffn_plan(B, d, I, E, 2, E, weights) == plan, (weights, B, d, I)
        seen.add((weights, plan[0], plan[1] > 1, plan[2] > 1))
    assert len(seen) == 3 * 3 * 2 * 2
    # the workspace covers the largest plan of every format
    for weights, B, d, I, E, plan in PLAN_CASES:
        MT, SU, SD = plan
        P = B * 2
        need = (2 * SU * P * I * 4 if SU > 1 else 0) + P * I * 2 + SD * P * d * 4
        assert native.apex_moe_ffn_workspace_bytes(B, d, I, 2) >= need

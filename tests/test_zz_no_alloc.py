"""apex_moe_ffn_noalloc (the expert FFN with its workspace in a fixed device array)
against apex_moe_ffn with a caller workspace, through the C ABI.

Two calls in a row per weight format, the second with a smaller batch, so the second
call runs over what the first left in the shared array.  The results must equal the
workspace entry point's bit for bit (same kernels, same plan) and the oracle within the
FFN tolerance.
"""
import numpy as np
import pytest

from paper_2608_11688_amd import native
from tests.parity import ffn_close
from tests.test_gpu_kernels import FfnCase, shape

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    native.lib()
    return t


def run_noalloc(torch, case, y0=None, accumulate=0):
    cfg, B = case.cfg, case.B
    y = (torch.from_numpy(np.ascontiguousarray(y0)).cuda() if y0 is not None
         else torch.full((B, cfg.d), float("nan"), device="cuda"))
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    native.apex_moe_ffn_noalloc(dev(case.x), B, cfg.d, cfg.I, cfg.E, cfg.k, dev(case.exec_idx),
                                dev(case.gate), dev(case.table), case.pool, case.n_slots,
                                case.weights, y, accumulate)
    torch.cuda.synchronize()
    return y.cpu().numpy()


@pytest.mark.parametrize("weights,d,I", [("bf16", 1024, 512), ("fp8", 1040, 528),
                                          ("mxfp4", 1056, 544)])
def test_noalloc_equals_workspace_entry_point(torch, weights, d, I):
    cfg = shape(f"noalloc_{weights}", 480, d, 24, 6, I=I)
    for i, B in enumerate((40, 7, 1)):          # each call smaller than the one before
        case = FfnCase(torch, cfg, B, seed=900 + i, resident_frac=0.8, weights=weights)
        ref = case.run()
        got = run_noalloc(torch, case)
        assert np.array_equal(got.view(np.uint32), ref.view(np.uint32)), (weights, B)
        ffn_close(got, case.oracle(), f"noalloc {weights} B{B}")
        # the second pass of the miss correction: accumulate onto an existing output
        y0 = np.random.default_rng(B).standard_normal((B, d)).astype(np.float32)
        acc_ref = case.run(y0=y0, accumulate=1)
        acc = run_noalloc(torch, case, y0=y0, accumulate=1)
        assert np.array_equal(acc.view(np.uint32), acc_ref.view(np.uint32)), (weights, B)


def test_noalloc_fp32_batch1(torch):
    # 32-bit experts run at batch 1 only: two calls in a row, the second smaller
    for i, (d, I) in enumerate(((1028, 516), (516, 260))):
        cfg = shape(f"noalloc_fp32_{d}", 481 + i, d, 24, 6, I=I)
        case = FfnCase(torch, cfg, 1, seed=910 + i, weights="fp32")
        ref = case.run()
        got = run_noalloc(torch, case)
        assert np.array_equal(got.view(np.uint32), ref.view(np.uint32)), d
        ffn_close(got, case.oracle(), f"noalloc fp32 d{d}")


def test_noalloc_largest_workload_shape(torch):
    # the largest workspace any workload needs (Mixtral shape, 32 tokens: 34 MiB) fits,
    # checked on sampled tokens against the workspace entry point
    from paper_2608_11688_amd import configs
    cfg = configs.MIXTRAL
    assert native.apex_moe_ffn_workspace_bytes(32, cfg.d, cfg.I, cfg.k) <= \
        native.NOALLOC_WORKSPACE_BYTES
    case = FfnCase(torch, cfg, 32, seed=77)
    ref = case.run()
    got = run_noalloc(torch, case)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))

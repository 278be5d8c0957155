"""Comparison rules shared by the GPU parity tests.

Index sets: bit-exact, except where the oracle's deciding margin is below TIE (a
near tie: a logit gap, a prefix sum at tau, or an ordinal threshold); such cases are
counted and reported.  The excuse is bounded: at every point of a test the mismatches
excused so far may not exceed MAX_EXCUSED_FRAC of the rows checked so far (at least one
is allowed), so a margin that comes out too small cannot silence a whole test.
FFN outputs, per (layer, step) tile: max|y - y_ref| <= 1e-2 max|y_ref| and
sum|y - y_ref| / sum|y_ref| <= 5e-3 (bf16 weights, fp32 accumulation).
"""
import numpy as np

TIE = 1e-5
MAX_EXCUSED_FRAC = 0.01
FFN_MAX_REL = 1e-2
FFN_L1_REL = 5e-3


class TieLedger:
    def __init__(self):
        self.checked = 0
        self.flagged_mismatch = 0
        self.flagged = 0

    def compare_rows(self, gpu, ref, margin, what=""):
        gpu, ref = np.asarray(gpu), np.asarray(ref)
        assert gpu.shape == ref.shape, (what, gpu.shape, ref.shape)
        for b in range(gpu.shape[0]):
            self.checked += 1
            near = margin[b] < TIE
            self.flagged += int(near)
            if not np.array_equal(gpu[b], ref[b]):
                assert near, f"{what} row {b}: gpu {gpu[b]} != oracle {ref[b]} (margin {margin[b]:.3g})"
                self.flagged_mismatch += 1
                assert self.flagged_mismatch <= self.limit(), (
                    f"{what} row {b}: too many mismatches excused as near ties: {self}")

    def limit(self):
        return max(1, int(MAX_EXCUSED_FRAC * self.checked))

    def __repr__(self):
        return (f"TieLedger(checked={self.checked}, near_ties={self.flagged}, "
                f"mismatches_at_near_ties={self.flagged_mismatch})")


def ffn_close(y, y_ref, what=""):
    y = np.asarray(y, np.float64)
    y_ref = np.asarray(y_ref, np.float64)
    scale = np.abs(y_ref).max()
    err = np.abs(y - y_ref)
    if scale == 0:
        assert err.max() == 0, f"{what}: expected zeros, max |y| = {err.max()}"
        return 0.0, 0.0
    max_rel = err.max() / scale
    l1 = err.sum() / np.abs(y_ref).sum()
    assert max_rel <= FFN_MAX_REL, f"{what}: max-abs error {max_rel:.3g} of max|y_ref|"
    assert l1 <= FFN_L1_REL, f"{what}: relative L1 error {l1:.3g}"
    return max_rel, l1

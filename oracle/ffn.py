"""Oracle: SwiGLU expert FFN and the gated sum over the executed experts.

Test infrastructure only.  Float64 throughout, weights widened exactly from bf16.

Paper passages followed: Sec. III-A (each expert is a smaller FFN; the selected
experts process the token independently and their outputs are combined by a weighted
sum) and Sec. IV-E (the final aggregation uses the original router weights).
Reading: the expert FFN is SwiGLU without biases, FFN(x) = W2 (silu(W1 x) * (W3 x)),
silu(u) = u / (1 + exp(-u)), as the workload definitions state.

With weights="fp8" every expert matrix is first quantised row by row to E4M3 with an
fp32 scale per row (``fp8``, the reading taken for the precision study of Sec. V-G) and
the FFN runs on the dequantised values s_r * q, in float64.  With weights="mxfp4" every
row is quantised in blocks of 32 along the reduction dimension to E2M1 codes with a
power-of-two scale per block (``mxfp4``) and the FFN runs on 2^X * q.  With weights="fp32"
(the 32-bit point of the same study: the bf16 experts stored as fp32) the weights are the
bf16 values themselves, since bf16 widens to fp32 exactly.
"""
from __future__ import annotations

import numpy as np

from . import fp8, mxfp4
from .bf16 import bf16_to_f64


def silu(u):
    with np.errstate(over="ignore"):
        return u / (1.0 + np.exp(-u))


def swiglu_expert(x, w1, w3, w2):
    """One expert on one token: W2 (silu(W1 x) * (W3 x)).  Weights float64."""
    u = w1 @ x
    v = w3 @ x
    return w2 @ (silu(u) * v)


def moe_ffn(x, exec_idx, exec_gate, expert_bits, skip=None, weights="bf16"):
    """y[b] = sum_j g[b, j] FFN_{e[b, j]}(x[b]) over the executed experts.

    x: [B, d]; exec_idx int [B, k] (-1 = unused position); exec_gate [B, k];
    expert_bits(e) -> (W1 bits [I,d], W3 bits [I,d], W2 bits [d,I]);
    skip: optional set of expert ids left out (a pass that only covers some experts);
    weights: "bf16" or "fp32" (the weights as given), "fp8" (quantised per row first) or
    "mxfp4" (quantised per block of 32 along each row first).
    """
    if weights not in ("bf16", "fp8", "mxfp4", "fp32"):
        raise ValueError(f"unknown weight format {weights}")
    x = np.atleast_2d(np.asarray(x, dtype=np.float64))
    B, d = x.shape
    y = np.zeros((B, d))
    cache = {}
    for b in range(B):
        for j in range(exec_idx.shape[1]):
            e = int(exec_idx[b, j])
            if e < 0 or (skip is not None and e in skip):
                continue
            if e not in cache:
                ws = tuple(bf16_to_f64(w) for w in expert_bits(e))
                if weights == "fp8":
                    ws = tuple(fp8.dequantize_rows(*fp8.quantize_rows(w)) for w in ws)
                elif weights == "mxfp4":
                    ws = tuple(mxfp4.dequantize_blocks(*mxfp4.quantize_blocks(w)) for w in ws)
                cache[e] = ws
            w1, w3, w2 = cache[e]
            y[b] += float(exec_gate[b, j]) * swiglu_expert(x[b], w1, w3, w2)
    return y

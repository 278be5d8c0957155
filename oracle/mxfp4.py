"""Oracle: MXFP4 expert weights (4-bit E2M1 elements with one 8-bit power-of-two scale
per block of 32 values along a row).

Test infrastructure only (see the package docstring).

The format is the OCP Microscaling (MX) MXFP4 encoding.  An element is FP4 E2M1: a sign
bit, two exponent bits with bias 1 and one mantissa bit; exponent field 0 holds the
subnormal 0.5 * m, so the magnitudes are 0, 0.5, 1, 1.5, 2, 3, 4 and 6.  A block of 32
consecutive values shares an E8M0 scale 2^X (the byte X + 127).

Quantisation follows the precision study of Sec. V-G, which only scales the bytes of
every expert; the format is this implementation's reading (4-bit weights in the form
gfx950 converts in hardware), with the MX specification's conversion: for each block,
X = floor(log2(max |v|)) - 2 (2 being the largest exponent of E2M1), and every element
becomes the E2M1 value nearest to v / 2^X, ties to the even code, magnitudes above 6
clamped to 6, the sign bit set for negative inputs.  A block of zeros takes X = -127
(scale byte 0) and codes 0.  The weights are then 2^X * q exactly.
"""
from __future__ import annotations

import numpy as np

BLOCK = 32
EMAX = 2            # largest exponent of an E2M1 value (6 = 1.5 * 2^2)
MAX_FINITE = 6.0
SCALE_BIAS = 127


def decode(code: int) -> float:
    """Value of one E2M1 code (the low four bits of `code`)."""
    code = int(code) & 0xF
    sign = -1.0 if code & 0x8 else 1.0
    e = (code >> 1) & 0x3
    m = code & 0x1
    if e == 0:
        return sign * 0.5 * m
    return sign * (1.0 + 0.5 * m) * 2.0 ** (e - 1)


# magnitudes of the non-negative codes 0 .. 7, increasing with the code
_MAGNITUDES = np.array([decode(c) for c in range(8)], dtype=np.float64)


def encode(x) -> np.ndarray:
    """Nearest E2M1 code of every value (ties to the even code), saturating at 6."""
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(x), MAX_FINITE)
    hi = np.minimum(np.searchsorted(_MAGNITUDES, a, side="left"), len(_MAGNITUDES) - 1)
    lo = np.maximum(hi - 1, 0)
    d_lo = a - _MAGNITUDES[lo]
    d_hi = _MAGNITUDES[hi] - a
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    code = np.where(pick_hi, hi, lo).astype(np.uint8)
    return np.where(x < 0, code | np.uint8(0x8), code).astype(np.uint8)


def decode_array(codes) -> np.ndarray:
    table = np.array([decode(c) for c in range(16)], dtype=np.float64)
    return table[np.asarray(codes, dtype=np.uint8) & 0xF]


def block_exponents(W) -> np.ndarray:
    """X per block: W [rows, K] (K a multiple of 32) -> int [rows, K / 32]."""
    W = np.asarray(W, dtype=np.float64)
    rows, K = W.shape
    if K % BLOCK:
        raise ValueError(f"row length {K} is not a multiple of {BLOCK}")
    amax = np.abs(W).reshape(rows, K // BLOCK, BLOCK).max(axis=2)
    _, e = np.frexp(amax)                      # amax = f * 2^e, f in [0.5, 1)
    X = np.where(amax > 0, e - 1 - EMAX, -SCALE_BIAS)
    return np.clip(X, -SCALE_BIAS, SCALE_BIAS).astype(np.int64)


def quantize_blocks(W):
    """W [rows, K] -> (codes uint8 [rows, K], one per element; X int [rows, K / 32])."""
    W = np.asarray(W, dtype=np.float64)
    rows, K = W.shape
    X = block_exponents(W)
    scaled = W.reshape(rows, K // BLOCK, BLOCK) / np.ldexp(1.0, X)[:, :, None]
    return encode(scaled).reshape(rows, K), X


def dequantize_blocks(codes, X) -> np.ndarray:
    codes = np.asarray(codes)
    rows, K = codes.shape
    v = decode_array(codes).reshape(rows, K // BLOCK, BLOCK)
    return (v * np.ldexp(1.0, np.asarray(X))[:, :, None]).reshape(rows, K)


def pack_nibbles(codes) -> np.ndarray:
    """Two codes per byte along each row: element 2j in the low nibble of byte j."""
    codes = np.asarray(codes, dtype=np.uint8)
    return (codes[:, 0::2] & 0xF) | ((codes[:, 1::2] & 0xF) << 4)


def scale_bytes(X) -> np.ndarray:
    return (np.asarray(X) + SCALE_BIAS).astype(np.uint8)

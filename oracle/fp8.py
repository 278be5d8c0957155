"""Oracle: 8-bit E4M3 floating point and per-row quantisation of expert weights.

Test infrastructure only (see the package docstring).

The format is the OCP 8-bit floating-point E4M3 encoding: one sign bit, four exponent
bits with bias 7, three mantissa bits.  Exponent field 0 holds the subnormals m/8 * 2^-6;
exponent field 15 with mantissa 7 is NaN; there are no infinities, so the largest
finite magnitude is 1.75 * 2^8 = 448.

Quantisation follows the precision study of Sec. V-G, which only scales the bytes of
every expert; the format and the scaling are this implementation's reading: each output
row r of W1, W3 and W2 gets s_r = fp32(max |W[r, :]| / 448) and codes q = the E4M3 value
nearest to W[r, :] / s_r (ties to the even code, sign bit set for negative inputs), so
W[r, :] is approximated by s_r * q.  A row of zeros gets s_r = 0 and codes 0.
"""
from __future__ import annotations

import numpy as np

MAX_FINITE = 448.0


def decode(code: int) -> float:
    """Value of one E4M3 code (NaN for the two NaN codes)."""
    code = int(code) & 0xFF
    sign = -1.0 if code & 0x80 else 1.0
    e = (code >> 3) & 0xF
    m = code & 0x7
    if e == 0xF and m == 0x7:
        return float("nan")
    if e == 0:
        return sign * (m / 8.0) * 2.0 ** -6
    return sign * (1.0 + m / 8.0) * 2.0 ** (e - 7)


# magnitudes of the finite non-negative codes 0x00 .. 0x7E, increasing with the code
_MAGNITUDES = np.array([decode(c) for c in range(0x7F)], dtype=np.float64)


def encode(x) -> np.ndarray:
    """Nearest E4M3 code of every value (ties to the even code); |x| <= 448 expected,
    larger magnitudes saturate to 448."""
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(x), MAX_FINITE)
    hi = np.searchsorted(_MAGNITUDES, a, side="left")          # first magnitude >= a
    hi = np.minimum(hi, len(_MAGNITUDES) - 1)
    lo = np.maximum(hi - 1, 0)
    d_lo = a - _MAGNITUDES[lo]
    d_hi = _MAGNITUDES[hi] - a
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    code = np.where(pick_hi, hi, lo).astype(np.uint8)
    return np.where(x < 0, code | np.uint8(0x80), code).astype(np.uint8)


def decode_array(codes) -> np.ndarray:
    table = np.array([decode(c) for c in range(256)], dtype=np.float64)
    return table[np.asarray(codes, dtype=np.uint8)]


def quantize_rows(W):
    """(codes uint8 [R, K], scales float32 [R]) for the rows of W."""
    W = np.asarray(W, dtype=np.float64)
    peak = np.abs(W).max(axis=1)
    scales = (peak / MAX_FINITE).astype(np.float32)
    s = scales.astype(np.float64)
    safe = np.where(s > 0, s, 1.0)
    codes = encode(W / safe[:, None])
    codes[s == 0] = 0
    return codes, scales


def dequantize_rows(codes, scales) -> np.ndarray:
    return decode_array(codes) * np.asarray(scales, dtype=np.float64)[:, None]

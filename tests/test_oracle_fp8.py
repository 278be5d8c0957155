"""Pins of the oracle's E4M3 codec and per-row quantisation (CPU only).

* code values fixed by the format definition (1.0, 448, the smallest normal and
  subnormal, -2, the NaN codes, negative zero);
* ties to the even code at exact midpoints;
* agreement with torch's float8_e4m3fn conversion on in-range values (a library routine
  with the same rounding);
* every finite code survives decode -> encode;
* quantised rows: the largest element maps to +-448 exactly, the error of every element
  is at most half the code spacing at its magnitude times the row scale, zero rows stay
  zero.
"""
import math

import numpy as np
import pytest

from oracle import fp8


def test_codes_from_the_format_definition():
    assert fp8.decode(0x38) == 1.0
    assert fp8.decode(0x7E) == 448.0
    assert fp8.decode(0x08) == 2.0 ** -6            # smallest normal
    assert fp8.decode(0x01) == 2.0 ** -9            # smallest subnormal
    assert fp8.decode(0x07) == 7 * 2.0 ** -9        # largest subnormal
    assert fp8.decode(0xC0) == -2.0
    assert fp8.decode(0x3C) == 1.5
    assert math.isnan(fp8.decode(0x7F)) and math.isnan(fp8.decode(0xFF))
    z = fp8.decode(0x80)
    assert z == 0.0 and math.copysign(1.0, z) == -1.0


def test_ties_go_to_the_even_code():
    # 1.0625 lies halfway between 1.0 (0x38) and 1.125 (0x39)
    assert fp8.encode([1.0625])[0] == 0x38
    # 1.1875 lies halfway between 1.125 (0x39) and 1.25 (0x3A)
    assert fp8.encode([1.1875])[0] == 0x3A
    # halfway between the two smallest subnormals
    assert fp8.encode([1.5 * 2.0 ** -9])[0] == 0x02
    assert fp8.encode([0.5 * 2.0 ** -9])[0] == 0x00
    assert fp8.encode([-1.0625])[0] == 0xB8
    # just past a midpoint rounds up
    assert fp8.encode([np.nextafter(1.0625, 2.0)])[0] == 0x39


def test_agrees_with_torch_float8_e4m3fn():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(31)
    x = np.concatenate([
        rng.uniform(-448, 448, 20000),
        rng.standard_normal(20000) * 2.0 ** -7,           # subnormal and small normals
        np.array([fp8.decode(c) for c in range(0x7F)]) * 1.0,
        # exact midpoints between neighbouring codes
        0.5 * (np.array([fp8.decode(c) for c in range(0x7E)]) +
               np.array([fp8.decode(c + 1) for c in range(0x7E)])),
    ])
    want = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    got = fp8.encode(x)
    # the one convention that differs: torch keeps the sign of a negative value that
    # rounds to zero, and so does the oracle (sign bit for every x < 0)
    assert np.array_equal(got, want)


def test_every_finite_code_round_trips():
    codes = [c for c in range(256) if c not in (0x7F, 0xFF)]
    vals = np.array([fp8.decode(c) for c in codes])
    back = fp8.encode(vals)
    for c, b, v in zip(codes, back, vals):
        if v == 0.0:
            assert b in (0x00, 0x80)
        else:
            assert b == c


def test_row_quantisation_error_bound():
    rng = np.random.default_rng(32)
    W = rng.standard_normal((40, 96)) * 0.02
    W[3] = 0.0
    W[5, 7] = -0.5                                     # a row whose peak is negative
    codes, scales = fp8.quantize_rows(W)
    assert scales.dtype == np.float32 and scales[3] == 0 and not codes[3].any()
    deq = fp8.dequantize_rows(codes, scales)
    for r in range(W.shape[0]):
        if scales[r] == 0:
            assert not deq[r].any()
            continue
        peak = np.abs(W[r]).argmax()
        assert codes[r, peak] & 0x7F == 0x7E           # the peak maps to +-448
        q = W[r] / float(scales[r])
        # half the spacing between neighbouring codes at each magnitude
        e = np.floor(np.log2(np.maximum(np.abs(q), 2.0 ** -6)))
        half_ulp = 0.5 * 2.0 ** (e - 3)
        assert np.all(np.abs(q - deq[r] / float(scales[r])) <= half_ulp * (1 + 1e-12))

"""Pins of the oracle's MXFP4 codec (CPU only): OCP MX FP4 E2M1 elements with an E8M0
scale per block of 32 values.

* the element values from the format definition (the eight magnitudes the MX
  specification lists for E2M1) and the sign bit;
* rounding against brute force over every code, ties to the even code, saturation;
* the block exponent rule on hand-made blocks, and the error bound it implies;
* representable blocks round-trip exactly; nibble order (element 2j in the low nibble).
"""
import numpy as np
import pytest

from oracle import mxfp4


def test_element_values_from_the_format_definition():
    assert [mxfp4.decode(c) for c in range(8)] == [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]
    assert [mxfp4.decode(c | 8) for c in range(1, 8)] == [-0.5, -1.0, -1.5, -2.0, -3.0, -4.0,
                                                          -6.0]
    z = mxfp4.decode(8)
    assert z == 0.0 and np.signbit(z)


def brute_force_code(v):
    """The code whose value is nearest to v among all 16 (ties: the code with an even
    mantissa bit), found by trying every code; magnitudes above 6 take 6."""
    a = min(abs(v), 6.0)
    best = None
    for c in range(8):
        dist = abs(a - mxfp4.decode(c))
        key = (dist, c & 1)          # nearer first, then the even mantissa bit
        if best is None or key < best[0]:
            best = (key, c)
    return best[1] | (8 if v < 0 else 0)


def test_rounding_matches_brute_force():
    rng = np.random.default_rng(71)
    v = np.concatenate([rng.uniform(-7.5, 7.5, 4000),
                        np.arange(-6.0, 6.25, 0.25),          # every tie point on the grid
                        [0.0, 6.0, -6.0, 8.0, -100.0]])
    got = mxfp4.encode(v)
    want = np.array([brute_force_code(x) for x in v], dtype=np.uint8)
    assert np.array_equal(got, want)


def test_ties_go_to_the_even_code():
    ties = {0.25: 0, 0.75: 2, 1.25: 2, 1.75: 4, 2.5: 4, 3.5: 6, 5.0: 6}
    for v, c in ties.items():
        assert mxfp4.encode([v])[0] == c, v
        assert mxfp4.encode([-v])[0] == c | 8, -v
        # off the tie the nearer neighbour wins: the grid values on either side
        below = mxfp4.decode(mxfp4.encode([np.nextafter(v, 0.0)])[0])
        above = mxfp4.decode(mxfp4.encode([np.nextafter(v, 10.0)])[0])
        assert below < v < above, (v, below, above)
    assert mxfp4.encode([6.9])[0] == 7 and mxfp4.encode([1e9])[0] == 7


def test_block_exponent_rule():
    W = np.zeros((4, 64))
    W[0, 3] = 1.0              # max 1 = 2^0: X = 0 - 2
    W[1, 40] = -6.0            # max 6 in [4, 8): X = 2 - 2 = 0
    W[2, :32] = 7.99           # max just under 8: X = 0, the elements clamp to 6
    X = mxfp4.block_exponents(W)
    assert X.tolist() == [[-2, -127], [-127, 0], [0, -127], [-127, -127]]
    codes, X = mxfp4.quantize_blocks(W)
    deq = mxfp4.dequantize_blocks(codes, X)
    assert deq[0, 3] == 1.0 and deq[1, 40] == -6.0
    assert np.all(deq[2, :32] == 6.0) and np.all(deq[3] == 0.0)
    assert np.array_equal(mxfp4.scale_bytes(X)[0], [125, 0])


def test_quantisation_error_bound():
    rng = np.random.default_rng(72)
    W = rng.standard_normal((64, 256)) * 0.02
    codes, X = mxfp4.quantize_blocks(W)
    deq = mxfp4.dequantize_blocks(codes, X)
    step = np.repeat(np.ldexp(1.0, X), mxfp4.BLOCK, axis=1)
    err = np.abs(deq - W)
    scaled = np.abs(W) / step
    # half the widest gap of the grid (4 .. 6) inside the range, and below 2 steps in
    # the clamped band [6, 8)
    assert np.all(err[scaled <= 6.0] <= step[scaled <= 6.0] * 1.0)
    assert np.all(err <= 2.0 * step)
    assert np.all(scaled < 8.0)


def test_representable_blocks_round_trip():
    rng = np.random.default_rng(73)
    codes = rng.integers(0, 16, size=(8, 64)).astype(np.uint8)
    codes[:, 0] = 7                          # every block holds a 6: its own exponent
    codes[:, 32] = 15
    X = rng.integers(-20, 5, size=(8, 2))
    W = mxfp4.dequantize_blocks(codes, X)
    c2, X2 = mxfp4.quantize_blocks(W)
    assert np.array_equal(X2, X)
    assert np.array_equal(mxfp4.decode_array(c2), mxfp4.decode_array(codes))


def test_nibble_order():
    codes = np.array([[1, 2, 3, 4]], np.uint8)
    assert mxfp4.pack_nibbles(codes).tolist() == [[0x21, 0x43]]


def test_rows_must_hold_whole_blocks():
    with pytest.raises(ValueError):
        mxfp4.block_exponents(np.zeros((2, 48)))


def test_ffn_on_representable_weights_is_the_bf16_ffn():
    # weights that are MXFP4 values in blocks along each row's reduction dimension (d for
    # W1 and W3, I for W2) quantise to themselves, so the FFN equals the bf16 one; a
    # quantiser working along the other axis would change them
    from oracle import ffn
    from paper_2608_11688_amd.inputs import to_bf16_bits
    rng = np.random.default_rng(74)
    d, I = 64, 96

    def representable(rows, cols):
        codes = rng.integers(0, 16, size=(rows, cols)).astype(np.uint8)
        codes[:, ::32] = 7                    # each block's largest magnitude is 6
        X = rng.integers(-9, -5, size=(rows, cols // 32))
        return to_bf16_bits(mxfp4.dequantize_blocks(codes, X).astype(np.float32))

    bits = {e: (representable(I, d), representable(I, d), representable(d, I)) for e in range(3)}
    x = rng.standard_normal((2, d))
    idx = np.array([[0, 2], [1, 0]])
    g = np.array([[0.7, 0.3], [0.5, 0.5]])
    a = ffn.moe_ffn(x, idx, g, lambda e: bits[e], weights="mxfp4")
    b = ffn.moe_ffn(x, idx, g, lambda e: bits[e], weights="bf16")
    assert np.array_equal(a, b)
    # and a generic expert does change under quantisation
    rnd = {0: tuple(to_bf16_bits((rng.standard_normal(s) * 0.02).astype(np.float32))
                    for s in ((I, d), (I, d), (d, I)))}
    c = ffn.moe_ffn(x, idx[:, :1] * 0, g[:, :1], lambda e: rnd[e], weights="mxfp4")
    e_ = ffn.moe_ffn(x, idx[:, :1] * 0, g[:, :1], lambda e: rnd[e], weights="bf16")
    assert not np.array_equal(c, e_)

"""Pins for the INT4 oracle (CPU).

Round-to-nearest (Section 3.3) is pinned by brute force over the whole code
grid (nearest point, ties to the even code), the RDN error bound of Table 1
(|x - s q| <= s/2 inside the range), symmetry, power-of-two equivariance and
the range of Appendix A.1 (alpha = Delta / (2^b - 1) for the unsigned grid).
"""
import numpy as np
import pytest

import synth
from oracle.int4 import int4_quantize, int4_decode_int, int4_decode


def _nearest_even(v, lo, hi):
    """Brute force: the grid integer in [lo, hi] nearest to v, ties to even."""
    best = None
    for q in range(lo, hi + 1):
        d = abs(float(v) - q)
        if best is None or d < best[0] or (d == best[0] and q % 2 == 0):
            best = (d, q)
    return best[1]


@pytest.mark.parametrize("signed", [True, False])
def test_brute_force_nearest_grid_point(signed):
    x = synth.normal((3001,), 1.0, [5, 1]) if signed else synth.half_normal((3001,), [5, 2])
    x[:8] = [0.0, -0.0, 1e-30, -1e-30, 0.5, -0.5, 2.5, -2.5]
    codes, s = int4_quantize(x, is_signed=signed)
    q = int4_decode_int(codes, x.size, signed)
    Q = 7 if signed else 15
    m = np.float32(np.abs(x).max() if signed else max(x.max(), 0))
    inv = np.float32(np.float32(Q) / m)
    lo = -7 if signed else 0
    for xi, qi in zip(x, q):
        v = np.float32(np.float32(xi) * inv)
        assert qi == _nearest_even(v, lo, Q), (xi, qi, v)


@pytest.mark.parametrize("signed", [True, False])
def test_rdn_error_bound_and_range(signed):
    x = synth.normal((50000,), 0.7, [6, 1])
    codes, s = int4_quantize(x, is_signed=signed)
    q = int4_decode_int(codes, x.size, signed)
    Q = 7 if signed else 15
    m = np.abs(x).max() if signed else x.max()
    assert float(s) == float(np.float32(np.float32(m) / np.float32(Q)))
    assert q.min() >= (-7 if signed else 0) and q.max() <= Q
    inside = x >= 0 if not signed else np.ones(x.size, bool)
    err = np.abs(x[inside].astype(np.float64) - q[inside] * float(s))
    assert np.all(err <= float(s) * (0.5 + 1e-5))          # Table 1: RDN bias <= half a bin
    # the extreme element maps to the end of the grid
    k = np.argmax(np.abs(x)) if signed else np.argmax(x)
    assert abs(q[k]) == Q
    if not signed:
        assert np.all(q[x <= 0] == 0)


def test_signed_symmetry_and_equivariance():
    x = synth.normal((4001,), 1.0, [7, 1])
    c0, s0 = int4_quantize(x, is_signed=True)
    c1, s1 = int4_quantize(-x, is_signed=True)
    assert np.array_equal(int4_decode_int(c0, x.size, True), -int4_decode_int(c1, x.size, True))
    assert s0 == s1
    for e in (-30, -4, 9):
        c2, s2 = int4_quantize((x * np.float32(2.0 ** e)).astype(np.float32), is_signed=True)
        assert np.array_equal(c0, c2) and float(s2) == float(s0) * 2.0 ** e


def test_clip_and_degenerate():
    x = synth.normal((1001,), 1.0, [8, 1])
    codes, s = int4_quantize(x, is_signed=True, clip=0.5)
    q = int4_decode_int(codes, x.size, True)
    assert np.all(q[x >= 0.5] == 7) and np.all(q[x <= -0.5] == -7)
    assert float(s) == float(np.float32(np.float32(0.5) / np.float32(7)))
    c, s = int4_quantize(np.zeros(9, np.float32), is_signed=True)
    assert s == 0 and not c.any()
    c, s = int4_quantize(-np.ones(9, np.float32), is_signed=False)
    assert s == 0 and not c.any()
    y = x.copy()
    y[3] = np.nan
    c, s = int4_quantize(y, is_signed=True)
    assert np.isnan(s) and not c.any()
    # bf16 input is the same as its exact float32 value
    xb = synth.to_bf16_bits(x)
    cb, sb = int4_quantize(xb, dtype="bf16", is_signed=True)
    cf, sf = int4_quantize(synth.bf16_bits_to_f32(xb), is_signed=True)
    assert np.array_equal(cb, cf) and sb == sf


def test_twos_complement_nibbles():
    x = np.array([-7, -1, 0, 1, 7, -3, 3], np.float32)
    codes, s = int4_quantize(x, is_signed=True)
    assert s == 1.0
    assert list(codes) == [0x9 | (0xF << 4), 0x0 | (0x1 << 4), 0x7 | (0xD << 4), 0x3]
    assert list(int4_decode(codes, 7, s, True)) == list(x)

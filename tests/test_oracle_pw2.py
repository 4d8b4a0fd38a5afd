"""Pins of the oracle's power-of-two LUQ (Appendix, "Power-of-two LUQ").

alpha_PW2 = 2^ceil(log2 max|x|) / 2^R: checked against a brute-force search
for the least power of two at or above the maximum (exact rationals, over
normal, subnormal, power-of-two and extreme maxima), the reduction to plain
LUQ when the maximum is itself a power of two, the exact rational field of
every element, no clipping of the maximum, unbiasedness, and the
combination with the in-hindsight maximum.
"""
from fractions import Fraction

import numpy as np
import pytest

import synth
from oracle.luq import (luq_quantize, luq_quantize_hindsight, luq_alpha_pw2, luq_alpha, luq_field_scalar,
                        unpack_nibbles, luq_decode)
from oracle.philox import luq_uniforms


def _least_pow2_at_or_above(m):
    P = Fraction(1)
    while P < m:
        P *= 2
    while P / 2 >= m:
        P /= 2
    return P


MAXIMA = [1.0, 0.75, 1.5, 2.0, 3.0, 1.0000001, 0.99999994, 16.0, 17.0, 1e-3, 6.1e-5, 3.4e38, 2.0 ** 127,
          1.7e38, 1e-38, 1.17549435e-38, 1e-40, 1.4e-45, 2.0 ** -140, 3 * 2.0 ** -149, 123.456]


@pytest.mark.parametrize("R", [4, 5, 6])
def test_alpha_is_least_power_of_two_at_or_above_max_over_2R(R):
    for m in MAXIMA:
        m32 = np.float32(m)
        mf = Fraction(float(m32))
        P = _least_pow2_at_or_above(mf)
        a = luq_alpha_pw2(m32, R)
        want = P / 2 ** R
        if want >= Fraction(2) ** -149:
            assert Fraction(float(a)) == want, (m, a)
        else:  # 2^(c-R) below the float32 subnormal range: rounds to 0
            assert a == 0, (m, a)
    assert luq_alpha_pw2(np.float32(0.0), 4) == 0


def test_power_of_two_max_reduces_to_plain_luq():
    x = synth.grad_1d(5000, "f32", 0.2, seed=31)
    x = (x / np.abs(x).max() * np.float32(2.0 ** -7)).astype(np.float32)  # max exactly 2^-7
    assert np.abs(x).max() == np.float32(2.0 ** -7)
    c0, a0, _ = luq_quantize(x, R=4, seed=2, counter=1)
    c1, a1, _ = luq_quantize(x, R=4, seed=2, counter=1, pw2=True)
    assert a0 == a1 and np.array_equal(c0, c1)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_fields_match_rational_restatement(dtype):
    x = synth.grad_1d(700, dtype, 0.2, seed=33)
    codes, alpha, m = luq_quantize(x, dtype=dtype, R=4, seed=9, counter=2, pw2=True)
    xf = synth.bf16_bits_to_f32(x) if dtype == "bf16" else x
    assert Fraction(float(alpha)) * 16 == _least_pow2_at_or_above(Fraction(float(m)))
    nib = unpack_nibbles(codes[0], x.size)
    j = luq_uniforms(x.size, 9, 2, 0)
    for i in range(x.size):
        e = luq_field_scalar(abs(float(xf[i])), float(alpha), 4, int(j[i]))
        assert int(nib[i]) == (e | (8 if (e and np.signbit(xf[i])) else 0)), i


def test_max_is_not_clipped_and_levels_are_powers_of_two():
    x = np.array([3.0, -0.2, 0.01, 1.1, -2.9, 0.0], np.float32)   # max 3 -> top level 4
    for c in range(64):
        codes, alpha, _ = luq_quantize(x, R=4, seed=1, counter=c, pw2=True)
        assert alpha == np.float32(0.25)
        v = luq_decode(codes[0], x.size, alpha)
        assert abs(v[0]) in (2.0, 4.0) and abs(v[4]) in (2.0, 4.0)
        nz = np.abs(v[v != 0])
        assert np.all(np.log2(nz) == np.round(np.log2(nz)))


def test_unbiased():
    x = np.array([3.0, -0.7, 1.1, 1.9, 0.01, -0.049, 0.26], np.float32)
    acc = np.zeros(x.size)
    reps = 300
    for c in range(reps):
        codes, a, _ = luq_quantize(np.tile(x, 64), R=4, seed=7, counter=c, pw2=True)
        acc += luq_decode(codes[0], x.size * 64, a).reshape(64, x.size).mean(axis=0)
    mean = acc / reps
    alpha = 0.25
    for xi, mi in zip(x.astype(np.float64), mean):
        levels = [0.0] + [alpha * 2 ** k for k in range(5)]
        mag = abs(xi)
        lo = max(v for v in levels if v <= mag)
        hi = min(v for v in levels if v > mag)
        sd = np.sqrt((mag - lo) * (hi - mag) / (64.0 * reps))
        assert abs(mi - xi) <= 5 * sd + (hi - lo) * 2.0 ** -16, (xi, mi)


@pytest.mark.parametrize("ns", [1, 2])
def test_hindsight_with_true_max_equals_pw2(ns):
    x = synth.grad_1d(2001, "f32", 0.3, seed=34)
    c, a, m = luq_quantize(x, R=5, seed=3, counter=4, n_samples=ns, pw2=True)
    ch, ah, mh, _ = luq_quantize_hindsight(x, m, R=5, seed=3, counter=4, n_samples=ns, pw2=True)
    assert np.array_equal(c, ch) and a == ah and m == mh
    # an estimate below the maximum: alpha from the estimate, larger magnitudes clip to the top
    ch, ah, _, _ = luq_quantize_hindsight(x, m * np.float32(0.3), R=5, seed=3, counter=4, pw2=True)
    assert ah == luq_alpha_pw2(m * np.float32(0.3), 5) and ah >= luq_alpha(m * np.float32(0.3), 5)

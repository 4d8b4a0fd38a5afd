"""Pins for the summed SMP operand of the oracle (``luq.luq_smp_sum``, CPU).

Section 5.1 averages n independent LUQ samples taken with one alpha; the
summed form keeps alpha / n outside and stores the per-element sum of the
decoded samples.  Pinned by: a bit-level decoder of the two planes written
here (sign bit 3, field bits 0..2, value +-2^(e-1)); the grid bracketing of
every element (each sample is one of the two grid points around |x|, so the
sum is 2l, l + u or 2u with the sign of x); the mean of (alpha / 2) * sum
against x and its variance against half the single-sample closed form
(x - l)(u - x); and a planted sign error that the bracketing pin catches.
"""
import math

import numpy as np
import pytest

import synth
from oracle.luq import luq_quantize, luq_smp_sum


def _bits_value(byte, high):
    nib = (int(byte) >> 4) if high else (int(byte) & 0xF)
    e = nib & 7
    if e == 0:
        return 0
    return -(1 << (e - 1)) if nib & 8 else (1 << (e - 1))


def _grid_bracket(a, alpha, R):
    """Grid points (in units of alpha) around a >= 0: 0, 1, 2, 4, ..., 2^R."""
    if a == 0:
        return 0, 0
    q = a / alpha
    if q >= 2 ** R:
        return 2 ** R, 2 ** R
    if q < 1:
        return 0, 1
    k = int(math.floor(math.log2(q)))
    while 2.0 ** k > q:
        k -= 1
    while 2.0 ** (k + 1) <= q:
        k += 1
    return 2 ** k, 2 ** (k + 1)


@pytest.mark.parametrize("R", [4, 5])
def test_sum_equals_bitwise_decoded_planes(R):
    x = synth.lognormal_grad((301,), -9.0, 2.5, 0.2, [5, R])
    planes, alpha, _ = luq_quantize(x, R=R, seed=3, counter=9, n_samples=2)
    s = luq_smp_sum(planes, x.size)
    assert s.dtype == np.int8 and s.shape == (x.size,)
    for i in range(x.size):
        want = sum(_bits_value(planes[p][i // 2], i & 1) for p in range(2))
        assert int(s[i]) == want


@pytest.mark.parametrize("R", [4, 5])
def test_sum_is_two_grid_points_with_the_sign_of_x(R):
    x = synth.lognormal_grad((4000,), -9.0, 3.0, 0.25, [6, R])
    planes, alpha, _ = luq_quantize(x, R=R, seed=11, counter=2, n_samples=2)
    s = luq_smp_sum(planes, x.size).astype(np.int64)
    assert np.all(np.abs(s) <= 2 ** (R + 1))
    for i in range(x.size):
        lo, hi = _grid_bracket(abs(float(x[i])), float(alpha), R)
        assert abs(int(s[i])) in (2 * lo, lo + hi, 2 * hi), (i, x[i], s[i])
        if s[i] != 0:
            assert (s[i] < 0) == bool(np.signbit(x[i]))


def test_sum_unbiased_and_variance_half_of_one_sample():
    reps = 1 << 18
    probes = [0.3, 1.5, 3.0, 6.5, 11.0, -2.25]
    x = np.concatenate([np.array([16.0], np.float32), np.repeat(np.asarray(probes, np.float32), reps)])
    planes, alpha, _ = luq_quantize(x, R=4, seed=123, counter=7, n_samples=2)
    assert alpha == 1.0
    avg = (float(alpha) / 2) * luq_smp_sum(planes, x.size)[1:].astype(np.float64).reshape(len(probes), reps)
    for i, p in enumerate(probes):
        lo, hi = _grid_bracket(abs(p), 1.0, 4)
        var1 = (abs(p) - lo) * (hi - abs(p))
        assert abs(avg[i].mean() - p) < 5 * math.sqrt(var1 / 2 / reps) + (hi - lo) * 2.0 ** -16
        assert abs(avg[i].var() / (var1 / 2) - 1) < 0.04


def test_planted_sign_error_is_caught():
    """A sum that drops the sign of the second sample breaks the bracketing pin."""
    x = synth.lognormal_grad((500,), -9.0, 2.0, 0.0, [7, 1])
    planes, alpha, _ = luq_quantize(x, R=4, seed=1, counter=1, n_samples=2)
    p1 = planes[1].copy()
    p1 &= 0x77                                   # clears both sign bits of each byte
    bad = luq_smp_sum(np.stack([planes[0], p1]), x.size).astype(np.int64)
    ok = True
    for i in range(x.size):
        lo, hi = _grid_bracket(abs(float(x[i])), float(alpha), 4)
        if abs(int(bad[i])) not in (2 * lo, lo + hi, 2 * hi):
            ok = False
            break
    assert not ok

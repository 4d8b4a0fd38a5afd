"""Pins of the oracle's single-pass LUQ with the in-hindsight maximum.

Section 4 ("Reducing the data movement") and the hindsight appendix: the
tensor is quantized with alpha from the estimate m carried over from the
previous step, and Eq. hindsight m^t = (1 - eta) max|x^(t-1)| + eta m^(t-1)
gives the next estimate.  Pinned against the exact two-pass oracle (equal
codes when the estimate is the true maximum), the independent rational
restatement of a field, the clipping of magnitudes above the estimated top
level, unbiasedness below it, and the closed form of the update.
"""
from fractions import Fraction

import numpy as np
import pytest

import synth
from oracle.luq import (luq_quantize, luq_quantize_hindsight, luq_field_scalar, unpack_nibbles, luq_decode,
                        hindsight_update, luq_alpha)
from oracle.philox import luq_uniforms


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("R,ns", [(4, 1), (4, 2), (5, 2), (6, 1)])
def test_true_max_estimate_reproduces_exact_luq(dtype, R, ns):
    x = synth.grad_1d(3001, dtype, 0.3, seed=R * 10 + ns)
    c, a, m = luq_quantize(x, dtype=dtype, R=R, seed=77, counter=3, n_samples=ns)
    ch, ah, mh, _ = luq_quantize_hindsight(x, m, dtype=dtype, R=R, seed=77, counter=3, n_samples=ns)
    assert np.array_equal(c, ch)
    assert ah.tobytes() == a.tobytes() and mh.tobytes() == m.tobytes()


@pytest.mark.parametrize("frac", [0.3, 0.6, 1.0, 1.7])
def test_fields_match_rational_restatement(frac):
    """Every element against the exact rational field, including magnitudes
    above the estimated top level (clipped to the top code)."""
    x = synth.grad_1d(600, "f32", 0.2, seed=9)
    m_hat = np.float32(np.abs(x).max() * frac)
    codes, alpha, _, _ = luq_quantize_hindsight(x, m_hat, R=4, seed=5, counter=1)
    nib = unpack_nibbles(codes[0], x.size)
    j = luq_uniforms(x.size, 5, 1, 0)
    for i in range(x.size):
        e = luq_field_scalar(abs(float(x[i])), float(alpha), 4, int(j[i]))
        want = e | (8 if (e and np.signbit(x[i])) else 0)
        assert int(nib[i]) == want, (i, x[i], e)


def test_magnitudes_above_estimate_clip_to_top_with_sign():
    x = np.array([10.0, -10.0, 3.0, -2.5, 1.0, -0.01, 0.0, 100.0], np.float32)
    codes, alpha, maxabs, _ = luq_quantize_hindsight(x, np.float32(2.0), R=4)
    assert alpha == np.float32(0.125) and maxabs == np.float32(100.0)
    nib = unpack_nibbles(codes[0], x.size)
    top = 5
    assert nib[0] == top and nib[1] == top | 8 and nib[2] == top and nib[3] == top | 8 and nib[7] == top
    assert nib[6] == 0 and nib[4] == 4  # 1.0 = alpha 2^3 is on a level and never moves


def test_unbiased_below_the_estimated_top():
    """E[Q(x)] = x (within the stated SR bias bound) for magnitudes below
    alpha 2^R, over 400 counters."""
    x = np.array([0.3, -0.7, 1.1, 1.9, 0.01, -0.049, 0.26], np.float32)
    m_hat = np.float32(2.0)
    alpha = luq_alpha(m_hat, 4)
    acc = np.zeros(x.size)
    for c in range(400):
        codes, a, _, _ = luq_quantize_hindsight(np.tile(x, 64), m_hat, R=4, seed=1, counter=c)
        acc += luq_decode(codes[0], x.size * 64, a).reshape(64, x.size).mean(axis=0)
    mean = acc / 400
    for xi, mi in zip(x.astype(np.float64), mean):
        # bin [l, u): variance (x - l)(u - x) per draw; 25600 draws
        mag = abs(xi)
        levels = [0.0] + [float(alpha) * 2 ** k for k in range(5)]
        lo = max(v for v in levels if v <= mag)
        hi = min(v for v in levels if v > mag)
        sd = np.sqrt((mag - lo) * (hi - mag) / 25600.0)
        assert abs(mi - xi) <= 5 * sd + (hi - lo) * 2.0 ** -16, (xi, mi)


def test_overflow_step_inside_a_sequence_keeps_the_estimate():
    """A run of steps with one overflowed gradient: the estimate after the
    overflow equals the estimate before it, and the following finite steps
    continue Eq. hindsight from there (alpha stays finite)."""
    m = np.float32(1.0)
    seq = []
    for t in range(4):
        x = synth.grad_1d(500, "f32", 0.1, seed=300 + t)
        if t == 2:
            x[17] = np.inf
        _, a, mx, m_next = luq_quantize_hindsight(x, m, R=4, seed=0, counter=t)
        seq.append((a, mx, m, m_next))
        m = m_next
    assert seq[2][3] == seq[2][2] and not np.isfinite(seq[2][1])
    assert np.isfinite(seq[3][0]) and seq[3][0] == luq_alpha(seq[2][2], 4)
    assert seq[3][3] == hindsight_update(seq[3][1], seq[3][2], 0.1)


def test_update_rule_closed_form_and_sequence():
    # eta = 1/2 and powers of two: exact averages
    assert hindsight_update(np.float32(8.0), np.float32(4.0), 0.5) == np.float32(6.0)
    # general eta: the float32 steps written out with exact rationals
    mx, mh, eta = np.float32(3.3), np.float32(2.9), 0.1
    c1 = np.float32(Fraction(1) - Fraction(float(np.float32(eta))))
    want = np.float32(float(np.float32(float(np.float32(Fraction(float(c1)) * Fraction(float(mx)))) +
                                      float(np.float32(Fraction(float(np.float32(eta))) * Fraction(float(mh)))))))
    assert hindsight_update(mx, mh, eta) == want
    # a sequence of steps carries the estimate forward
    m = np.float32(1.0)
    for t in range(5):
        x = synth.grad_1d(999, "f32", 0.1, seed=100 + t)
        _, a, mx, m_next = luq_quantize_hindsight(x, m, R=4, seed=0, counter=t)
        assert a == luq_alpha(m, 4)
        assert mx == np.float32(np.abs(x).max())
        assert m_next == hindsight_update(mx, m, 0.1)
        m = m_next


def test_degenerate_estimates_and_inputs():
    x = synth.grad_1d(64, "f32", 0.0, seed=4)
    for bad in [0.0, -1.0, -0.0]:
        codes, a, _, m_next = luq_quantize_hindsight(x, np.float32(bad), R=4)
        assert a == 0 and not codes.any()
        assert m_next == hindsight_update(np.float32(np.abs(x).max()), np.float32(0.0), 0.1)
    for bad in [np.nan, np.inf]:
        codes, a, _, _ = luq_quantize_hindsight(x, np.float32(bad), R=4)
        assert np.isnan(a) and not codes.any()
    y = x.copy()
    y[7] = np.nan
    y[9] = -np.inf
    codes, a, mx, m_next = luq_quantize_hindsight(y, np.float32(1.0), R=4)
    nib = unpack_nibbles(codes[0], y.size)
    assert nib[7] & 7 == 5 and nib[9] == 5 | 8
    # an overflowed step is not averaged into the estimate: it stays as it was
    assert np.isnan(mx) and m_next == np.float32(1.0)
    y[7] = 0.0
    codes, a, mx, m_next = luq_quantize_hindsight(y, np.float32(0.5), R=4)
    assert mx == np.float32(np.inf) and m_next == np.float32(0.5)
    # a stored estimate that reads as 0 is kept as stored
    _, _, _, m_next = luq_quantize_hindsight(y, np.float32(-3.0), R=4)
    assert m_next == np.float32(-3.0)
    codes, a, mx, m_next = luq_quantize_hindsight(np.zeros(0, np.float32), np.float32(2.0), R=4)
    assert mx == 0 and m_next == hindsight_update(np.float32(0.0), np.float32(2.0), 0.1)

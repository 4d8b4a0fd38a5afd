"""Pins for the LUQ oracle (CPU): closed forms, invariants, brute force.

Each test checks the oracle against something other than itself: the
underflow threshold of Eq. alpha, the SR mean and variance of Eq. SR_eq /
Table 1, exhaustive enumeration of the 2^16 uniforms, bin bracketing computed
independently with math.frexp, power-of-two scale equivariance, the 1/N
variance of SMP (Section 5.1) and the unbiased weight gradient of Eq. update.
"""
import math

import numpy as np
import pytest

import synth
from oracle import luq
from oracle.luq import (luq_quantize, luq_decode, luq_decode_int, luq_fields, luq_field_scalar, unpack_nibbles,
                        luq_nibbles_at)
from oracle.int4 import int4_quantize, int4_decode
from oracle.gemm import gemm_wgrad_ref


def _bracket(x, alpha, R):
    """Independent bin finder: (lower, upper) grid points around |x| via frexp."""
    a = abs(float(x))
    if a == 0:
        return 0.0, 0.0
    if a < alpha:
        return 0.0, float(alpha)
    if a >= alpha * 2 ** R:
        return alpha * 2 ** R, alpha * 2 ** R
    m, e = math.frexp(a / alpha)          # a/alpha = m * 2^e, m in [0.5, 1)
    k = e - 1
    # guard against rounding of a/alpha right at a level
    while alpha * 2 ** k > a:
        k -= 1
    while alpha * 2 ** (k + 1) <= a:
        k += 1
    return alpha * 2 ** k, alpha * 2 ** (k + 1)


@pytest.mark.parametrize("R", [4, 5, 6])
def test_alpha_is_max_over_2_pow_R(R):
    g = synth.grad_1d(10001, zero_frac=0.3, seed=11)
    _, alpha, m = luq_quantize(g, R=R, seed=1)
    assert m == np.float32(np.abs(g).max())
    assert float(alpha) * 2 ** R == float(m)          # Eq. alpha, exact for normal m
    assert float(alpha) == float(m) / 2 ** R


@pytest.mark.parametrize("R", [4, 6])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_code_set_sign_and_bracketing(R, dtype):
    g = synth.grad_1d(20000, dtype=dtype, zero_frac=0.25, seed=12, sigma=2.0)
    xf = synth.bf16_bits_to_f32(g) if dtype == "bf16" else g
    codes, alpha, m = luq_quantize(g, dtype=dtype, R=R, seed=3, counter=5)
    v = luq_decode(codes[0], g.size, alpha)
    allowed = {0.0} | {float(alpha) * 2 ** k for k in range(R + 1)}
    assert set(np.unique(np.abs(v)).tolist()) <= allowed
    nz = v != 0
    assert np.all(np.sign(v[nz]) == np.sign(xf[nz]))
    for x, q in zip(xf[:4000], v[:4000]):
        lo, hi = _bracket(x, float(alpha), R)
        assert abs(q) in (lo, hi), (x, q, lo, hi)
    # no negative zero nibble: field 0 always has the sign bit clear
    nib = unpack_nibbles(codes[0], g.size)
    assert not np.any(nib == 8)


def test_max_element_gets_top_code_and_zero_gets_zero():
    g = synth.grad_1d(999, zero_frac=0.5, seed=13)
    g[5] = -np.abs(g).max() * 1.5
    g[6] = -0.0
    codes, alpha, m = luq_quantize(g, R=4, seed=9)
    nib = unpack_nibbles(codes[0], g.size)
    assert nib[5] == (8 | 5)                          # sign | field R+1
    assert nib[6] == 0
    assert np.all(nib[g == 0] == 0)
    assert luq_decode(codes[0], g.size, alpha)[5] == -float(m)
    # odd length: the last byte's high nibble is 0
    assert codes.shape[1] == 500 and (codes[0, -1] >> 4) == 0


def test_values_on_levels_never_move():
    alpha = 1.0
    x = np.array([16.0] + [2.0 ** k for k in range(5)] * 50 + [-4.0] * 50, dtype=np.float32)
    for c in range(5):
        codes, a, _ = luq_quantize(x, R=4, seed=c, counter=c)
        assert a == alpha
        assert np.array_equal(luq_decode(codes[0], x.size, a), x.astype(np.float64))


def _probe_tensor(probes, reps, top=16.0):
    x = np.concatenate([np.array([top], np.float32), np.repeat(np.asarray(probes, np.float32), reps)])
    return x


PROBES = [1e-4, 0.0625, 0.3, 0.5, 0.77, float(np.nextafter(np.float32(1), np.float32(0))),
          1.0, float(np.nextafter(np.float32(1), np.float32(2))), 1.25, 1.5, 1.999, 2.5, 3.0, 3.75,
          5.0, 6.0, 7.3, 8.0, 9.0, 11.0, 12.0, 15.0, float(np.nextafter(np.float32(16), np.float32(0))),
          -0.3, -1.5, -6.0, -13.0, 0.01, 0.99, 4.0001, 2.0e-3, 14.5]


def test_unbiased_over_a_million_draws_and_sr_variance():
    """E[Q(x)] = x (Eq. expecration_SR) and Var = (x-l)(u-x) (Table 1)."""
    reps = 1 << 20
    x = _probe_tensor(PROBES, reps)
    codes, alpha, m = luq_quantize(x, R=4, seed=2024, counter=1)
    assert alpha == 1.0
    v = luq_decode(codes[0], x.size, alpha)[1:].reshape(len(PROBES), reps)
    for i, p in enumerate(PROBES):
        lo, hi = _bracket(p, 1.0, 4)
        w = hi - lo
        var = (abs(p) - lo) * (hi - abs(p))
        mean = v[i].mean()
        # the draws are Bernoulli with the exact achieved probability
        # ceil(2^16 d / w) / 2^16, which differs from d / w by < 2^-16
        p_eff = math.ceil((abs(p) - lo) / w * 2 ** 16) / 2 ** 16 if w > 0 else 0.0
        sd = w * math.sqrt(p_eff * (1 - p_eff) / reps)
        bias_bound = w * 2.0 ** -16
        dev = (mean - p) * (1 if p >= 0 else -1)        # bias is toward larger magnitude
        assert -5 * sd - 1e-12 <= dev <= 5 * sd + bias_bound + 1e-12, (p, mean)
        if w > 0:
            pp = (abs(p) - lo) / w
            if 0.01 <= pp <= 0.99:
                emp = v[i].var()
                rel_se = abs(1 - 2 * pp) / math.sqrt(reps * pp * (1 - pp)) + 2.0 ** -16 / pp
                assert abs(emp / var - 1) <= 5 * rel_se + 2e-3, (p, emp, var)


@pytest.mark.parametrize("a,alpha,R", [
    (0.3, 1.0, 4), (1.7, 1.0, 4), (5.2, 1.0, 4), (1e-3, 1.0, 4), (15.99, 1.0, 4),
    (3.1e-40, 2.2e-39, 4),          # subnormal magnitude, subnormal alpha
    (7.0e-39, 1.5e-39, 4),          # subnormal alpha, a few binades up
    (2.9e37, 3.1e36, 4),            # near the top of the float32 range
    (0.33, 0.125, 6), (63.0, 1.0, 6),
])
def test_bruteforce_all_uniforms(a, alpha, R):
    """Exhaustive over j in [0, 2^16): exact P(up) and one-sided bias < w 2^-16."""
    a32 = float(np.float32(a))
    al = float(np.float32(alpha))
    j = np.arange(1 << 16)
    e = luq_fields(np.full(j.size, a32), np.float32(al), R, j)
    lo, hi = _bracket(a32, al, R)
    w = hi - lo
    vals = np.where(e == 0, 0.0, al * 2.0 ** (e.astype(np.float64) - 1))
    assert set(np.unique(vals).tolist()) <= {lo, hi}
    ups = int((vals == hi).sum()) if w > 0 else 0
    if w > 0:
        from fractions import Fraction
        exact = Fraction(a32) - Fraction(lo)
        need = math.ceil(exact * (1 << 16) / Fraction(w))
        assert ups == need
        bias = Fraction(lo) + Fraction(w) * Fraction(ups, 1 << 16) - Fraction(a32)
        assert 0 <= bias < Fraction(w) / (1 << 16)
    # rational-arithmetic restatement agrees on a spread of j
    for jj in list(range(0, 1 << 16, 997)) + [0, 1, (1 << 16) - 1]:
        assert luq_field_scalar(a32, al, R, jj) == int(e[jj])


def test_scale_equivariance_by_powers_of_two():
    g = synth.grad_1d(5000, zero_frac=0.2, seed=21)
    c0, a0, m0 = luq_quantize(g, R=4, seed=5, counter=2)
    for s in (-20, -3, 7, 30):
        c1, a1, m1 = luq_quantize((g * np.float32(2.0 ** s)).astype(np.float32), R=4, seed=5, counter=2)
        assert np.array_equal(c0, c1)
        assert float(a1) == float(a0) * 2.0 ** s


def test_bf16_path_equals_f32_path():
    g = synth.grad_1d(3001, dtype="bf16", seed=22)
    cb, ab, mb = luq_quantize(g, dtype="bf16", R=4, seed=1, counter=1)
    cf, af, mf = luq_quantize(synth.bf16_bits_to_f32(g), dtype="f32", R=4, seed=1, counter=1)
    assert np.array_equal(cb, cf) and ab == af and mb == mf


def test_degenerate_inputs():
    z = np.zeros(17, np.float32)
    c, a, m = luq_quantize(z)
    assert a == 0 and m == 0 and not c.any()
    c, a, m = luq_quantize(np.zeros(0, np.float32))
    assert c.shape == (1, 0)
    x = synth.grad_1d(100, seed=3)
    x[50] = np.inf
    c, a, m = luq_quantize(x)
    assert np.isnan(a) and np.isinf(m) and not c.any()
    x[51] = np.nan
    c, a, m = luq_quantize(x)
    assert np.isnan(a) and np.isnan(m)
    # max so small that max / 2^R underflows to zero in float32
    tiny = np.array([1e-45, -1e-45, 0.0], np.float32)
    c, a, m = luq_quantize(tiny, R=4)
    assert m > 0 and a == 0 and not c.any()


def test_smp_variance_halves():
    """Section 5.1: averaging N independent samples divides the variance by N."""
    reps = 1 << 19
    probes = [0.3, 1.5, 3.0, 6.5, 11.0]
    x = _probe_tensor(probes, reps)
    codes, alpha, _ = luq_quantize(x, R=4, seed=77, counter=3, n_samples=2)
    v0 = luq_decode(codes[0], x.size, alpha)[1:].reshape(len(probes), reps)
    v1 = luq_decode(codes[1], x.size, alpha)[1:].reshape(len(probes), reps)
    avg = 0.5 * (v0 + v1)
    for i, p in enumerate(probes):
        lo, hi = _bracket(p, 1.0, 4)
        var1 = (p - lo) * (hi - p)
        assert abs(avg[i].var() / (var1 / 2) - 1) < 0.03
        assert abs(np.corrcoef(v0[i], v1[i])[0, 1]) < 0.01
        assert abs(avg[i].mean() - p) < 5 * math.sqrt(var1 / 2 / reps) + (hi - lo) * 2.0 ** -16


def test_unbiased_weight_gradient():
    """Eq. update: E[Q(delta)^T Q(a)] equals delta^T Q(a), over 300 counters."""
    T, Nout, Kin = 64, 32, 16
    d = synth.small(seed=31)
    g = np.ascontiguousarray(d["g"][:T, :Nout])
    a = np.ascontiguousarray(d["a"][:T, :Kin])
    ca, sa = int4_quantize(a, is_signed=False)
    aq = int4_decode(ca, a.size, sa, False).reshape(T, Kin)
    exact = g.astype(np.float64).T @ aq
    draws = []
    for c in range(300):
        codes, alpha, _ = luq_quantize(g, R=4, seed=99, counter=c)
        ref, _ = gemm_wgrad_ref(codes, alpha, ca, sa, False, T, Nout, Kin)
        draws.append(ref)
    draws = np.array(draws)
    mean = draws.mean(0)
    se = draws.std(0, ddof=1) / math.sqrt(len(draws))
    _, alpha, _ = luq_quantize(g, R=4)
    bias_bound = (np.abs(aq).sum(0)[None, :] * float(alpha) * 2 ** 3 * 2.0 ** -16)
    assert np.all(np.abs(mean - exact) <= 5 * se + bias_bound + 1e-18)


def test_index_addressed_codes_equal_whole_tensor_codes():
    """Codes computed one by one from flat indices equal those of the whole
    tensor (unsorted, repeated and tail indices; both SMP samples)."""
    x = synth.lognormal_grad((5001,), -10.0, 2.0, 0.3, [77, 1])
    codes, alpha, _ = luq_quantize(x, R=4, seed=99, counter=4, n_samples=2)
    idx = np.array([5000, 0, 7, 8, 4999, 7, 1234, 2500, 3], dtype=np.int64)
    for s in range(2):
        whole = unpack_nibbles(codes[s], x.size)
        got = luq_nibbles_at(x[idx], idx, alpha, 4, 99, 4, s)
        assert np.array_equal(got, whole[idx])

"""Planted mistakes in the oracle must be caught by its pins (CPU only).

Each mutant replaces one piece of the oracle with a plausible mistake (a
dropped term, a reversed comparison, a wrong threshold, a lost sign, a
transposed operand, a missing Philox round) and the test asserts that at
least one of the pin checks used by the other oracle tests rejects it, while
the unmodified oracle passes all of them.
"""
import math

import numpy as np
import pytest

import oracle.luq as L
import oracle.philox as P
import synth
from oracle.gemm import gemm_dgrad_ref
from oracle.int4 import int4_quantize

TWO16 = 65536
PROBES = [0.02, 0.3, 0.77, 1.2, 1.5, 2.9, 3.3, 5.0, 6.5, 11.0, 13.7, -2.2, -0.4]


def _bracket(a, alpha, R):
    a = abs(a)
    if a < alpha:
        return 0.0, alpha
    k = int(math.floor(math.log2(a / alpha)))
    return alpha * 2 ** k, alpha * 2 ** (k + 1)


def pins_pass():
    """Runs the pin checks against the current oracle; returns a list of failures."""
    fails = []
    reps = 1 << 16
    x = np.concatenate([np.array([16.0], np.float32), np.repeat(np.array(PROBES, np.float32), reps)])
    codes, alpha, m = L.luq_quantize(x, R=4, seed=11, counter=3)
    if float(alpha) != 1.0:
        fails.append("alpha")
    v = L.luq_decode(codes[0], x.size, alpha)
    nib = L.unpack_nibbles(codes[0], x.size)
    if (nib[0] & 7) != 5:
        fails.append("top")
    vv = v[1:].reshape(len(PROBES), reps)
    for i, p in enumerate(PROBES):
        lo, hi = _bracket(p, 1.0, 4)
        if not set(np.unique(np.abs(vv[i])).tolist()) <= {lo, hi}:
            fails.append("bracket")
        if np.any(np.sign(vv[i][vv[i] != 0]) != np.sign(p)):
            fails.append("sign")
        w = hi - lo
        sd = w * 0.5 / math.sqrt(reps)
        if abs(vv[i].mean() - p) > 6 * sd + w * 2.0 ** -16:
            fails.append("unbiased")
    return sorted(set(fails))


def test_unmodified_oracle_passes():
    assert pins_pass() == []


def _rdn_fields(a, alpha, R, j):
    a = np.asarray(a, np.float64)
    Lv = L.luq_levels(alpha, R)
    n = np.zeros(a.shape, np.int64)
    for k in range(1, R):
        n += a >= Lv[k]
    under = a < Lv[0]
    lo = np.where(under, 0.0, Lv[n])
    hi = np.where(under, Lv[0], 2 * Lv[n])
    e = np.where(under, 0, n + 1) + ((a - lo) > (hi - a))
    return np.where(a >= Lv[R], R + 1, e).astype(np.uint8)


def _no_underflow_fields(a, alpha, R, j):
    e = ORIG_FIELDS(a, alpha, R, j)
    return np.where(np.asarray(a) < float(alpha), 0, e).astype(np.uint8)


def _double_width_fields(a, alpha, R, j):
    # rounding probability doubled (bin width taken as half the lower level)
    return ORIG_FIELDS(a, alpha, R, np.asarray(j, np.float64) * 2)


ORIG_FIELDS = L.luq_fields


@pytest.mark.parametrize("mutant", [_rdn_fields, _no_underflow_fields, _double_width_fields])
def test_field_mutants_are_caught(monkeypatch, mutant):
    monkeypatch.setattr(L, "luq_fields", mutant)
    assert pins_pass() != []


def test_reversed_comparison_is_caught(monkeypatch):
    def rev(a, alpha, R, j):
        a = np.asarray(a, np.float64)
        Lv = L.luq_levels(alpha, R)
        n = np.zeros(a.shape, np.int64)
        for k in range(1, R):
            n += a >= Lv[k]
        under = a < Lv[0]
        lo = np.where(under, 0.0, Lv[n])
        w = np.where(under, Lv[0], Lv[n])
        up = np.asarray(j, np.float64) * w > (a - lo) * TWO16
        e = np.where(under, 0, n + 1) + up
        return np.where(a >= Lv[R], R + 1, e).astype(np.uint8)
    monkeypatch.setattr(L, "luq_fields", rev)
    assert "unbiased" in pins_pass()


def test_wrong_threshold_is_caught(monkeypatch):
    monkeypatch.setattr(L, "luq_alpha", lambda m, R: np.float32(float(m) * 2.0 ** (-(R + 1))))
    f = pins_pass()
    assert "alpha" in f or "top" in f


def test_lost_sign_is_caught(monkeypatch):
    orig = L.pack_nibbles
    monkeypatch.setattr(L, "pack_nibbles", lambda nib: orig(np.asarray(nib) & 7))
    assert "sign" in pins_pass()


def test_missing_philox_round_is_caught(monkeypatch):
    monkeypatch.setattr(P, "ROUNDS", 9)
    got = P.philox4x32_10(np.zeros(4, np.uint32), (0, 0))
    assert [int(v) for v in got] != [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]


def test_transposed_operand_is_caught():
    """A GEMM that reads W transposed differs from the triple-loop pin."""
    M, N, K = 4, 6, 6
    g = synth.lognormal_grad((M, K), -3, 2, 0.2, [50, 1])
    w = synth.normal((K, N), 1.0, [50, 2])
    planes, alpha, _ = L.luq_quantize(g, R=4, seed=1)
    wc, ws = int4_quantize(w, is_signed=True)
    wt, _ = int4_quantize(np.ascontiguousarray(w.T), is_signed=True)
    good, _ = gemm_dgrad_ref(planes, alpha, wc, ws, True, M, N, K)
    bad, _ = gemm_dgrad_ref(planes, alpha, wt, ws, True, M, N, K)
    assert not np.allclose(good, bad)


def _fwd_pin_fails():
    """The forward pins (rounding bound against the float product, and the
    closed form 49 K s_x s_W) against the current oracle.gemm."""
    import oracle.gemm as G
    fails = []
    M, N, K = 12, 10, 64
    x = synth.normal((M, K), 1.0, [51, 1])
    w = synth.normal((N, K), 0.1, [51, 2])
    xc, xs = int4_quantize(x, is_signed=True)
    wc, ws = int4_quantize(w, is_signed=True)
    ref, _ = G.gemm_fwd_ref(xc, xs, True, wc, ws, True, M, N, K)
    exact = x.astype(np.float64) @ w.astype(np.float64).T
    dx, dw = float(xs) / 2 * (1 + 1e-6), float(ws) / 2 * (1 + 1e-6)
    bound = np.abs(x) @ np.full((K, N), dw) + np.full((M, K), dx) @ np.abs(w).T.astype(np.float64) + K * dx * dw
    if not np.all(np.abs(ref - exact) <= bound):
        fails.append("bound")
    x7 = np.full(K // 2, 0x77, np.uint8)
    r7, _ = G.gemm_fwd_ref(x7, np.float32(0.5), True, x7, np.float32(0.25), True, 1, 1, K)
    if r7[0, 0] != 49 * K * 0.125:
        fails.append("closed")
    # triple loop over nibbles read from the bytes directly
    m, n, k = 3, 4, 6
    xb, wb = xc[: m * k // 2], wc[: n * k // 2]
    nib = lambda c, i: (int(c[i // 2]) >> (4 * (i & 1))) & 15
    val = lambda v: v - 16 if v >= 8 else v
    loop = [[sum(val(nib(xb, a * k + t)) * val(nib(wb, b * k + t)) for t in range(k)) * float(xs) * float(ws)
             for b in range(n)] for a in range(m)]
    small, _ = G.gemm_fwd_ref(xb, xs, True, wb, ws, True, m, n, k)
    if not np.array_equal(small, np.array(loop)):
        fails.append("loop")
    return fails


def test_fwd_mutants_are_caught(monkeypatch):
    import oracle.gemm as G
    assert _fwd_pin_fails() == []
    good_rows = G._rows_int4
    # lost sign extension: signed codes decoded as unsigned
    monkeypatch.setattr(G, "_rows_int4", lambda c, r, n, signed: good_rows(c, r, n, False))
    assert _fwd_pin_fails()
    monkeypatch.setattr(G, "_rows_int4", good_rows)
    # reduction index reversed on one operand
    good_mm = G._matmul_exact
    monkeypatch.setattr(G, "_matmul_exact", lambda A, B: good_mm(A, B[::-1]))
    assert "loop" in _fwd_pin_fails()
    monkeypatch.setattr(G, "_matmul_exact", good_mm)
    # the weight scale dropped
    good_ref = G.gemm_fwd_ref
    monkeypatch.setattr(G, "gemm_fwd_ref", lambda xc, xs, xsig, wc, ws, *a, **k: good_ref(xc, xs, xsig, wc, 1.0, *a, **k))
    assert "closed" in _fwd_pin_fails()


def test_pw2_floor_instead_of_ceil_is_caught(monkeypatch):
    """alpha_PW2 with floor(log2 max) clips the maximum: the pin that the top
    level is at or above max|x| rejects it, the real oracle passes it."""
    from fractions import Fraction
    import math

    def top_at_or_above_max():
        for m in [3.0, 1.5, 17.0, 1e-3, 123.456]:
            x = np.array([m, -m / 3, m / 7], np.float32)
            _, a, mx = L.luq_quantize(x, R=4, pw2=True)
            if not Fraction(float(a)) * 16 >= Fraction(float(mx)):
                return False
        return True

    assert top_at_or_above_max()

    def floor_alpha(maxabs, R):
        return np.float32(2.0 ** (math.floor(math.log2(float(maxabs))) - R))

    monkeypatch.setattr(L, "luq_alpha_pw2", floor_alpha)
    assert not top_at_or_above_max()


def test_conv_dgrad_tap_mistakes_are_caught(monkeypatch):
    """A gradient that reads the tap offsets with the wrong sign, or drops a
    border tap, fails the adjoint pin against scipy's correlation."""
    from scipy.signal import correlate2d
    import oracle.conv as CV
    from oracle.luq import luq_decode_int
    from oracle.int4 import int4_decode_int
    B, H, W, C, Cout = 1, 5, 6, 2, 3
    g = synth.lognormal_grad((B * H * W, Cout), -4.0, 2.0, 0.3, [70, 1])
    w = synth.normal((Cout, 9 * C), 1.0, [70, 2])
    planes, alpha, _ = L.luq_quantize(g, R=4, seed=1)
    wc, ws = int4_quantize(w, is_signed=True)

    def adjoint_holds():
        G = luq_decode_int(planes[0], B * H * W * Cout).reshape(B, H, W, Cout).astype(np.float64)
        Wq = int4_decode_int(wc, Cout * 9 * C, True).reshape(Cout, 3, 3, C).astype(np.float64)
        act = np.random.default_rng(3).integers(-7, 8, size=(B, H, W, C)).astype(np.float64)
        z = np.zeros((B, H, W, Cout))
        for o in range(Cout):
            for c in range(C):
                z[0, :, :, o] += correlate2d(act[0, :, :, c], Wq[o, :, :, c], mode="same")
        dact, _ = CV.conv3x3_dgrad_ref(planes, np.float32(1), wc, np.float32(1), True, B, H, W, C, Cout)
        return np.sum(z * G) == np.sum(act.reshape(-1, C) * dact)

    assert adjoint_holds()
    good = CV.conv3x3_dgrad_ref
    src = open(CV.__file__).read()
    bad_src = src.replace("ys, xs = y - kh + 1, x - kw + 1", "ys, xs = y + kh - 1, x + kw - 1")
    assert bad_src != src
    ns = {}
    exec(compile(bad_src, CV.__file__, "exec"), CV.__dict__ | ns, ns)
    monkeypatch.setattr(CV, "conv3x3_dgrad_ref", ns["conv3x3_dgrad_ref"])
    assert not adjoint_holds()
    monkeypatch.setattr(CV, "conv3x3_dgrad_ref", good)

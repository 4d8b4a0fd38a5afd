"""Pins for the GEMM oracle (CPU).

The backward / update products are pinned by a pure-Python triple loop over
codes decoded from the bit layout directly (not through the oracle's
decoders), by the MF-BPROP worked example of Appendix A.8.1 (FP4 field 011
times INT4 3 is 12), and by the linearity of SMP averaging (Section 5.1).
The forward product (Eq. forward, Appendix A.1) is pinned by the same kind
of triple loop, by closed forms on constant codes, and by the round-to-
nearest error bound: |Q(x)_k - x_k| <= s_x / 2 and |Q(w)_k - w_k| <= s_W / 2
bound |y - x W^T| per output.
"""
import numpy as np
import pytest

import synth
from oracle.luq import luq_quantize
from oracle.int4 import int4_quantize
from oracle.gemm import gemm_dgrad_ref, gemm_wgrad_ref, gemm_fwd_ref


def _nib(codes, i):
    b = int(codes[i // 2])
    return (b >> 4) if (i & 1) else (b & 0xF)


def _luq_val(n):
    e, neg = n & 7, n >> 3
    if e == 0:
        return 0
    return -(2 ** (e - 1)) if neg else 2 ** (e - 1)


def _int4_val(n, signed):
    return n - 16 if (signed and n >= 8) else n


def _loop_dgrad(planes, alpha, wc, ws, wsig, M, N, K):
    out = [[0.0] * N for _ in range(M)]
    for m in range(M):
        for n in range(N):
            acc = 0
            for k in range(K):
                a = sum(_luq_val(_nib(p, m * K + k)) for p in planes)
                acc += a * _int4_val(_nib(wc, k * N + n), wsig)
            out[m][n] = acc * float(alpha) / len(planes) * float(ws)
    return np.array(out)


def _loop_wgrad(planes, alpha, ac, as_, asig, T, No, Ki):
    out = np.zeros((No, Ki))
    for o in range(No):
        for i in range(Ki):
            acc = 0
            for t in range(T):
                g = sum(_luq_val(_nib(p, t * No + o)) for p in planes)
                acc += g * _int4_val(_nib(ac, t * Ki + i), asig)
            out[o, i] = acc * float(alpha) / len(planes) * float(as_)
    return out


@pytest.mark.parametrize("n_samples", [1, 2])
@pytest.mark.parametrize("signed", [True, False])
def test_dgrad_matches_triple_loop(n_samples, signed):
    M, N, K = 5, 6, 8
    g = synth.lognormal_grad((M, K), -3, 2, 0.3, [40, 1])
    w = synth.normal((K, N), 1.0, [40, 2])
    planes, alpha, _ = luq_quantize(g, R=4, seed=3, counter=1, n_samples=n_samples)
    wc, ws = int4_quantize(w if signed else np.abs(w), is_signed=signed)
    ref, absref = gemm_dgrad_ref(planes, alpha, wc, ws, signed, M, N, K)
    assert np.array_equal(ref, _loop_dgrad(list(planes), alpha, wc, ws, signed, M, N, K))
    assert np.all(absref >= np.abs(ref))


@pytest.mark.parametrize("n_samples", [1, 2])
def test_wgrad_matches_triple_loop(n_samples):
    T, No, Ki = 7, 4, 6
    g = synth.lognormal_grad((T, No), -3, 2, 0.3, [41, 1])
    a = synth.half_normal((T, Ki), [41, 2])
    planes, alpha, _ = luq_quantize(g, R=4, seed=4, counter=2, n_samples=n_samples)
    ac, as_ = int4_quantize(a, is_signed=False)
    ref, _ = gemm_wgrad_ref(planes, alpha, ac, as_, False, T, No, Ki)
    assert np.array_equal(ref, _loop_wgrad(list(planes), alpha, ac, as_, False, T, No, Ki))
    # row subset and reduction slices compose
    r1, _ = gemm_wgrad_ref(planes, alpha, ac, as_, False, T, No, Ki, rows=[1, 3], t_range=(0, 3))
    r2, _ = gemm_wgrad_ref(planes, alpha, ac, as_, False, T, No, Ki, rows=[1, 3], t_range=(3, T))
    assert np.allclose(r1 + r2, ref[[1, 3]], rtol=0, atol=1e-300)


def test_mf_bprop_worked_example():
    """Appendix A.8.1: FP4 [1,3,0] bits 011 (= 4) times INT4 3 gives 12."""
    g_codes = np.array([[0b0011 | (0 << 4)]], np.uint8)      # G = [[4, 0]] with alpha = 1
    w_codes = np.array([0x3, 0x0], np.uint8)                   # W = [[3, 0], [0, 0]]
    ref, _ = gemm_dgrad_ref(g_codes, np.float32(1), w_codes, np.float32(1), True, 1, 2, 2)
    assert ref[0, 0] == 12.0 and ref[0, 1] == 0.0
    # negative gradient sign: the product sign is the XOR of the signs
    g_neg = np.array([[0b1011]], np.uint8)
    ref, _ = gemm_dgrad_ref(g_neg, np.float32(1), w_codes, np.float32(1), True, 1, 2, 2)
    assert ref[0, 0] == -12.0


def test_smp_gemm_is_mean_of_single_plane_gemms():
    M, N, K = 16, 12, 20
    g = synth.lognormal_grad((M, K), -5, 2, 0.2, [42, 1])
    w = synth.normal((K, N), 1.0, [42, 2])
    planes, alpha, _ = luq_quantize(g, R=4, seed=8, counter=0, n_samples=2)
    wc, ws = int4_quantize(w, is_signed=True)
    both, _ = gemm_dgrad_ref(planes, alpha, wc, ws, True, M, N, K)
    p0, _ = gemm_dgrad_ref(planes[0], alpha, wc, ws, True, M, N, K)
    p1, _ = gemm_dgrad_ref(planes[1], alpha, wc, ws, True, M, N, K)
    assert np.allclose(both, 0.5 * (p0 + p1), rtol=1e-15, atol=0)


def _loop_fwd(xc, xs, xsig, wc, ws, wsig, M, N, K):
    out = np.zeros((M, N))
    for m in range(M):
        for n in range(N):
            acc = 0
            for k in range(K):
                acc += _int4_val(_nib(xc, m * K + k), xsig) * _int4_val(_nib(wc, n * K + k), wsig)
            out[m, n] = acc * float(xs) * float(ws)
    return out


@pytest.mark.parametrize("xsig,wsig", [(True, True), (False, True), (True, False), (False, False)])
def test_fwd_matches_triple_loop(xsig, wsig):
    M, N, K = 5, 7, 10
    x = synth.normal((M, K), 1.0, [43, 1])
    w = synth.normal((N, K), 0.5, [43, 2])
    xc, xs = int4_quantize(x if xsig else np.abs(x), is_signed=xsig)
    wc, ws = int4_quantize(w if wsig else np.abs(w), is_signed=wsig)
    ref, absref = gemm_fwd_ref(xc, xs, xsig, wc, ws, wsig, M, N, K)
    assert np.array_equal(ref, _loop_fwd(xc, xs, xsig, wc, ws, wsig, M, N, K))
    assert np.all(absref >= np.abs(ref))
    sub, _ = gemm_fwd_ref(xc, xs, xsig, wc, ws, wsig, M, N, K, rows=[4, 0])
    assert np.array_equal(sub, ref[[4, 0]])


def test_fwd_closed_forms():
    K = 6
    # every code 7 (signed) / 15 (unsigned): y = 49 K s_x s_W and 105 K s_x s_W
    x7 = np.full((2 * K + 1) // 2, 0x77, np.uint8)
    ref, _ = gemm_fwd_ref(x7, np.float32(0.5), True, x7, np.float32(0.25), True, 1, 1, K)
    assert ref[0, 0] == 49 * K * 0.125
    xf = np.full(K // 2, 0xFF, np.uint8)
    ref, _ = gemm_fwd_ref(xf, np.float32(1), False, x7, np.float32(1), True, 1, 1, K)
    assert ref[0, 0] == 105 * K
    # the signed code 0xF is -1, unsigned 15
    ref, _ = gemm_fwd_ref(xf, np.float32(1), True, x7, np.float32(1), True, 1, 1, K)
    assert ref[0, 0] == -7 * K
    # a ReLU-like row against alternating +-7 weights cancels pairwise
    alt = np.full(K // 2, 0x97, np.uint8)   # codes 7, -7, 7, -7, ...
    ref, _ = gemm_fwd_ref(xf, np.float32(1), False, alt, np.float32(1), True, 1, 1, K)
    assert ref[0, 0] == 0


@pytest.mark.parametrize("xsig", [True, False])
def test_fwd_within_rounding_error_of_the_float_product(xsig):
    M, N, K = 24, 16, 96
    x = synth.normal((M, K), 1.0, [44, 1])
    if not xsig:
        x = np.maximum(x, 0)
    w = synth.normal((N, K), 0.05, [44, 2])
    xc, xs = int4_quantize(x, is_signed=xsig)
    wc, ws = int4_quantize(w, is_signed=True)
    ref, _ = gemm_fwd_ref(xc, xs, xsig, wc, ws, True, M, N, K)
    exact = x.astype(np.float64) @ w.astype(np.float64).T
    dx, dw = float(xs) / 2 * (1 + 1e-6), float(ws) / 2 * (1 + 1e-6)
    bound = (np.abs(x) @ np.full((K, N), dw) + np.full((M, K), dx) @ np.abs(w).T.astype(np.float64)
             + K * dx * dw)
    assert np.all(np.abs(ref - exact) <= bound)
    # and the bound is not vacuous: the product is far from zero on average
    assert np.mean(np.abs(ref - exact)) < 0.25 * np.mean(np.abs(exact))

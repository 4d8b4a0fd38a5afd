"""Pins for the convolution gradient oracles (CPU): activation gradient,
weight gradient and the lowering (im2col) of the activations.

Pinned by pure-Python loops over the definitions of the gradients of a 3x3,
stride 1, zero-padded convolution with codes decoded from the bits directly;
by the adjoint identities <conv(a), g> = <a, dact> and <dW, K> = <g, conv(a;
K)> with the forward convolution computed by scipy's 2-D correlation (an
independent library routine); by the equality of the per-tap sums with the
lowered GEMMs (Eqs. backward and update); and the lowering by a direct
gather with explicit bounds checks.
"""
import numpy as np
import pytest
from scipy.signal import correlate2d

import synth
from oracle.luq import luq_quantize, luq_decode_int
from oracle.int4 import int4_quantize, int4_decode_int
from oracle.gemm import gemm_dgrad_ref
from oracle.conv import conv3x3_dgrad_ref


def _nib(codes, i):
    b = int(codes[i // 2])
    return (b >> 4) if (i & 1) else (b & 0xF)


def _luq_val(n):
    e, neg = n & 7, n >> 3
    return 0 if e == 0 else (-(2 ** (e - 1)) if neg else 2 ** (e - 1))


def _int4_val(n, signed):
    return n - 16 if (signed and n >= 8) else n


def _case(B, H, W, C, Cout, ns, seed, wsig=True):
    g = synth.lognormal_grad((B * H * W, Cout), -4.0, 2.0, 0.3, [seed, 1])
    w = synth.normal((Cout, 9 * C), 1.0, [seed, 2])
    planes, alpha, _ = luq_quantize(g, R=4, seed=seed, counter=2, n_samples=ns)
    wc, ws = int4_quantize(w if wsig else np.abs(w), is_signed=wsig)
    return planes, alpha, wc, ws


@pytest.mark.parametrize("ns", [1, 2])
def test_matches_loop_over_the_definition(ns):
    B, H, W, C, Cout = 2, 3, 4, 2, 3
    planes, alpha, wc, ws = _case(B, H, W, C, Cout, ns, seed=60)
    ref, absref = conv3x3_dgrad_ref(planes, alpha, wc, ws, True, B, H, W, C, Cout)
    want = np.zeros((B * H * W, C))
    for b in range(B):
        for y in range(H):
            for x in range(W):
                for c in range(C):
                    acc = 0
                    for kh in range(3):
                        for kw in range(3):
                            yo, xo = y - kh + 1, x - kw + 1
                            if not (0 <= yo < H and 0 <= xo < W):
                                continue
                            t = (b * H + yo) * W + xo
                            for o in range(Cout):
                                gv = sum(_luq_val(_nib(p, t * Cout + o)) for p in planes)
                                wv = _int4_val(_nib(wc, o * 9 * C + (kh * 3 + kw) * C + c), True)
                                acc += gv * wv
                    want[(b * H + y) * W + x, c] = acc * float(alpha) / ns * float(ws)
    assert np.array_equal(ref, want)
    assert np.all(absref >= np.abs(ref))


def test_adjoint_of_scipy_correlation():
    """<conv(a), g> = <a, dact> on integer codes, the forward convolution by
    scipy.signal.correlate2d ('same' size, zero fill)."""
    B, H, W, C, Cout = 2, 7, 9, 3, 4
    planes, alpha, wc, ws = _case(B, H, W, C, Cout, 1, seed=61)
    G = luq_decode_int(planes[0], B * H * W * Cout).reshape(B, H, W, Cout).astype(np.float64)
    Wq = int4_decode_int(wc, Cout * 9 * C, True).reshape(Cout, 3, 3, C).astype(np.float64)
    act = np.random.default_rng(5).integers(-7, 8, size=(B, H, W, C)).astype(np.float64)
    z = np.zeros((B, H, W, Cout))
    for b in range(B):
        for o in range(Cout):
            for c in range(C):
                z[b, :, :, o] += correlate2d(act[b, :, :, c], Wq[o, :, :, c], mode="same", fillvalue=0)
    dact, _ = conv3x3_dgrad_ref(planes, np.float32(1), wc, np.float32(1), True, B, H, W, C, Cout)
    assert np.sum(z * G) == np.sum(act.reshape(-1, C) * dact)
    # and a wrong tap orientation breaks it
    assert np.sum(z * G) != np.sum(np.flip(act, axis=(1, 2)).reshape(-1, C) * dact)


@pytest.mark.parametrize("ns,wsig", [(1, True), (2, True), (1, False)])
def test_equals_lowered_gemm_folded_onto_pixels(ns, wsig):
    B, H, W, C, Cout = 2, 5, 6, 4, 8
    planes, alpha, wc, ws = _case(B, H, W, C, Cout, ns, seed=62, wsig=wsig)
    T = B * H * W
    # the lowered GEMM (Eq. backward): dcol [T][9C] = Q(g) [T][Cout] Q(W) [Cout][9C]
    dcol, _ = gemm_dgrad_ref(planes, alpha, wc, ws, wsig, T, 9 * C, Cout)
    dcol = dcol.reshape(B, H, W, 3, 3, C)
    pad = np.zeros((B, H + 2, W + 2, C))
    for kh in range(3):
        for kw in range(3):
            pad[:, kh:kh + H, kw:kw + W, :] += dcol[:, :, :, kh, kw, :]
    want = pad[:, 1:H + 1, 1:W + 1, :].reshape(T, C)
    ref, _ = conv3x3_dgrad_ref(planes, alpha, wc, ws, wsig, B, H, W, C, Cout)
    assert np.allclose(ref, want, rtol=1e-12, atol=0)
    # a subset of pixels equals the same rows of the whole result
    pix = [0, 7, T - 1, 31]
    sub, _ = conv3x3_dgrad_ref(planes, alpha, wc, ws, wsig, B, H, W, C, Cout, pixels=pix)
    assert np.array_equal(sub, ref[pix])


# ----------------------------- weight gradient -----------------------------

from oracle.conv import conv3x3_wgrad_ref  # noqa: E402
from oracle.gemm import gemm_wgrad_ref  # noqa: E402
from oracle.im2col import im2col3x3_codes  # noqa: E402


def _wcase(B, H, W, C, Cout, ns, seed, asig):
    g = synth.lognormal_grad((B * H * W, Cout), -4.0, 2.0, 0.3, [seed, 1])
    a = synth.normal((B * H * W, C), 1.0, [seed, 2])
    planes, alpha, _ = luq_quantize(g, R=4, seed=seed, counter=3, n_samples=ns)
    ac, sa = int4_quantize(a if asig else np.abs(a), is_signed=asig)
    return planes, alpha, ac, sa


@pytest.mark.parametrize("ns,asig", [(1, False), (2, True)])
def test_wgrad_matches_loop_over_the_definition(ns, asig):
    B, H, W, C, Cout = 2, 3, 4, 2, 3
    planes, alpha, ac, sa = _wcase(B, H, W, C, Cout, ns, 70, asig)
    ref, absref = conv3x3_wgrad_ref(planes, alpha, ac, sa, asig, B, H, W, C, Cout)
    want = np.zeros((Cout, 9 * C))
    for o in range(Cout):
        for kh in range(3):
            for kw in range(3):
                for c in range(C):
                    acc = 0
                    for b in range(B):
                        for y in range(H):
                            for x in range(W):
                                ys, xs = y + kh - 1, x + kw - 1
                                if not (0 <= ys < H and 0 <= xs < W):
                                    continue
                                t, ts = (b * H + y) * W + x, (b * H + ys) * W + xs
                                gv = sum(_luq_val(_nib(p, t * Cout + o)) for p in planes)
                                av = _int4_val(_nib(ac, ts * C + c), asig)
                                acc += gv * av
                    want[o, (kh * 3 + kw) * C + c] = acc * float(alpha) / ns * float(sa)
    assert np.array_equal(ref, want)
    assert np.all(absref >= np.abs(ref))


@pytest.mark.parametrize("ns,asig", [(1, False), (2, True), (1, True)])
def test_wgrad_equals_gemm_on_lowered_activations(ns, asig):
    """Two formulations: the per-tap sum and Eq. update on the im2col lowering."""
    B, H, W, C, Cout = 2, 5, 7, 4, 6
    planes, alpha, ac, sa = _wcase(B, H, W, C, Cout, ns, 71, asig)
    T = B * H * W
    ref, absref = conv3x3_wgrad_ref(planes, alpha, ac, sa, asig, B, H, W, C, Cout)
    col = im2col3x3_codes(ac, B, H, W, C)
    low, lowabs = gemm_wgrad_ref(planes, alpha, col, sa, asig, T, Cout, 9 * C)
    assert np.allclose(ref, low, rtol=1e-12, atol=0)
    assert np.allclose(absref, lowabs, rtol=1e-12, atol=0)


def test_wgrad_adjoint_of_scipy_correlation():
    """<dW, K> = <g, conv(a; K)> on integer codes for a random integer kernel
    K [Cout][3][3][C], the forward convolution by scipy.signal.correlate2d."""
    B, H, W, C, Cout = 2, 6, 5, 3, 4
    planes, alpha, ac, sa = _wcase(B, H, W, C, Cout, 1, 72, True)
    G = luq_decode_int(planes[0], B * H * W * Cout).reshape(B, H, W, Cout).astype(np.float64)
    A = int4_decode_int(ac, B * H * W * C, True).reshape(B, H, W, C).astype(np.float64)
    K = np.random.default_rng(9).integers(-5, 6, size=(Cout, 3, 3, C)).astype(np.float64)
    z = np.zeros((B, H, W, Cout))
    for b in range(B):
        for o in range(Cout):
            for c in range(C):
                z[b, :, :, o] += correlate2d(A[b, :, :, c], K[o, :, :, c], mode="same", fillvalue=0)
    dW, _ = conv3x3_wgrad_ref(planes, np.float32(1), ac, np.float32(1), True, B, H, W, C, Cout)
    assert np.sum(z * G) == np.sum(dW.reshape(Cout, 3, 3, C) * K)
    # a flipped tap orientation breaks it
    assert np.sum(z * G) != np.sum(np.flip(dW.reshape(Cout, 3, 3, C), axis=(1, 2)) * K)


def test_im2col_lowering_against_padded_slices():
    """The lowering oracle against a direct gather with explicit bounds checks."""
    B, H, W, C = 2, 4, 5, 3
    codes = np.random.default_rng(3).integers(0, 256, size=(B * H * W * C + 1) // 2, dtype=np.uint8)
    col = im2col3x3_codes(codes, B, H, W, C)
    for t in range(B * H * W):
        b, rem = divmod(t, H * W)
        y, x = divmod(rem, W)
        for kh in range(3):
            for kw in range(3):
                for c in range(C):
                    ys, xs = y + kh - 1, x + kw - 1
                    want = _nib(codes, ((b * H + ys) * W + xs) * C + c) if (0 <= ys < H and 0 <= xs < W) else 0
                    assert _nib(col, t * 9 * C + (kh * 3 + kw) * C + c) == want

"""Activation and weight gradients of a 3x3 convolution on 4-bit codes -- oracle.

Test infrastructure only.  The convolution (stride 1, zero padding 1, NHWC,
weights [Cout][kh][kw][c]) is the GEMM of the lowered activations, so its
backward GEMM (Eq. backward) yields the gradient of the lowered activations;
the activation gradient sums, for every input pixel and channel, the entries
of the taps that read it (the adjoint of the lowering):

    dact[b, y, x, c] = sum over (kh, kw) and o of
                       g[b, y - kh + 1, x - kw + 1, o] * W[o, kh, kw, c]

with terms whose output pixel lies outside the image left out.  As in the
backward GEMM, every MAC is on codes -- LUQ integers of g (the SMP planes
summed, Section 5.1) times INT4 integers of W -- and the scales alpha / n and
s_W are applied once to the sum (Appendix A.1).  The sum is written per tap:
the code rows of g shifted by the tap's pixel offset (zero rows where the
source pixel is outside the image) times that tap's [Cout][C] slice of W.

The weight gradient (Eq. update on the lowered activations) sums, for every
output channel o, tap (kh, kw) and input channel c, over the output pixels
whose tap source lies on the image:

    dW[o, (kh*3 + kw)*C + c] = sum over (b, y, x) of
                               g[b, y, x, o] * act[b, y + kh - 1, x + kw - 1, c]

on codes: LUQ integers of g (planes summed) times INT4 integers of the
activations, scales alpha / n and s_a applied once.  Written per tap, not
through the lowered matrix.
"""

import numpy as np

from .luq import luq_decode_int
from .int4 import int4_decode_int


def _luq_matrix(g_planes, T, Cout):
    g_planes = np.asarray(g_planes, dtype=np.uint8)
    if g_planes.ndim == 1:
        g_planes = g_planes[None]
    A = np.zeros((T, Cout), dtype=np.int64)
    for p in g_planes:
        A += luq_decode_int(p, T * Cout).reshape(T, Cout)
    return A, g_planes.shape[0]


def conv3x3_dgrad_ref(g_planes, alpha, w_codes, w_scale, w_signed, B, H, W, C, Cout, pixels=None):
    """dact [len(pixels), C] (all B*H*W pixels if None) as float64, with the
    per-output sum of |a_k b_k| that the parity tolerance is relative to.

    g_planes: LUQ codes of g [B*H*W][Cout] (n planes); w_codes: INT4 codes of
    W [Cout][9*C] with columns in (kh, kw, c) order.
    """
    T = B * H * W
    A, n_s = _luq_matrix(g_planes, T, Cout)
    Wq = int4_decode_int(w_codes, Cout * 9 * C, w_signed).reshape(Cout, 3, 3, C)
    pix = np.arange(T) if pixels is None else np.asarray(pixels, dtype=np.int64)
    b, rem = np.divmod(pix, H * W)
    y, x = np.divmod(rem, W)
    acc = np.zeros((pix.size, C), dtype=np.float64)
    absacc = np.zeros((pix.size, C), dtype=np.float64)
    for kh in range(3):
        for kw in range(3):
            ys, xs = y - kh + 1, x - kw + 1
            ok = (ys >= 0) & (ys < H) & (xs >= 0) & (xs < W)
            src = np.where(ok, (b * H + ys) * W + xs, 0)
            rows = np.where(ok[:, None], A[src], 0).astype(np.float64)
            wt = Wq[:, kh, kw, :].astype(np.float64)          # [Cout, C]
            acc += rows @ wt
            absacc += np.abs(rows) @ np.abs(wt)
    bound = np.abs(A).max(initial=0) * np.abs(Wq).max(initial=0) * 9 * Cout
    assert bound < 2.0 ** 53, "sums would not be exact in float64"
    sc = float(alpha) / n_s * float(w_scale)
    return acc * sc, absacc * abs(sc)


def conv3x3_wgrad_ref(g_planes, alpha, a_codes, a_scale, a_signed, B, H, W, C, Cout):
    """dW [Cout, 9*C] as float64, with the per-output sum of |a_k b_k|.

    g_planes: LUQ codes of g [B*H*W][Cout] (n planes); a_codes: INT4 codes of
    the activations [B*H*W][C] (NHWC pixels).
    """
    T = B * H * W
    A, n_s = _luq_matrix(g_planes, T, Cout)
    X = int4_decode_int(a_codes, T * C, a_signed).reshape(B, H, W, C).astype(np.float64)
    G = A.reshape(B, H, W, Cout).astype(np.float64)
    acc = np.zeros((Cout, 3, 3, C), dtype=np.float64)
    absacc = np.zeros((Cout, 3, 3, C), dtype=np.float64)
    for kh in range(3):
        for kw in range(3):
            # output pixels (y, x) whose source (y + kh - 1, x + kw - 1) is on the image
            y0, y1 = max(0, 1 - kh), min(H, H + 1 - kh)
            x0, x1 = max(0, 1 - kw), min(W, W + 1 - kw)
            if y0 >= y1 or x0 >= x1:
                continue
            gs = G[:, y0:y1, x0:x1, :].reshape(-1, Cout)
            xs = X[:, y0 + kh - 1:y1 + kh - 1, x0 + kw - 1:x1 + kw - 1, :].reshape(-1, C)
            acc[:, kh, kw, :] = gs.T @ xs
            absacc[:, kh, kw, :] = np.abs(gs).T @ np.abs(xs)
    bound = np.abs(A).max(initial=0) * np.abs(X).max(initial=0) * T
    assert bound < 2.0 ** 53, "sums would not be exact in float64"
    sc = float(alpha) / n_s * float(a_scale)
    return (acc * sc).reshape(Cout, 9 * C), (absacc * abs(sc)).reshape(Cout, 9 * C)

"""The three 4-bit GEMMs on codes -- oracle.

Test infrastructure only.  Eq. forward, Eq. backward and Eq. update of the
paper:

    z_l       = Q_INT(W_l) Q_INT(a_{l-1})   (fwd, here y = Q(x) Q(W)^T)
    g_{l-1}   = Q_INT(W^T) Q_FP(delta)      (dgrad, here dX = Q(g) Q(W))
    dC/dW_l   = Q_FP(delta) Q_INT(a^T)      (wgrad, here dW = Q(g)^T Q(a))

Appendix A.1: every MAC runs on the low-precision codes and the per-tensor
scales (alpha of LUQ, s of INT4) are applied once to the sum.  This oracle
decodes the codes to small integers (LUQ: 0 or +-2^(e-1); INT4: q), sums the
SMP planes (Section 5.1: the averaged sample is (1/n) * sum of planes, so
the scale becomes alpha / n), forms the exact integer product with a float64
matrix multiply (every partial sum is an integer far below 2^53) and
multiplies by the scales in float64.

Layouts (row-major, two codes per byte along the row):
  fwd:   X [M, K] (tokens x input features), W [N, K] (the [out, in]
         weight); y [M, N].
  dgrad: G [M, K] (K = output features), W [K, N] (the [out, in] weight);
         dX [M, N].
  wgrad: G [T, Nout], A [T, Kin]; dW [Nout, Kin].

Each function also returns absref = (|A| @ |B|) * scale, the per-output sum
of |a_k b_k| that the parity tolerance is relative to.
"""

import numpy as np

from .luq import luq_decode_int, unpack_nibbles
from .int4 import int4_decode_int


def _rows_luq(planes, rows, ncols):
    """Summed LUQ integers of the selected rows of a [*, ncols] matrix."""
    planes = np.asarray(planes, dtype=np.uint8)
    if planes.ndim == 1:
        planes = planes[None]
    rb = ncols // 2
    out = np.zeros((len(rows), ncols), dtype=np.int64)
    for p in planes:
        mat = p[: (p.size // rb) * rb].reshape(-1, rb)[rows]
        out += luq_decode_int(mat.ravel(), len(rows) * ncols).reshape(len(rows), ncols)
    return out


def _rows_int4(codes, rows, ncols, signed):
    rb = ncols // 2
    codes = np.asarray(codes, dtype=np.uint8)
    mat = codes[: (codes.size // rb) * rb].reshape(-1, rb)[rows]
    return int4_decode_int(mat.ravel(), len(rows) * ncols, signed).reshape(len(rows), ncols)


def _matmul_exact(A, B):
    """Exact integer product through float64 BLAS (|sums| < 2^53 asserted)."""
    Af = A.astype(np.float64)
    Bf = B.astype(np.float64)
    bound = np.abs(Af).max(initial=0) * np.abs(Bf).max(initial=0) * A.shape[1]
    assert bound < 2.0 ** 53, "partial sums would not be exact in float64"
    return Af @ Bf, np.abs(Af) @ np.abs(Bf)


def _scale(alpha, n_samples, s):
    return float(alpha) / n_samples * float(s)


def gemm_dgrad_ref(g_planes, alpha, w_codes, w_scale, w_signed, M, N, K, rows=None):
    """dX[m, n] = sum_k (alpha/n_s sum_s c_g^s[m, k]) (s_W c_W[k, n]).

    rows: optional subset of output rows (all rows if None).
    Returns (ref, absref) as float64 arrays of shape (len(rows), N).
    """
    rows = np.arange(M) if rows is None else np.asarray(rows)
    g_planes = np.asarray(g_planes, dtype=np.uint8)
    n_s = 1 if g_planes.ndim == 1 else g_planes.shape[0]
    A = _rows_luq(g_planes, rows, K)
    B = _rows_int4(w_codes, np.arange(K), N, w_signed)
    ref, absref = _matmul_exact(A, B)
    sc = _scale(alpha, n_s, w_scale)
    return ref * sc, absref * abs(sc)


def gemm_wgrad_ref(g_planes, alpha, a_codes, a_scale, a_signed, T, Nout, Kin, rows=None, t_range=None):
    """dW[o, i] = sum_t (alpha/n_s sum_s c_g^s[t, o]) (s_a c_a[t, i]).

    rows: optional subset of output rows o.  t_range: optional (t0, t1) slice
    of the reduction, used to bound the work on very large inputs.
    Returns (ref, absref) of shape (len(rows), Kin).
    """
    rows = np.arange(Nout) if rows is None else np.asarray(rows)
    g_planes = np.asarray(g_planes, dtype=np.uint8)
    n_s = 1 if g_planes.ndim == 1 else g_planes.shape[0]
    t0, t1 = (0, T) if t_range is None else t_range
    ts = np.arange(t0, t1)
    G = _rows_luq(g_planes, ts, Nout)[:, rows]          # [T', len(rows)]
    X = _rows_int4(a_codes, ts, Kin, a_signed)         # [T', Kin]
    ref, absref = _matmul_exact(G.T, X)
    sc = _scale(alpha, n_s, a_scale)
    return ref * sc, absref * abs(sc)


def gemm_fwd_ref(x_codes, x_scale, x_signed, w_codes, w_scale, w_signed, M, N, K, rows=None):
    """y[m, n] = (s_x s_W) sum_k q_x[m, k] q_W[n, k] (Appendix A.1: the
    scales of the two INT4 tensors leave the sum, every MAC is on codes).

    rows: optional subset of output rows (all rows if None).
    Returns (ref, absref) as float64 arrays of shape (len(rows), N).
    """
    rows = np.arange(M) if rows is None else np.asarray(rows)
    X = _rows_int4(x_codes, rows, K, x_signed)         # [len(rows), K]
    Wm = _rows_int4(w_codes, np.arange(N), K, w_signed)  # [N, K]
    ref, absref = _matmul_exact(X, Wm.T)
    sc = float(x_scale) * float(w_scale)
    return ref * sc, absref * abs(sc)


def decode_plane_matrix(plane, rows, cols):
    """Unpacked nibbles of a [rows, cols] code matrix (diagnostics)."""
    return unpack_nibbles(plane, rows * cols).reshape(rows, cols)

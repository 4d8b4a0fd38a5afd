"""Uniform INT4 round-to-nearest quantizer for weights and activations -- oracle.

Test infrastructure only.  Section 3.3 of the paper fixes round-to-nearest for
Q_INT in every phase; Appendix A.1 gives the per-tensor scale
alpha = Delta / (2^b - 1) with Delta the quantized range, applied once after
the low-precision MACs.  The paper picks Delta with SAWB, whose regression
coefficients it does not give, so here Delta is max-abs (or a caller clip).

Readings adopted:

* signed codes q in -7..7 with scale s = m / 7 (symmetric, zero-point 0, as
  the scale factorisation of Appendix A.1 requires); unsigned codes q in 0..15
  with s = m / 15 (the literal Delta / (2^4 - 1)), negatives clamp to 0;
* m = clip if clip > 0, else max|x| (signed) or max(max x, 0) (unsigned);
* inv = fl32(Q / m), s = fl32(m / Q), q = clamp(rint_half_even(fl32(x * inv)));
  a product that is NaN (0 * inf when m is tiny) gives q = 0;
* m = 0 gives s = 0 and all codes 0; a non-finite max gives s = NaN and all
  codes 0;
* signed codes are stored as 4-bit two's complement, two per byte, element 2b
  in the low nibble.
"""

import numpy as np

from .luq import to_float32, pack_nibbles, unpack_nibbles


def int4_quantize(x, dtype="f32", is_signed=True, clip=0.0):
    """Returns (codes uint8 of length ceil(N/2), scale float32)."""
    xf = to_float32(x, dtype).ravel()
    N = xf.size
    codes = np.zeros((N + 1) // 2, dtype=np.uint8)
    if N == 0:
        return codes, np.float32(0.0)
    Q = np.float32(7.0 if is_signed else 15.0)
    if clip > 0:
        m = np.float32(clip)
    else:
        if not np.all(np.isfinite(xf)):
            return codes, np.float32(np.nan)
        m = np.float32(np.abs(xf).max()) if is_signed else np.float32(max(xf.max(), 0.0))
    if not np.isfinite(m):
        return codes, np.float32(np.nan)
    if m == 0:
        return codes, np.float32(0.0)
    with np.errstate(over="ignore", invalid="ignore"):
        inv = np.float32(Q / m)
        s = np.float32(m / Q)
        v = (xf * inv).astype(np.float32)
        q = np.rint(v)
    q = np.where(np.isnan(q), 0.0, q)
    lo = -7.0 if is_signed else 0.0
    q = np.clip(q, lo, float(Q)).astype(np.int64)
    nib = (q & 0xF).astype(np.uint8)
    return pack_nibbles(nib), s


def int4_decode_int(codes, n, is_signed):
    nib = unpack_nibbles(codes, n).astype(np.int64)
    if is_signed:
        return np.where(nib >= 8, nib - 16, nib)
    return nib


def int4_decode(codes, n, scale, is_signed):
    return int4_decode_int(codes, n, is_signed).astype(np.float64) * float(scale)

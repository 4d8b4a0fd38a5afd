"""Logarithmic unbiased quantization (LUQ) of neural gradients -- oracle.

Test infrastructure only.  Follows Section 4 of the paper in its order:

1. Underflow threshold (Eq. alpha): alpha = max|x| / 2^(2^(b-1)).  With b = 3
   exponent bits this is max|x| / 16; the exponent 2^(b-1) is called R here
   and is a parameter (default 4).  alpha is rounded once to float32.
2. Quantization levels alpha * 2^n, n = 0..R.  The largest level equals
   max|x|, so nothing is clipped (Section 4, "Above FP maximum").
3. Stochastic underflow T_alpha (Eq. StochasticPruning): |x| < alpha becomes
   sign(x)*alpha with probability |x|/alpha, else 0.
4. Logarithmic stochastic rounding Q_alpha (Eq. unbiasedFpQ): inside the bin
   [alpha*2^(n-1), alpha*2^n] round up with probability
   (|x| - alpha*2^(n-1)) / (alpha*2^(n-1)).
5. X_q = Q_alpha(T_alpha(x)) is unbiased by the law of total expectation.
6. SMP (Section 5.1): n independent samples with the same alpha; their mean
   has 1/n of the variance.

Power-of-two LUQ (Appendix, "Power-of-two LUQ"): alpha is replaced by
alpha_PW2 = 2^ceil(log2 max|x|) / 2^R, so every level is a power of two and
the top level is the least power of two at or above max|x| (nothing is
clipped); steps 2-6 are unchanged.

Readings of points the paper leaves open (each also listed in the design
notes of the repository):

* R (number of binades above alpha) defaults to 4 (Eq. alpha with b = 3).
* Code format: a 4-bit nibble, bit 3 = sign, bits 2..0 = exponent field e;
  e = 0 encodes zero (sign bit forced to 0), e >= 1 encodes
  (-1)^sign * alpha * 2^(e-1).  The MF-BPROP worked example (Appendix A.8.1:
  FP4 bits 011 times INT4 3 gives 12) fixes field 011 <-> 4 = 2^(3-1).
* T_alpha and Q_alpha share one uniform per element: applying T_alpha then
  Q_alpha is stochastic rounding on the grid {0, alpha, 2alpha, ..., 2^R alpha}
  with bins [0, alpha] and [alpha 2^n, alpha 2^(n+1)], which has the same
  distribution as the two-draw composition.
* The uniform is a 16-bit integer j (see ``philox``) and the rounding decision
  is exact: round up iff j * w < d * 2^16, with w the bin width and
  d = |x| - (bin lower level).  So P(up) = ceil(2^16 d / w) / 2^16 and
  0 <= E[Q(x)] - x < w * 2^-16.
* A value exactly on a level never moves; |x| >= alpha*2^R maps to the top
  level deterministically (only possible for the max itself, or above it
  when alpha was rounded as a subnormal).
* If alpha rounds to 0 (max|x| = 0, or so small that max/2^R underflows
  float32) every code is 0.
* Non-finite input: alpha = NaN and every code is 0.  In-hindsight mode: a
  step whose measured maximum is not finite leaves the estimate unchanged.
* Packing: two codes per byte, element 2b in the low nibble of byte b; an
  odd element count leaves the last high nibble 0.
"""

import math
from fractions import Fraction

import numpy as np

from .philox import luq_uniforms, luq_uniforms_at

TWO16 = 65536


def to_float32(x, dtype="f32"):
    """Exact float32 view of the input (bfloat16 is given as its uint16 bits)."""
    x = np.asarray(x)
    if dtype == "bf16":
        if x.dtype != np.uint16:
            raise TypeError("bf16 input must be given as uint16 bit patterns")
        return (x.astype(np.uint32) << np.uint32(16)).view(np.float32)
    if dtype == "f32":
        return x.astype(np.float32, copy=False)
    raise ValueError(dtype)


def luq_alpha(maxabs, R):
    """Eq. alpha: alpha = max|x| / 2^R, rounded to float32 (exact unless subnormal)."""
    return np.float32(float(maxabs) * 2.0 ** (-R))


def luq_alpha_pw2(maxabs, R):
    """Power-of-two alpha (Appendix, power-of-two LUQ): 2^ceil(log2 max|x|) / 2^R
    as float32 -- exact, or 0 where 2^(ceil - R) is below half the smallest
    float32 subnormal (it rounds to 0, as the plain alpha does there)."""
    m = float(maxabs)
    if not m > 0:
        return np.float32(0.0)
    mant, e = math.frexp(m)            # m = mant * 2^e, 0.5 <= mant < 1
    c = e - 1 if mant == 0.5 else e    # ceil(log2 m)
    return np.float32(math.ldexp(1.0, c - R))


def luq_levels(alpha, R):
    """Levels alpha * 2^n for n = 0..R, exact in float64."""
    return np.array([float(alpha) * 2.0 ** n for n in range(R + 1)], dtype=np.float64)


def pack_nibbles(nib):
    """Two 4-bit codes per byte, element 2b in the low nibble."""
    nib = np.asarray(nib, dtype=np.uint8).ravel()
    if nib.size % 2:
        nib = np.concatenate([nib, np.zeros(1, dtype=np.uint8)])
    return (nib[0::2] & 0xF) | ((nib[1::2] & 0xF) << 4)


def unpack_nibbles(codes, n):
    codes = np.asarray(codes, dtype=np.uint8).ravel()
    out = np.empty(codes.size * 2, dtype=np.uint8)
    out[0::2] = codes & 0xF
    out[1::2] = codes >> 4
    return out[:n]


def luq_fields(a, alpha, R, j):
    """Exponent field e (0..R+1) for magnitudes a (float64) given uniforms j.

    Section 4: bins are [0, alpha) (stochastic underflow, lower value 0) and
    [alpha 2^n, alpha 2^(n+1)) for n = 0..R-1 (logarithmic SR); magnitudes at
    or above alpha 2^R take the top level.
    """
    a = np.asarray(a, dtype=np.float64)
    j = np.asarray(j, dtype=np.float64)
    L = luq_levels(alpha, R)
    top = a >= L[R]
    # n = index of the highest level <= a (only meaningful where a >= alpha)
    n = np.zeros(a.shape, dtype=np.int64)
    for k in range(1, R):
        n += (a >= L[k])
    under = a < L[0]
    lo = np.where(under, 0.0, L[np.minimum(n, R)])
    w = np.where(under, L[0], L[np.minimum(n, R)])
    base = np.where(under, 0, n + 1)
    d = a - lo  # exact: Sterbenz when lo <= a < 2 lo, trivially when lo = 0
    up = (j * w) < (d * TWO16)  # both sides exact in float64
    e = base + up.astype(np.int64)
    e = np.where(top, R + 1, e)
    return e.astype(np.uint8)


def luq_quantize(x, dtype="f32", R=4, seed=0, counter=0, n_samples=1, pw2=False):
    """Quantize a gradient tensor with LUQ (with pw2: power-of-two LUQ).

    Returns (codes, alpha, maxabs): codes is uint8 of shape
    (n_samples, ceil(N/2)) -- one packed plane per SMP sample -- and alpha,
    maxabs are float32 scalars.
    """
    xf = to_float32(x, dtype).ravel()
    N = xf.size
    nbytes = (N + 1) // 2
    codes = np.zeros((n_samples, nbytes), dtype=np.uint8)
    if N == 0:
        return codes, np.float32(0.0), np.float32(0.0)
    a = np.abs(xf.astype(np.float64))
    if not np.all(np.isfinite(a)):
        mx = np.float32(np.nan) if np.any(np.isnan(a)) else np.float32(np.inf)
        return codes, np.float32(np.nan), mx
    maxabs = np.float32(a.max())
    alpha = luq_alpha_pw2(maxabs, R) if pw2 else luq_alpha(maxabs, R)
    if alpha == 0:
        return codes, alpha, maxabs
    for s in range(n_samples):
        codes[s] = pack_nibbles(luq_nibbles_range(xf, 0, alpha, R, seed, counter, s))
    return codes, alpha, maxabs


def hindsight_estimate(m_hat):
    """The estimate as the quantizer reads it: NaN stays NaN, anything not
    positive is 0."""
    m = np.float32(m_hat)
    if np.isnan(m):
        return np.float32(np.nan)
    return m if m > 0 else np.float32(0.0)


def hindsight_update(maxabs, m_hat, eta):
    """Eq. hindsight: m^t = (1 - eta) max|x^(t-1)| + eta m^(t-1), in float32:
    fl32(fl32(fl32(1 - eta) * max) + fl32(fl32(eta) * m))."""
    c1 = np.float32(np.float32(1.0) - np.float32(eta))
    c0 = np.float32(eta)
    with np.errstate(invalid="ignore", over="ignore"):
        return np.float32(np.float32(c1 * np.float32(maxabs)) + np.float32(c0 * np.float32(m_hat)))


def luq_quantize_hindsight(x, m_hat, dtype="f32", R=4, seed=0, counter=0, n_samples=1, eta=0.1, pw2=False):
    """LUQ in one pass with the in-hindsight maximum (Section 4, "Reducing the
    data movement"; Appendix on hindsight).

    The tensor is quantized with alpha = fl32(m_hat / 2^R) from the estimate
    carried over from the previous step, while its own max|x| is measured;
    the estimate for the next step follows Eq. hindsight.  Magnitudes at or
    above alpha 2^R (the estimate may be below this tensor's maximum) take the
    top level with their sign, as does a NaN element; codes are otherwise
    those of ``luq_fields`` (Section 4).  A non-finite estimate gives alpha =
    NaN and all codes 0, a zero estimate all codes 0.  With pw2 the alpha of
    the estimate is the power-of-two one (the combination of the appendix's
    power-of-two LUQ with hindsight).

    Eq. hindsight is an average of measured maxima and says nothing of a
    step whose maximum is not a number (an overflowed gradient).  Reading:
    such a step, which a training loop skips, does not enter the average, so
    m_next is m_hat unchanged; otherwise one overflow would make every later
    alpha NaN.

    Returns (codes, alpha, maxabs, m_next).
    """
    xf = to_float32(x, dtype).ravel()
    N = xf.size
    codes = np.zeros((n_samples, (N + 1) // 2), dtype=np.uint8)
    m = hindsight_estimate(m_hat)
    alpha = np.float32(np.nan) if not np.isfinite(m) else (luq_alpha_pw2(m, R) if pw2 else luq_alpha(m, R))
    a = np.abs(xf.astype(np.float64))
    if N == 0:
        maxabs = np.float32(0.0)
    elif np.any(np.isnan(a)):
        maxabs = np.float32(np.nan)
    else:
        maxabs = np.float32(a.max())
    if np.isfinite(alpha) and alpha > 0 and N > 0:
        a_top = np.where(np.isnan(a), np.inf, a)
        for s in range(n_samples):
            e = luq_fields(a_top, alpha, R, luq_uniforms(N, seed, counter, s))
            nib = e | np.where((e != 0) & np.signbit(xf), 8, 0).astype(np.uint8)
            codes[s] = pack_nibbles(nib)
    m_next = hindsight_update(maxabs, m, eta) if np.isfinite(maxabs) else np.float32(m_hat)
    return codes, alpha, maxabs, m_next


def luq_nibbles_range(xf, start, alpha, R, seed, counter, sample):
    """Unpacked codes of the elements start .. start+len(xf)-1 of a tensor
    whose alpha is already known (xf: their float32 values).  The codes of a
    slice equal the slice of the whole tensor's codes: the uniforms depend
    only on the element's flat index."""
    xf = np.asarray(xf, dtype=np.float32).ravel()
    if not (float(alpha) > 0):  # zero or NaN alpha: all codes 0
        return np.zeros(xf.size, dtype=np.uint8)
    a = np.abs(xf.astype(np.float64))
    j = luq_uniforms(xf.size, seed, counter, sample, start=start)
    e = luq_fields(a, alpha, R, j)
    return e | np.where((e != 0) & np.signbit(xf), 8, 0).astype(np.uint8)


def luq_nibbles_at(xf, idx, alpha, R, seed, counter, sample):
    """Unpacked codes of the elements at flat indices idx of a tensor whose
    alpha is already known (xf: their float32 values, in the order of idx)."""
    xf = np.asarray(xf, dtype=np.float32).ravel()
    if not (float(alpha) > 0):
        return np.zeros(xf.size, dtype=np.uint8)
    a = np.abs(xf.astype(np.float64))
    e = luq_fields(a, alpha, R, luq_uniforms_at(idx, seed, counter, sample))
    return e | np.where((e != 0) & np.signbit(xf), 8, 0).astype(np.uint8)


def luq_decode_int(codes, n):
    """Signed integer multiples of alpha: 0 or +-2^(e-1) (int64 array of length n)."""
    nib = unpack_nibbles(codes, n).astype(np.int64)
    e = nib & 7
    mag = np.where(e == 0, 0, np.left_shift(1, np.maximum(e - 1, 0)))
    return np.where(nib & 8, -mag, mag)


def luq_smp_sum(planes, n):
    """SMP operand (Section 5.1) as one integer per element: the sum over the
    n_s sample planes of the signed multiples of alpha, so that the averaged
    gradient is (alpha / n_s) * sum.  int8 array of length n; |sum| <= n_s *
    2^R, which fits int8 for two samples with R <= 5."""
    planes = np.asarray(planes, dtype=np.uint8)
    if planes.ndim == 1:
        planes = planes[None]
    tot = np.zeros(n, dtype=np.int64)
    for p in planes:
        tot += luq_decode_int(p, n)
    assert np.all(np.abs(tot) <= 127), "sum does not fit int8"
    return tot.astype(np.int8)


def luq_decode(codes, n, alpha):
    """Dequantized values (float64)."""
    return luq_decode_int(codes, n).astype(np.float64) * float(alpha)


def luq_field_scalar(a, alpha, R, j):
    """One element's field in exact rational arithmetic (independent restatement).

    a, alpha: floats (taken exactly); j: integer uniform in [0, 2^16).
    """
    a = Fraction(float(a))
    alpha = Fraction(float(alpha))
    if alpha == 0:
        return 0
    levels = [alpha * 2 ** n for n in range(R + 1)]
    if a >= levels[R]:
        return R + 1
    if a < levels[0]:
        lo, w, base = Fraction(0), alpha, 0
    else:
        n = max(k for k in range(R) if levels[k] <= a)
        lo, w, base = levels[n], levels[n], n + 1
    return base + (1 if j * w < (a - lo) * TWO16 else 0)

"""Seeded synthetic inputs shared by the oracle side and the HIP side.

This module draws tensors and nothing else: it holds none of the quantizers'
or GEMMs' arithmetic.  Distributions follow the near-lognormal model of
neural gradients that the paper builds on (Section 1; Chmiel et al. 2020),
normal / half-normal activations and He- or std-initialised weights.

Notation: ``lognormal(mu, sigma)`` means ln|g| ~ N(mu, sigma^2) with a random
sign (p = 1/2); ``zero_frac`` of the entries are set to exact zeros (as a ReLU
derivative would); He weights have variance 2 / fan_in.  bfloat16 tensors are
drawn in float32 and rounded to nearest-even, returned as uint16 bit patterns.

Workloads (shapes of the paper's ResNet-50 and Transformer layers):
  small   -- one linear layer: g 256x512 lognormal(-10, 2) with 50% zeros,
             a 256x512 half-normal, W 512x512 He.                    seed 0
  resnet  -- ResNet-50 3x3 conv (64->64 channels, 56x56, batch 64) as GEMMs:
             act NHWC [64,56,56,64] half-normal, g [200704, 64]
             lognormal(-12, 2.5) with 50% zeros, W [64, 576] He.       seed 2
  mlp     -- Transformer MLP linear (8192 tokens, 4096 -> 16384): g [8192,
             16384] bf16 lognormal(-14, 3), x [8192, 4096] bf16 N(0,1),
             W [16384, 4096] fp32 N(0, 0.02^2).                        seed 3
  sweep   -- 1-D gradients of 2^k elements, lognormal(-10, 3), zero
             fraction 0..0.5, fp32 or bf16.
"""

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

CHUNK = 1 << 24


def _rng(seed):
    return np.random.default_rng(seed)


def _chunked(n, seed, fill):
    """float32 array of n entries drawn chunk by chunk; chunk c uses its own
    generator seeded with seed + [c], so the result does not depend on how
    many threads fill the chunks."""
    out = np.empty(n, dtype=np.float32)
    base = [int(s) for s in np.atleast_1d(seed)]

    def one(c0):
        c1 = min(n, c0 + CHUNK)
        out[c0:c1] = fill(_rng(base + [c0 // CHUNK]), c1 - c0)

    starts = range(0, n, CHUNK)
    if n > CHUNK:
        with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
            list(ex.map(one, starts))
    else:
        for c0 in starts:
            one(c0)
    return out


def lognormal_grad(shape, mu, sigma, zero_frac, seed):
    """float32 tensor with ln|g| ~ N(mu, sigma^2), random sign, exact zeros."""
    def fill(r, m):
        z = r.standard_normal(m, dtype=np.float32)
        mag = np.exp(np.float32(mu) + np.float32(sigma) * z)
        u = r.random(m, dtype=np.float32)
        sgn = np.where(r.random(m, dtype=np.float32) < 0.5, -1.0, 1.0).astype(np.float32)
        v = mag * sgn
        if zero_frac > 0:
            v = np.where(u < zero_frac, np.float32(0.0), v)
        return v

    return _chunked(int(np.prod(shape)), seed, fill).reshape(shape)


def normal(shape, std, seed):
    def fill(r, m):
        return r.standard_normal(m, dtype=np.float32) * np.float32(std)

    return _chunked(int(np.prod(shape)), seed, fill).reshape(shape)


def half_normal(shape, seed):
    return np.abs(normal(shape, 1.0, seed))


def to_bf16_bits(x):
    """Round float32 to bfloat16 (nearest-even); returns uint16 bit patterns."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
    out = (rounded >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(np.asarray(x, dtype=np.float32))
    if nan.any():
        out = np.where(nan, np.uint16(0x7FC0), out)
    return out


def bf16_bits_to_f32(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def small(seed=0):
    """One linear layer backward: M=256 tokens, 512 -> 512 features."""
    return {
        "g": lognormal_grad((256, 512), -10.0, 2.0, 0.5, [seed, 1]),
        "a": half_normal((256, 512), [seed, 2]),
        "W": normal((512, 512), np.sqrt(2.0 / 512), [seed, 3]),
    }


RESNET = dict(B=64, H=56, W=56, C=64, Cout=64)


def resnet(seed=2):
    """ResNet-50 3x3 conv backward lowered to GEMMs (im2col on codes)."""
    p = RESNET
    T = p["B"] * p["H"] * p["W"]
    return {
        "act": half_normal((p["B"], p["H"], p["W"], p["C"]), [seed, 1]),
        "g": lognormal_grad((T, p["Cout"]), -12.0, 2.5, 0.5, [seed, 2]),
        "W": normal((p["Cout"], 9 * p["C"]), np.sqrt(2.0 / (9 * p["C"])), [seed, 3]),
    }


MLP = dict(T=8192, D=4096, F=16384)


def mlp(seed=3, T=None, D=None, F=None):
    """Transformer MLP up-projection backward (bf16 gradients and activations).

    T, D, F override the token count and feature sizes (same distributions),
    which the parity tests use for scaled-down shapes.
    """
    T = T or MLP["T"]
    D = D or MLP["D"]
    F = F or MLP["F"]
    return {
        "g": to_bf16_bits(lognormal_grad((T, F), -14.0, 3.0, 0.0, [seed, 1])),
        "x": to_bf16_bits(normal((T, D), 1.0, [seed, 2])),
        "W": normal((F, D), 0.02, [seed, 3]),
    }


def sweep(k, dtype="f32", zero_frac=0.25, seed=4):
    """1-D gradient of 2^k elements (k may also be given as an explicit count via n=)."""
    n = 1 << k
    g = lognormal_grad((n,), -10.0, 3.0, zero_frac, [seed, k, 0 if dtype == "f32" else 1, int(zero_frac * 100)])
    return to_bf16_bits(g) if dtype == "bf16" else g


def grad_1d(n, dtype="f32", zero_frac=0.25, seed=5, mu=-10.0, sigma=3.0):
    """1-D gradient of an arbitrary length n."""
    g = lognormal_grad((n,), mu, sigma, zero_frac, [seed, n])
    return to_bf16_bits(g) if dtype == "bf16" else g

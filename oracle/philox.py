"""Philox4x32-10 counter-based generator (oracle; test infrastructure only).

Definition (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as
1, 2, 3", SC'11): a 128-bit counter (x0, x1, x2, x3) and a 64-bit key (k0, k1)
go through ten rounds.  Each round forms the two full 64-bit products
M0*x0 and M1*x2 and replaces the counter by

    (hi(M1*x2) ^ x1 ^ k0,  lo(M1*x2),  hi(M0*x0) ^ x3 ^ k1,  lo(M0*x0))

after which the key is bumped by the Weyl constants (W0, W1) mod 2^32.  The
output block is the counter after the tenth round.

How LUQ draws from it (this implementation's convention; the paper does not
name a generator): element i of a tensor, stochastic sample s (Section 5.1
SMP plane index) and step counter c use

    key = (seed mod 2^32, seed >> 32)
    ctr = (blk mod 2^32, blk >> 32, s, c)          with blk = i >> 3
    j_i = (y[(i >> 1) & 3] >> (16 * (i & 1))) & 0xFFFF

so one Philox call yields the 16-bit uniforms of 8 consecutive elements.

Two formulations are given: ``philox4x32_10`` (vectorised NumPy on uint64)
and ``philox4x32_10_scalar`` (Python integers); the tests check them against
each other and against an independent library implementation.
"""

import numpy as np

M0 = 0xD2511F53
M1 = 0xCD9E8D57
W0 = 0x9E3779B9
W1 = 0xBB67AE85
MASK32 = 0xFFFFFFFF
ROUNDS = 10


def philox4x32_10(ctr, key):
    """Vectorised Philox4x32-10.

    ctr: uint32 array of shape (..., 4); key: sequence of two uint32.
    Returns a uint32 array of shape (..., 4).
    """
    ctr = np.asarray(ctr, dtype=np.uint32)
    x0 = ctr[..., 0].astype(np.uint64)
    x1 = ctr[..., 1].astype(np.uint64)
    x2 = ctr[..., 2].astype(np.uint64)
    x3 = ctr[..., 3].astype(np.uint64)
    k0 = int(key[0]) & MASK32
    k1 = int(key[1]) & MASK32
    m32 = np.uint64(MASK32)
    s32 = np.uint64(32)
    for _ in range(ROUNDS):
        # both factors are below 2^32, so the uint64 products are exact
        p0 = np.uint64(M0) * x0
        p1 = np.uint64(M1) * x2
        hi0, lo0 = p0 >> s32, p0 & m32
        hi1, lo1 = p1 >> s32, p1 & m32
        x0, x1, x2, x3 = (hi1 ^ x1 ^ np.uint64(k0), lo1,
                          hi0 ^ x3 ^ np.uint64(k1), lo0)
        k0 = (k0 + W0) & MASK32
        k1 = (k1 + W1) & MASK32
    return np.stack([x0, x1, x2, x3], axis=-1).astype(np.uint32)


def philox4x32_10_scalar(ctr, key):
    """The same function on Python integers, one block at a time."""
    x = [int(v) & MASK32 for v in ctr]
    k0, k1 = int(key[0]) & MASK32, int(key[1]) & MASK32
    for _ in range(ROUNDS):
        p0 = M0 * x[0]
        p1 = M1 * x[2]
        x = [((p1 >> 32) ^ x[1] ^ k0) & MASK32, p1 & MASK32,
             ((p0 >> 32) ^ x[3] ^ k1) & MASK32, p0 & MASK32]
        k0 = (k0 + W0) & MASK32
        k1 = (k1 + W1) & MASK32
    return tuple(x)


def luq_uniforms(n, seed, counter, sample, start=0):
    """16-bit uniforms j_i for elements i = start .. start+n-1 (uint32 array)."""
    if n <= 0:
        return np.zeros(0, dtype=np.uint32)
    idx = np.arange(start, start + n, dtype=np.uint64)
    blk_first = int(start) >> 3
    blk_last = (int(start) + n - 1) >> 3
    blks = np.arange(blk_first, blk_last + 1, dtype=np.uint64)
    ctr = np.empty((blks.size, 4), dtype=np.uint32)
    ctr[:, 0] = (blks & np.uint64(MASK32)).astype(np.uint32)
    ctr[:, 1] = (blks >> np.uint64(32)).astype(np.uint32)
    ctr[:, 2] = np.uint32(sample & MASK32)
    ctr[:, 3] = np.uint32(counter & MASK32)
    key = (seed & MASK32, (seed >> 32) & MASK32)
    y = philox4x32_10(ctr, key)
    b = (idx >> np.uint64(3)) - np.uint64(blk_first)
    word = (idx >> np.uint64(1)) & np.uint64(3)
    half = idx & np.uint64(1)
    yw = y[b.astype(np.int64), word.astype(np.int64)].astype(np.uint32)
    return (yw >> (np.uint32(16) * half.astype(np.uint32))) & np.uint32(0xFFFF)


def luq_uniforms_at(idx, seed, counter, sample):
    """16-bit uniforms j_i for arbitrary flat element indices idx (uint32 array).

    The same mapping as ``luq_uniforms``: element i reads half (i & 1) of word
    ((i >> 1) & 3) of the Philox block for counter (i >> 3, sample, counter)."""
    idx = np.asarray(idx, dtype=np.uint64).ravel()
    if idx.size == 0:
        return np.zeros(0, dtype=np.uint32)
    blks, inv = np.unique(idx >> np.uint64(3), return_inverse=True)
    ctr = np.empty((blks.size, 4), dtype=np.uint32)
    ctr[:, 0] = (blks & np.uint64(MASK32)).astype(np.uint32)
    ctr[:, 1] = (blks >> np.uint64(32)).astype(np.uint32)
    ctr[:, 2] = np.uint32(sample & MASK32)
    ctr[:, 3] = np.uint32(counter & MASK32)
    y = philox4x32_10(ctr, (seed & MASK32, (seed >> 32) & MASK32))
    word = ((idx >> np.uint64(1)) & np.uint64(3)).astype(np.int64)
    half = (idx & np.uint64(1)).astype(np.uint32)
    yw = y[inv.ravel(), word].astype(np.uint32)
    return (yw >> (np.uint32(16) * half)) & np.uint32(0xFFFF)

"""Pins for the oracle's Philox4x32-10 generator (CPU).

The generator is pinned to rocRAND's independent implementation (stored blocks
in tests/golden/philox_rocrand.txt, and a live host build when hipcc is
present), to a second formulation on Python integers, and to basic uniformity
of the 16-bit draws LUQ takes from it.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle.philox import philox4x32_10, philox4x32_10_scalar, luq_uniforms, luq_uniforms_at

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden():
    rows = []
    with open(os.path.join(GOLDEN, "philox_rocrand.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            v = [int(t, 16) for t in line.split()]
            rows.append(v)
    return rows


def _ctr(blk, s, c):
    return np.array([blk & 0xFFFFFFFF, blk >> 32, s, c], dtype=np.uint32)


def test_philox_matches_rocrand_golden():
    rows = _golden()
    assert len(rows) >= 60
    for seed, blk, s, c, *y in rows:
        got = philox4x32_10(_ctr(blk, s, c), (seed & 0xFFFFFFFF, seed >> 32))
        assert [int(v) for v in got] == y, (hex(seed), hex(blk), s, c)


def test_philox_zero_block_known_answer():
    # counter 0, key 0: the first block rocRAND's engine produces
    got = philox4x32_10(np.zeros(4, np.uint32), (0, 0))
    assert [int(v) for v in got] == [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]


@pytest.mark.skipif(shutil.which("hipcc") is None, reason="hipcc not available")
def test_philox_matches_rocrand_live(tmp_path):
    exe = tmp_path / "pin"
    subprocess.run(["hipcc", "-O1", "-x", "hip", "--offload-arch=gfx950", "-I/opt/rocm/include",
                    os.path.join(GOLDEN, "philox_rocrand_pin.cpp"), "-o", str(exe)], check=True)
    rng = np.random.default_rng(123)
    items = []
    for _ in range(200):
        seed = int(rng.integers(0, 2**63)) * 2 + int(rng.integers(0, 2))
        blk = int(rng.integers(0, 2**62))
        items.append((seed, blk, int(rng.integers(0, 2)), int(rng.integers(0, 2**32))))
    inp = "".join("%x %x %x %x\n" % it for it in items)
    out = subprocess.run([str(exe)], input=inp, capture_output=True, text=True, check=True).stdout
    for (seed, blk, s, c), line in zip(items, out.splitlines()):
        y = [int(t, 16) for t in line.split()[4:]]
        got = philox4x32_10(_ctr(blk, s, c), (seed & 0xFFFFFFFF, seed >> 32))
        assert [int(v) for v in got] == y


def test_two_formulations_agree():
    rng = np.random.default_rng(7)
    ctr = rng.integers(0, 2**32, size=(300, 4), dtype=np.uint64).astype(np.uint32)
    for key in [(0, 0), (0xFFFFFFFF, 0xFFFFFFFF), (12345, 67890)]:
        vec = philox4x32_10(ctr, key)
        for i in range(ctr.shape[0]):
            assert tuple(int(v) for v in vec[i]) == philox4x32_10_scalar(ctr[i], key)


def test_uniform_layout_eight_elements_per_block():
    seed, c, s = 0xDEADBEEF12345678, 9, 1
    j = luq_uniforms(40, seed, c, s)
    for i in range(40):
        y = philox4x32_10_scalar([i >> 3, 0, s, c], (seed & 0xFFFFFFFF, seed >> 32))
        w = y[(i >> 1) & 3]
        assert int(j[i]) == (w >> (16 * (i & 1))) & 0xFFFF
    # an offset start sees the same stream
    assert np.array_equal(luq_uniforms(17, seed, c, s, start=13), j[13:30])


def test_index_addressed_uniforms_match_scalar_and_ranges():
    """Arbitrary indices (unsorted, repeated, above 2^32) against the scalar
    formulation, and against the contiguous-range generator."""
    seed, c, s = 0x0123456789ABCDEF, 3, 1
    idx = np.array([5, 0, 1 << 33, (1 << 33) + 7, 5, 64, 63, 12345678901], dtype=np.uint64)
    j = luq_uniforms_at(idx, seed, c, s)
    for i, v in zip(idx.tolist(), j.tolist()):
        y = philox4x32_10_scalar([(i >> 3) & 0xFFFFFFFF, i >> 35, s, c], (seed & 0xFFFFFFFF, seed >> 32))
        assert v == (y[(i >> 1) & 3] >> (16 * (i & 1))) & 0xFFFF
    r = luq_uniforms(1000, seed, c, s, start=777)
    assert np.array_equal(luq_uniforms_at(np.arange(777, 1777), seed, c, s), r)


def test_samples_and_counters_are_distinct_streams():
    a = luq_uniforms(4096, 1, 0, 0)
    b = luq_uniforms(4096, 1, 0, 1)
    c = luq_uniforms(4096, 1, 1, 0)
    assert np.mean(a == b) < 0.01 and np.mean(a == c) < 0.01


def test_uniform_chi_square():
    j = luq_uniforms(1 << 20, 42, 0, 0)
    counts = np.bincount((j >> 8).astype(np.int64), minlength=256)
    exp = j.size / 256
    chi2 = ((counts - exp) ** 2 / exp).sum()
    # 255 dof: mean 255, sd ~22.6; 6 sd either side
    assert 120 < chi2 < 390, chi2
    low = np.bincount((j & 0xFF).astype(np.int64), minlength=256)
    chi2l = ((low - exp) ** 2 / exp).sum()
    assert 120 < chi2l < 390, chi2l

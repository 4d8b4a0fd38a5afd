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

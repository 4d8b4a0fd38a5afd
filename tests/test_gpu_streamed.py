"""GPU parity for tensors larger than the 256 MB last-level cache.

Such tensors are streamed: the max pass reads all but their last part with
non-temporal loads, and the encode pass (non-temporal loads and code stores)
walks the tensor from its end.  Every encoder variant that this path selects
is run once at such a size: LUQ row-major and transposed (one sample, two
planes, int8 sums, fp32 and bf16), LUQ with the in-hindsight maximum, and
INT4 signed (both layouts) and unsigned.  Codes are compared with the oracle
on sampled ranges (the first and last elements included) and, for the
transposed layout, against the row-major codes over the whole tensor.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import synth  # noqa: E402
from oracle import luq as oluq, int4 as oint4  # noqa: E402
from oracle.luq import unpack_nibbles, pack_nibbles  # noqa: E402
from gpu_util import announce, to_dev, host, transpose_codes, assert_codes_equal  # noqa: E402

# fp32 [9224, 8192]: 302 MB; rows a multiple of 8 (the transposed layout needs
# it) but not of a tile height
ROWS, COLS = 9224, 8192
# bf16 [16400, 8192]: 269 MB
BROWS = 16400


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2112_10769_amd as lib
    return lib


@pytest.fixture(scope="module")
def g32():
    g = synth.lognormal_grad((ROWS, COLS), -12.0, 2.5, 0.25, [40, 1])
    assert g.nbytes > (256 << 20)
    return g


def _ranges(n, seed, count=16, length=4096):
    rng = np.random.default_rng(seed)
    starts = [0, n - length] + list(rng.integers(0, n - length, size=count))
    return [(int(s), int(s) + length) for s in starts]


def _alpha_checked(alpha, gmax, gf):
    m = np.float32(np.abs(gf).max())
    assert host(gmax)[0].tobytes() == m.tobytes()
    a = np.float32(oluq.luq_alpha(m, 4))
    assert host(alpha)[0].tobytes() == a.tobytes()
    return a


def _check_plane(plane_bytes, gf, a, s, seed, what):
    n = gf.size
    nib = unpack_nibbles(plane_bytes, n)
    for lo, hi in _ranges(n, seed):
        ref = oluq.luq_nibbles_range(gf.ravel()[lo:hi], lo, a, 4, 0, 0, s)
        assert np.array_equal(nib[lo:hi], ref), f"{what}: sample {s} codes [{lo}, {hi})"
    return nib


def test_luq_fp32_both_layouts(L, g32):
    announce("streamed luq fp32 both layouts", g32.shape)
    codes, codes_t, alpha, gmax = L.luq_quantize_grad(to_dev(g32), R=4, codes_t=True)
    a = _alpha_checked(alpha, gmax, g32)
    n = g32.size
    nib = _check_plane(host(codes)[0], g32, a, 0, 1, "fp32")
    tnib = unpack_nibbles(host(codes_t)[0], n).reshape(COLS, ROWS)
    assert np.array_equal(tnib, nib.reshape(ROWS, COLS).T), "fp32 transposed layout"


def test_luq_fp32_two_planes(L, g32):
    announce("streamed luq fp32 two planes", g32.shape)
    codes, _, alpha, gmax = L.luq_quantize_grad(to_dev(g32), R=4, n_samples=2)
    a = _alpha_checked(alpha, gmax, g32)
    c = host(codes)
    for s in range(2):
        _check_plane(c[s], g32, a, s, 2 + s, "fp32 planes")


def test_luq_fp32_int8_sums_both_layouts(L, g32):
    announce("streamed luq fp32 int8 sums", g32.shape)
    codes, codes_t, alpha, gmax = L.luq_quantize_grad(to_dev(g32), R=4, n_samples=L.SMP_SUM | 2, codes_t=True)
    a = _alpha_checked(alpha, gmax, g32)
    n = g32.size
    sums = host(codes).view(np.int8)[:n]
    gf = g32.ravel()
    for lo, hi in _ranges(n, 4):
        planes = np.stack([pack_nibbles(oluq.luq_nibbles_range(gf[lo:hi], lo, a, 4, 0, 0, s)) for s in range(2)])
        assert np.array_equal(sums[lo:hi], oluq.luq_smp_sum(planes, hi - lo)), f"sums [{lo}, {hi})"
    sums_t = host(codes_t).view(np.int8)[:n].reshape(COLS, ROWS)
    assert np.array_equal(sums_t, sums.reshape(ROWS, COLS).T), "sums transposed layout"


def test_luq_bf16_transposed_only(L):
    bits = synth.to_bf16_bits(synth.lognormal_grad((BROWS, COLS), -14.0, 3.0, 0.0, [40, 2]))
    assert bits.nbytes > (256 << 20)
    gf = synth.bf16_bits_to_f32(bits)
    announce("streamed luq bf16 transposed only", bits.shape)
    _, codes_t, alpha, gmax = L.luq_quantize_grad(to_dev(bits), R=4, codes=False, codes_t=True)
    a = _alpha_checked(alpha, gmax, gf)
    n = gf.size
    tnib = unpack_nibbles(host(codes_t)[0], n).reshape(COLS, BROWS)
    # sampled rows of the original layout, read out of the transposed codes
    rows = np.random.default_rng(5).choice(BROWS, 24, replace=False)
    rows = np.concatenate([[0, BROWS - 1], rows])
    for r in rows:
        ref = oluq.luq_nibbles_range(gf[r], int(r) * COLS, a, 4, 0, 0, 0)
        assert np.array_equal(tnib[:, r], ref), f"bf16 row {r}"


def test_luq_hindsight_fp32(L, g32):
    """An estimate above the tensor's maximum: alpha comes from it, and no
    element reaches the top level's clamp."""
    m = np.float32(np.abs(g32).max())
    est = np.float32(1.5) * m
    announce("streamed luq hindsight fp32", g32.shape)
    state = torch.full((1,), float(est), dtype=torch.float32, device="cuda:0")
    codes, _, alpha, gmax = L.luq_quantize_grad_hindsight(to_dev(g32), state, R=4, eta=0.1)
    a = np.float32(oluq.luq_alpha(est, 4))
    assert host(alpha)[0].tobytes() == a.tobytes()
    assert host(gmax)[0].tobytes() == m.tobytes()
    assert host(state)[0].tobytes() == oluq.hindsight_update(m, est, 0.1).tobytes()
    _check_plane(host(codes)[0], g32, a, 0, 6, "hindsight fp32")


def test_int4_fp32_signed_both_layouts_and_unsigned(L):
    x = synth.normal((ROWS, COLS), 1.0, [40, 3])
    announce("streamed int4 fp32 signed both layouts", x.shape)
    xd = to_dev(x)
    codes, codes_t, scale = L.int4_quantize(xd, is_signed=True, codes_t=True)
    ref, s = oint4.int4_quantize(x, is_signed=True)
    assert host(scale)[0].tobytes() == np.float32(s).tobytes()
    assert_codes_equal(host(codes), ref, "int4 signed")
    assert_codes_equal(host(codes_t), transpose_codes(ref, ROWS, COLS), "int4 signed transposed")
    announce("streamed int4 fp32 unsigned", x.shape)
    codes, _, scale = L.int4_quantize(xd, is_signed=False)
    ref, s = oint4.int4_quantize(x, is_signed=False)
    assert host(scale)[0].tobytes() == np.float32(s).tobytes()
    assert_codes_equal(host(codes), ref, "int4 unsigned")

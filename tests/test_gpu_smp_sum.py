"""GPU parity of the summed SMP operand (LUQ_SMP_SUM): two LUQ samples stored
as one int8 sum per element (Section 5.1), through the C ABI.

The quantizers' sums (row-major and transposed, flat and tiled encoders,
fp32 and bf16, R = 4 and 5, exact and in-hindsight maximum) are compared
bit for bit with the oracle's ``luq_smp_sum`` of its two planes; the
backward GEMMs on the summed operand are compared with the oracle's GEMMs
on the planes (within 1e-5 of sum |a_k b_k|, and bit-exact in the fp32
epilogue on the exact integer sums), over every tile configuration.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import synth  # noqa: E402
from oracle import luq as oluq, int4 as oint4, gemm as ogemm  # noqa: E402
from gpu_util import announce, to_dev, host, assert_gemm_close, epilogue_replica  # noqa: E402

SUM2 = 0x12


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2112_10769_amd as lib
    return lib


def _sums(L, x, rows, cols, R=4, seed=0, counter=0, want_t=False, want_rows=True, dtype="f32", what=""):
    announce("smp sum quantize", what, rows, cols, R, dtype)
    xd = to_dev(x)
    gc, gct, alpha, gmax = L.luq_quantize_grad(xd.reshape(rows, cols) if rows > 1 else xd, R=R, seed=seed,
                                              counter=counter, n_samples=SUM2, codes=want_rows, codes_t=want_t)
    planes, ra, rm = oluq.luq_quantize(x, dtype=dtype, R=R, seed=seed, counter=counter, n_samples=2)
    n = rows * cols
    ref = oluq.luq_smp_sum(planes, n)
    assert host(alpha)[0].tobytes() == np.float32(ra).tobytes(), f"{what}: alpha"
    if want_rows:
        got = host(gc).view(np.int8)[:n]
        bad = np.nonzero(got != ref)[0]
        assert bad.size == 0, f"{what}: {bad.size} sums differ, first {bad[:8]}: {got[bad[:8]]} vs {ref[bad[:8]]}"
    if want_t:
        got_t = host(gct).view(np.int8)[:n].reshape(cols, rows)
        assert np.array_equal(got_t, ref.reshape(rows, cols).T), f"{what}: transposed sums"
    return planes, ra


@pytest.mark.parametrize("n", [1, 7, 8, 9, 1001, 65536 + 5, 1 << 20])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_flat_sums(L, n, dtype):
    g = synth.lognormal_grad((n,), -10.0, 3.0, 0.25, [n, 3])
    x = synth.to_bf16_bits(g) if dtype == "bf16" else g
    _sums(L, x, 1, n, dtype=dtype, seed=n, counter=2, what=f"flat {n}")


@pytest.mark.parametrize("shape", [(256, 512), (200, 96), (8, 8), (1024, 64), (64, 4104)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_tile_sums_both_layouts(L, shape, dtype):
    rows, cols = shape
    g = synth.lognormal_grad(shape, -12.0, 2.5, 0.5, [rows, cols])
    x = synth.to_bf16_bits(g) if dtype == "bf16" else g
    _sums(L, x, rows, cols, want_t=True, dtype=dtype, seed=rows + cols, counter=4, what=f"tile {shape}")
    _sums(L, x, rows, cols, want_t=True, want_rows=False, dtype=dtype, seed=rows, counter=1,
          what=f"tile {shape} transposed only")


def test_sums_R5_and_edges(L):
    g = synth.lognormal_grad((96, 64), -8.0, 2.0, 0.1, [5, 5])
    _sums(L, g, 96, 64, R=5, want_t=True, what="R=5")
    z = np.zeros((64, 64), np.float32)
    _sums(L, z, 64, 64, want_t=True, what="all zero")
    one = np.zeros(1000, np.float32)
    one[123] = -3.5
    _sums(L, one, 1, 1000, what="single non-zero")


def test_sums_reject_R6(L):
    g = to_dev(np.ones(64, np.float32))
    with pytest.raises(L.LuqError):
        L.luq_quantize_grad(g, R=6, n_samples=SUM2)


def test_hindsight_sums(L):
    g = synth.lognormal_grad((128, 256), -10.0, 2.0, 0.3, [9, 9])
    m = np.float32(np.abs(g).max()) * np.float32(0.75)     # an estimate below the maximum: clipping
    state = torch.tensor([m], dtype=torch.float32, device="cuda")
    announce("smp sum hindsight")
    gc, gct, alpha, _ = L.luq_quantize_grad_hindsight(to_dev(g), state, R=4, seed=3, counter=8, n_samples=SUM2,
                                                      codes=True, codes_t=True)
    planes, ra, _, m_next = oluq.luq_quantize_hindsight(g, m, R=4, seed=3, counter=8, n_samples=2)
    ref = oluq.luq_smp_sum(planes, g.size)
    assert host(alpha)[0].tobytes() == np.float32(ra).tobytes()
    assert np.array_equal(host(gc).view(np.int8)[:g.size], ref)
    assert np.array_equal(host(gct).view(np.int8)[:g.size].reshape(256, 128), ref.reshape(128, 256).T)
    assert host(state)[0].tobytes() == np.float32(m_next).tobytes()


def _dgrad_sum_case(L, M, N, K, signed, seed):
    g = synth.lognormal_grad((M, K), -10.0, 2.5, 0.3, [seed, 1])
    w = synth.normal((K, N), 0.05, [seed, 2])
    if not signed:
        w = np.abs(w)
    announce("dgrad sum", M, N, K, signed)
    gc, _, alpha, _ = L.luq_quantize_grad(to_dev(g), R=4, seed=seed, counter=1, n_samples=SUM2)
    _, wct, ws = L.int4_quantize(to_dev(w), is_signed=signed, codes=False, codes_t=True)
    dx = host(L.luq_gemm_dgrad(gc, alpha, wct, ws, signed, M, N, K, n_samples=SUM2))
    rc, ra, _ = oluq.luq_quantize(g, R=4, seed=seed, counter=1, n_samples=2)
    wc, wsr = oint4.int4_quantize(w, is_signed=signed)
    ref, absref = ogemm.gemm_dgrad_ref(rc, ra, wc, wsr, signed, M, N, K)
    assert_gemm_close(dx, ref, absref, f"dgrad sum {M}x{N}x{K}")
    A = oluq.luq_smp_sum(rc, M * K).reshape(M, K).astype(np.int64)
    B = oint4.int4_decode_int(wc, K * N, signed).reshape(K, N)
    acc = (A.astype(np.float64) @ B.astype(np.float64)).astype(np.int64)
    assert np.array_equal(dx, epilogue_replica(acc, ra, 2, wsr)), "dgrad sum epilogue not bit-exact"


@pytest.mark.parametrize("M,N,K", [(256, 512, 512), (300, 200, 160), (37, 8, 32), (129, 136, 1056),
                                   (64, 64, 32768), (512, 384, 2048), (1500, 1400, 224), (4192, 4128, 288)])
def test_dgrad_sum_parity(L, M, N, K):
    _dgrad_sum_case(L, M, N, K, True, seed=M + N + K)


def test_dgrad_sum_unsigned_weights(L):
    _dgrad_sum_case(L, 200, 96, 256, False, seed=7)


@pytest.mark.parametrize("T,Nout,Kin", [(256, 512, 512), (96, 40, 24), (4096, 64, 96), (8192, 8, 136),
                                         (160, 1544, 1416), (96, 4104, 4120), (200704 // 4, 64, 576)])
def test_wgrad_sum_parity(L, T, Nout, Kin):
    seed = T + Nout + Kin
    g = synth.lognormal_grad((T, Nout), -12.0, 2.5, 0.5, [seed, 1])
    a = synth.normal((T, Kin), 1.0, [seed, 2])
    announce("wgrad sum", T, Nout, Kin)
    _, gct, alpha, _ = L.luq_quantize_grad(to_dev(g), R=4, seed=seed, counter=3, n_samples=SUM2,
                                           codes=False, codes_t=True)
    _, act, sa = L.int4_quantize(to_dev(a), is_signed=True, codes=False, codes_t=True)
    dw = host(L.luq_gemm_wgrad(gct, alpha, act, sa, True, T, Nout, Kin, n_samples=SUM2))
    rc, ra, _ = oluq.luq_quantize(g, R=4, seed=seed, counter=3, n_samples=2)
    ac, sar = oint4.int4_quantize(a, is_signed=True)
    ref, absref = ogemm.gemm_wgrad_ref(rc, ra, ac, sar, True, T, Nout, Kin)
    assert_gemm_close(dw, ref, absref, f"wgrad sum {T}x{Nout}x{Kin}")
    G = oluq.luq_smp_sum(rc, T * Nout).reshape(T, Nout).astype(np.int64)
    X = oint4.int4_decode_int(ac, T * Kin, True).reshape(T, Kin)
    acc = (G.T.astype(np.float64) @ X.astype(np.float64)).astype(np.int64)
    assert np.array_equal(dw, epilogue_replica(acc, ra, 2, sar)), "wgrad sum epilogue not bit-exact"


def test_sum_gemm_equals_plane_gemm(L):
    """The GEMM on the summed operand and on the two planes give the same bits."""
    M, N, K = 512, 256, 1024
    g = synth.lognormal_grad((M, K), -11.0, 2.0, 0.2, [44, 1])
    w = synth.normal((K, N), 0.05, [44, 2])
    announce("sum vs planes")
    gd = to_dev(g)
    gs, _, alpha, _ = L.luq_quantize_grad(gd, R=4, seed=5, counter=6, n_samples=SUM2)
    gp, _, alpha2, _ = L.luq_quantize_grad(gd, R=4, seed=5, counter=6, n_samples=2)
    _, wct, ws = L.int4_quantize(to_dev(w), is_signed=True, codes=False, codes_t=True)
    a = host(L.luq_gemm_dgrad(gs, alpha, wct, ws, True, M, N, K, n_samples=SUM2))
    b = host(L.luq_gemm_dgrad(gp, alpha2, wct, ws, True, M, N, K, n_samples=2))
    assert np.array_equal(a, b)

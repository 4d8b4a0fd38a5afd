"""GPU parity of the FP6 carrier (LUQ_CARRIER_FP6 on luq_gemm_dgrad and
luq_gemm_wgrad) through the C ABI.

Every output is compared with the oracle -- within 1e-5 of sum_k |a_k b_k|
of the float64 result and bit for bit with the fp32 epilogue applied to the
exact integer sums -- and with the INT8 carrier on the same codes, bit for
bit.  Shapes select both tile sizes (128 and 256), ragged M and N, K not a
multiple of 64 (a zero half block), K below one stage, split reductions for
occupancy and for exactness (K above 16384); codes cover R = 4 and R = 6,
signed and unsigned INT4, and the largest products at the longest unsplit
reduction.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import synth  # noqa: E402
from oracle import luq as oluq, int4 as oint4, gemm as ogemm  # noqa: E402
from gpu_util import announce, to_dev, host, assert_gemm_close, epilogue_replica  # noqa: E402


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2112_10769_amd as lib
    return lib


def _dgrad_fp6_case(L, M, N, K, signed, R=4, seed=0, oracle=True):
    g = synth.lognormal_grad((M, K), -10.0, 2.5, 0.3, [seed, 1])
    w = synth.normal((K, N), 0.05, [seed, 2])
    if not signed:
        w = np.abs(w)
    announce("dgrad fp6", M, N, K, signed, R)
    gc, _, alpha, _ = L.luq_quantize_grad(to_dev(g), R=R, seed=seed, counter=1)
    _, wct, ws = L.int4_quantize(to_dev(w), is_signed=signed, codes=False, codes_t=True)
    dx6 = host(L.luq_gemm_dgrad(gc, alpha, wct, ws, signed, M, N, K, n_samples=L.CARRIER_FP6 | 1))
    dx8 = host(L.luq_gemm_dgrad(gc, alpha, wct, ws, signed, M, N, K, n_samples=1))
    assert np.array_equal(dx6.view(np.uint32), dx8.view(np.uint32)), "FP6 and INT8 carriers differ"
    if not oracle:
        return
    rc, ra, _ = oluq.luq_quantize(g, R=R, seed=seed, counter=1)
    wc, wsr = oint4.int4_quantize(w, is_signed=signed)
    ref, absref = ogemm.gemm_dgrad_ref(rc, ra, wc, wsr, signed, M, N, K)
    assert_gemm_close(dx6, ref, absref, f"fp6 dgrad {M}x{N}x{K}")
    A = oluq.luq_decode_int(rc[0], M * K).reshape(M, K)
    B = oint4.int4_decode_int(wc, K * N, signed).reshape(K, N)
    acc = (A.astype(np.float64) @ B.astype(np.float64)).astype(np.int64)
    assert np.array_equal(dx6, epilogue_replica(acc, ra, 1, wsr)), "fp6 dgrad epilogue not bit-exact"


@pytest.mark.parametrize("M,N,K", [
    (256, 512, 512),      # 128 tiles, one split
    (300, 200, 160),      # ragged M and N; K = 160: a zero half block
    (37, 8, 32),          # K below one 64-deep block
    (129, 136, 1056),     # ragged, split for occupancy
    (64, 64, 32768),      # K above 16384: split for exactness
    (1500, 1400, 224),
    (4100, 4104, 1024),   # 256 tiles with ragged edges
])
def test_fp6_dgrad_parity(L, M, N, K):
    _dgrad_fp6_case(L, M, N, K, True, seed=M + N + K)


@pytest.mark.parametrize("M,N,K", [(200, 96, 256), (4096, 4096, 1088)])
def test_fp6_dgrad_unsigned_weights(L, M, N, K):
    _dgrad_fp6_case(L, M, N, K, False, seed=5 + K)


@pytest.mark.parametrize("signed", [True, False])
def test_fp6_dgrad_R6(L, signed):
    """R = 6: levels up to 2^6 alpha (e3m2 2^4), still exact."""
    _dgrad_fp6_case(L, 512, 256, 2048, signed, R=6, seed=61)


def _wgrad_fp6_case(L, T, Nout, Kin, signed, seed):
    g = synth.lognormal_grad((T, Nout), -12.0, 2.5, 0.5, [seed, 1])
    a = synth.normal((T, Kin), 1.0, [seed, 2]) if signed else synth.half_normal((T, Kin), [seed, 2])
    announce("wgrad fp6", T, Nout, Kin, signed)
    _, gct, alpha, _ = L.luq_quantize_grad(to_dev(g), R=4, seed=seed, counter=3, codes=False, codes_t=True)
    _, act, sa = L.int4_quantize(to_dev(a), is_signed=signed, codes=False, codes_t=True)
    dw6 = host(L.luq_gemm_wgrad(gct, alpha, act, sa, signed, T, Nout, Kin, n_samples=L.CARRIER_FP6 | 1))
    dw8 = host(L.luq_gemm_wgrad(gct, alpha, act, sa, signed, T, Nout, Kin, n_samples=1))
    assert np.array_equal(dw6.view(np.uint32), dw8.view(np.uint32)), "FP6 and INT8 carriers differ"
    rc, ra, _ = oluq.luq_quantize(g, R=4, seed=seed, counter=3)
    ac, sar = oint4.int4_quantize(a, is_signed=signed)
    ref, absref = ogemm.gemm_wgrad_ref(rc, ra, ac, sar, signed, T, Nout, Kin)
    assert_gemm_close(dw6, ref, absref, f"fp6 wgrad {T}x{Nout}x{Kin}")
    G = oluq.luq_decode_int(rc[0], T * Nout).reshape(T, Nout)
    X = oint4.int4_decode_int(ac, T * Kin, signed).reshape(T, Kin)
    acc = (G.T.astype(np.float64) @ X.astype(np.float64)).astype(np.int64)
    assert np.array_equal(dw6, epilogue_replica(acc, ra, 1, sar)), "fp6 wgrad epilogue not bit-exact"


@pytest.mark.parametrize("T,Nout,Kin,signed", [(256, 512, 512, False), (96, 40, 24, False),
                                                (4096, 64, 96, True), (66560, 64, 576, False),
                                                (160, 1544, 1416, False)])
def test_fp6_wgrad_parity(L, T, Nout, Kin, signed):
    _wgrad_fp6_case(L, T, Nout, Kin, signed, seed=T + Nout)


@pytest.mark.parametrize("K", [16384, 16384 + 64])
@pytest.mark.parametrize("signed", [True, False])
def test_fp6_largest_products(L, K, signed):
    """Every product at its largest -- the LUQ top code of R = 6 (2^6) times
    INT4 7 (signed) or 15 (unsigned) -- at the longest unsplit reduction and
    one block past it (split): the sums equal the INT8 carrier's and the
    closed form K * 2^6 * qmax in value units."""
    M, N = 512, 512
    announce("fp6 largest products", K, signed)
    byte_g = 0x77  # field 7, sign +: 2^6 (R = 6)
    byte_w = 0x77 if signed else 0xFF
    gc = torch.full((M * K // 2,), byte_g, dtype=torch.uint8, device="cuda:0")
    wct = torch.full((N * K // 2,), byte_w, dtype=torch.uint8, device="cuda:0")
    alpha = torch.tensor([2.0 ** -6], dtype=torch.float32, device="cuda:0")
    s = torch.tensor([1.0 / (7 if signed else 15)], dtype=torch.float32, device="cuda:0")
    dx6 = host(L.luq_gemm_dgrad(gc, alpha, wct, s, signed, M, N, K, n_samples=L.CARRIER_FP6 | 1))
    dx8 = host(L.luq_gemm_dgrad(gc, alpha, wct, s, signed, M, N, K, n_samples=1))
    assert np.array_equal(dx6.view(np.uint32), dx8.view(np.uint32))
    q = 7 if signed else 15
    want = epilogue_replica(np.full((1,), K * 64 * q, np.int64), np.float32(2.0 ** -6), 1, host(s)[0])[0]
    assert np.all(dx6 == want), (np.unique(dx6)[:4], want)


def test_fp6_rejects_two_samples(L):
    announce("fp6 two samples rejected")
    gc = torch.zeros(2 * 256, dtype=torch.uint8, device="cuda:0")
    one = torch.ones(1, dtype=torch.float32, device="cuda:0")
    with pytest.raises(L.LuqError) as e:
        L.luq_gemm_dgrad(gc, one, gc, one, True, 8, 8, 64, n_samples=L.CARRIER_FP6 | 2)
    assert e.value.status == 4

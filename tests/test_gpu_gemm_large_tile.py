"""GPU parity of the 256 x 256 GEMM tile (eight waves, the INT4 operand read
straight into registers) through the C ABI.

Shapes are chosen so that the planner picks that tile (at least 256 output
tiles and K >= 1024): ragged M and N, K a multiple of 128 (whole stages) and
not (a half-filled last stage), every A operand kind (LUQ, two SMP planes,
the int8 SMP sums, signed and unsigned INT4) and both INT4 signednesses of
B.  Outputs are compared with the oracle within 1e-5 of sum |a b| and bit
for bit with the fp32 epilogue applied to the exact integer sums.  The
largest codes at the longest unsplit reduction (K = 2^18) and one stage past
it (a split reduction) check the int32 bound and the sign handling against
the closed form.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import synth  # noqa: E402
from test_gpu_parity import _gemm_case, _wgrad_case, _fwd_case  # noqa: E402
from test_gpu_smp_sum import _dgrad_sum_case  # noqa: E402
from gpu_util import announce, host, epilogue_replica  # noqa: E402


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2112_10769_amd as lib
    return lib


@pytest.mark.parametrize("ns", [1, 2])
def test_large_tile_dgrad_ragged(L, ns):
    _gemm_case(L, 4100, 4104, 1056, ns, True, seed=17 + ns)


def test_large_tile_dgrad_whole_stages_unsigned(L):
    _gemm_case(L, 4096, 4096, 1024, 1, False, seed=23)


def test_large_tile_dgrad_smp_sum(L):
    _dgrad_sum_case(L, 4100, 4104, 1056, True, seed=29)


@pytest.mark.parametrize("signed", [False, True])
def test_large_tile_wgrad(L, signed):
    _wgrad_case(L, 1056, 4104, 4120, 1, signed=signed, seed=31)


@pytest.mark.parametrize("xsig,wsig", [(True, True), (False, True), (True, False), (False, False)])
def test_large_tile_fwd(L, xsig, wsig):
    _fwd_case(L, 4100, 4104, 1056, xsig, wsig, seed=37)


@pytest.mark.parametrize("K", [1 << 18, (1 << 18) + 128])
@pytest.mark.parametrize("signed", [True, False])
@pytest.mark.parametrize("neg", [False, True])
def test_large_tile_largest_products(L, K, signed, neg):
    """Every A code the top LUQ level of R = 6 (2^6, either sign) and every B
    code the largest INT4 (7 signed, 15 unsigned): each output is K * 2^6 * q
    in value units (its int32 carrier sum is at most 2^18 * 64 * 120 < 2^31)."""
    M = N = 4096
    announce("large tile largest products", K, signed, neg)
    byte_g = 0xFF if neg else 0x77   # field 7 with the sign bit set / clear
    byte_w = 0x77 if signed else 0xFF
    gc = torch.full((M * K // 2,), byte_g, dtype=torch.uint8, device="cuda:0")
    wct = torch.full((N * K // 2,), byte_w, dtype=torch.uint8, device="cuda:0")
    alpha = torch.tensor([2.0 ** -6], dtype=torch.float32, device="cuda:0")
    q = 7 if signed else 15
    s = torch.tensor([1.0 / q], dtype=torch.float32, device="cuda:0")
    dx = host(L.luq_gemm_dgrad(gc, alpha, wct, s, signed, M, N, K))
    del gc, wct
    acc = np.full((1,), (-1 if neg else 1) * K * 64 * q, np.int64)
    want = epilogue_replica(acc, np.float32(2.0 ** -6), 1, host(s)[0])[0]
    assert np.all(dx == want), (np.unique(dx)[:4], want)

"""GPU tests of luq_query_status: the data status (Eq. alpha and the INT4
scale of Appendix A.1 exist only for a finite maximum) that every quantizer
call leaves in its workspace, read back through the C ABI.

Finite tensors report LUQ_OK, tensors with a NaN or infinite element
LUQ_ERR_NONFINITE, for LUQ (flat and tiled encoders, fp32 and bf16, one
and two samples), the in-hindsight LUQ (non-finite elements and
non-finite estimates; an overflowed step leaves the estimate unchanged)
and INT4 (signed, unsigned, the small-tensor path, clip); empty tensors
report LUQ_OK; a workspace no quantizer wrote is refused.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import synth  # noqa: E402
from gpu_util import announce, to_dev, host  # noqa: E402


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2112_10769_amd as lib
    return lib


def _ws(L, n):
    return torch.zeros(L.workspace_size(L.OP_QUANTIZE_GRAD, n), dtype=torch.uint8, device="cuda:0")


def _poison(x, kind, at):
    y = x.copy()
    if y.dtype == np.uint16:  # bf16 bit patterns
        y[at] = {"inf": 0x7F80, "-inf": 0xFF80, "nan": 0x7FC0}[kind]
    else:
        y[at] = {"inf": np.inf, "-inf": -np.inf, "nan": np.nan}[kind]
    return y


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape,tiled", [((1, 70001), False), ((512, 1024), True), ((4104, 64), True)])
@pytest.mark.parametrize("ns", [1, 2])
def test_luq_status(L, dtype, shape, tiled, ns):
    r, c = shape
    n = r * c
    x = synth.grad_1d(n, dtype, 0.2, seed=n % 101)
    ws = _ws(L, n)
    for kind in (None, "inf", "-inf", "nan"):
        y = x if kind is None else _poison(x, kind, n // 3)
        announce("luq status", dtype, shape, ns, kind)
        xd = to_dev(y.reshape(r, c) if r > 1 else y)
        _, _, alpha, _ = L.luq_quantize_grad(xd, R=4 if ns == 1 else 5, n_samples=ns, codes=True, codes_t=tiled,
                                             ws=ws)
        st = L.query_status(ws)
        if kind is None:
            assert st == L.LUQ_OK and np.isfinite(host(alpha)[0])
        else:
            assert st == L.LUQ_ERR_NONFINITE and np.isnan(host(alpha)[0])


def test_luq_status_smp_sum_and_empty(L):
    x = synth.grad_1d(1 << 16, "f32", 0.2, seed=3)
    ws = _ws(L, x.size)
    announce("luq status smp sum")
    L.luq_quantize_grad(to_dev(_poison(x, "nan", 5).reshape(256, 256)), R=4, n_samples=L.SMP_SUM | 2,
                        codes=True, codes_t=True, ws=ws)
    assert L.query_status(ws) == L.LUQ_ERR_NONFINITE
    announce("luq status empty")
    L.luq_quantize_grad(torch.zeros(0, dtype=torch.float32, device="cuda:0"), ws=ws)
    assert L.query_status(ws) == L.LUQ_OK


@pytest.mark.parametrize("n", [4096, 300001])
def test_hindsight_status_and_overflow_step(L, n):
    x = synth.grad_1d(n, "f32", 0.2, seed=7)
    m = float(np.abs(x).max())
    ws = _ws(L, n)
    state = torch.tensor([m], dtype=torch.float32, device="cuda:0")
    announce("hindsight status finite", n)
    L.luq_quantize_grad_hindsight(to_dev(x), state, ws=ws)
    assert L.query_status(ws) == L.LUQ_OK
    before = host(state)[0]
    announce("hindsight status overflow step", n)
    _, _, alpha, maxabs = L.luq_quantize_grad_hindsight(to_dev(_poison(x, "inf", 11)), state, ws=ws)
    assert L.query_status(ws) == L.LUQ_ERR_NONFINITE
    assert host(maxabs)[0] == np.inf and np.isfinite(host(alpha)[0])
    assert host(state)[0].tobytes() == before.tobytes(), "an overflowed step changed the estimate"
    announce("hindsight status after the overflow", n)
    L.luq_quantize_grad_hindsight(to_dev(x), state, ws=ws)
    assert L.query_status(ws) == L.LUQ_OK and np.isfinite(host(state)[0])
    for bad in (np.nan, np.inf):
        announce("hindsight status estimate", bad)
        st = torch.tensor([bad], dtype=torch.float32, device="cuda:0")
        L.luq_quantize_grad_hindsight(to_dev(x), st, ws=ws)
        assert L.query_status(ws) == L.LUQ_ERR_NONFINITE


@pytest.mark.parametrize("n", [1000, 1 << 16, (1 << 16) + 8, 1 << 20])
@pytest.mark.parametrize("signed", [True, False])
@pytest.mark.parametrize("tiled", [False, True])
def test_int4_status(L, n, signed, tiled):
    rows = 8 if tiled else 1
    if tiled and n % 64:
        n = (n + 63) // 64 * 64
    x = synth.normal((n,), 1.0, [n, 1])
    ws = _ws(L, n)
    for kind in (None, "nan", "-inf"):
        y = x if kind is None else _poison(x, kind, n // 2)
        announce("int4 status", n, signed, tiled, kind)
        xd = to_dev(y.reshape(rows, -1) if rows > 1 else y)
        _, _, sc = L.int4_quantize(xd, is_signed=signed, codes=True, codes_t=tiled, ws=ws)
        st = L.query_status(ws)
        assert st == (L.LUQ_OK if kind is None else L.LUQ_ERR_NONFINITE), (kind, st)
    announce("int4 status clip", n)
    L.int4_quantize(to_dev(_poison(x, "nan", 3)), is_signed=signed, clip=2.0, ws=ws)
    assert L.query_status(ws) == L.LUQ_OK


def test_status_of_an_unwritten_workspace_is_refused(L):
    announce("status of a zeroed workspace")
    ws = _ws(L, 1)
    with pytest.raises(L.LuqError) as e:
        L.query_status(ws)
    assert e.value.status == 5

"""GPU test of luq_quantize_grad_noalloc, the allocation-free LUQ entry point
(its workspace is the library's static per-device scratch array), through
the C ABI: its codes, alpha and maxabs must equal luq_quantize_grad's (with
a caller workspace) bit for bit, on calls in a row that share the scratch --
a large tensor whose partial maxima take the folded path first, then
smaller ones -- over the flat and transposing encoders, fp32 and bf16, one
and two samples, the int8 sums and the power-of-two alpha.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from gpu_util import announce, host  # noqa: E402


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2112_10769_amd as lib
    return lib


def _grad(shape, dtype, seed):
    """Lognormal-magnitude gradient drawn on the device (inputs only)."""
    gen = torch.Generator(device="cuda:0")
    gen.manual_seed(seed)
    n = int(np.prod(shape))
    g = torch.randn(n, generator=gen, device="cuda:0").mul_(3.0).sub_(10.0).exp_()
    g[torch.rand(n, generator=gen, device="cuda:0") < 0.5] *= -1.0
    g[torch.rand(n, generator=gen, device="cuda:0") < 0.25] = 0.0
    g = g.view(*shape)
    return g if dtype == "f32" else g.to(torch.bfloat16)


def _outputs(L, n, ns, want_t):
    summed = bool(ns & L.SMP_SUM)
    nbytes = n if summed else (ns & 0xF) * L.plane_bytes(n)
    mk = lambda: torch.full((max(nbytes, 1),), 0xA5, dtype=torch.uint8, device="cuda:0")
    return mk(), (mk() if want_t else None), torch.full((1,), -1.0, device="cuda:0"), torch.full((1,), -1.0, device="cuda:0")


def _compare(L, g, ns=1, want_t=False, R=4, pw2=False, seed=11, counter=3, what=""):
    n = g.numel()
    announce("noalloc", what, tuple(g.shape), g.dtype, ns, want_t, R, pw2)
    c0, t0, a0, m0 = _outputs(L, n, ns, want_t)
    L.luq_quantize_grad(g, R=R, seed=seed, counter=counter, n_samples=ns, codes=c0,
                        codes_t=t0 if want_t else False, alpha=a0, maxabs=m0, pw2=pw2)
    c1, t1, a1, m1 = _outputs(L, n, ns, want_t)
    L.luq_quantize_grad_noalloc(g, c1, t1, a1, m1, R=R, seed=seed, counter=counter, n_samples=ns, pw2=pw2)
    torch.cuda.synchronize()
    assert host(a1).tobytes() == host(a0).tobytes(), (what, host(a1), host(a0))
    assert host(m1).tobytes() == host(m0).tobytes(), (what, host(m1), host(m0))
    assert torch.equal(c1, c0), f"{what}: codes differ"
    if want_t:
        assert torch.equal(t1, t0), f"{what}: transposed codes differ"


def test_noalloc_matches_the_workspace_entry_point_on_calls_in_a_row(L):
    # a streamed tensor with more than 2048 partial maxima (the folded path),
    # then smaller tensors that reuse the scratch it left behind
    _compare(L, _grad((1 << 27,), "f32", 1), what="2^27 fp32 flat")
    _compare(L, _grad((8192, 4096), "bf16", 2), want_t=True, what="8192x4096 bf16 both layouts")
    _compare(L, _grad((1000003 * 2,), "f32", 3), what="ragged flat")
    _compare(L, _grad((264, 200), "f32", 4), ns=2, R=5, want_t=True, what="two planes")
    _compare(L, _grad((512, 1024), "bf16", 5), ns=L.SMP_SUM | 2, want_t=True, what="int8 sums")
    _compare(L, _grad((4104, 64), "f32", 6), want_t=True, pw2=True, what="power-of-two alpha, narrow")
    _compare(L, _grad((7,), "f32", 7), what="seven elements")


def test_noalloc_second_call_with_a_smaller_input(L):
    """Two calls in a row, the second on a smaller tensor: the second call's
    results must not depend on what the first left in the scratch."""
    _compare(L, _grad((4096, 4096), "f32", 8), want_t=True, R=6, what="first, 4096x4096")
    _compare(L, _grad((256, 512), "f32", 9), want_t=True, R=6, what="second, 256x512")


def test_noalloc_nonfinite_and_empty(L):
    g = _grad((70001 * 2,), "f32", 10)
    g[12345] = float("nan")
    _compare(L, g, what="nan element")
    announce("noalloc empty")
    alpha = torch.full((1,), 5.0, device="cuda:0")
    maxabs = torch.full((1,), 5.0, device="cuda:0")
    L.luq_quantize_grad_noalloc(torch.zeros(0, device="cuda:0"), None, None, alpha, maxabs)
    assert host(alpha)[0] == 0 and host(maxabs)[0] == 0

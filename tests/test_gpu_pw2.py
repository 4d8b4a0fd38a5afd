"""GPU parity of power-of-two LUQ (the LUQ_ALPHA_PW2 flag) against the
oracle: codes, alpha and the maximum bit-exact over ragged and tiled shapes,
both dtypes, one and two SMP planes, R = 4..6, power-of-two, subnormal,
tiny and near-overflow maxima, and with the in-hindsight maximum.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import synth  # noqa: E402
from oracle import luq as oluq  # noqa: E402
from gpu_util import announce, to_dev, host, transpose_codes, assert_codes_equal  # noqa: E402


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2112_10769_amd as lib
    return lib


def _same(a, b):
    a, b = np.float32(a), np.float32(b)
    return (np.isnan(a) and np.isnan(b)) or a.tobytes() == b.tobytes()


def _check(L, x, rows, cols, R=4, seed=0, counter=0, ns=1, want_t=False, what=""):
    dt = "bf16" if x.dtype == np.uint16 else "f32"
    announce("pw2", what, rows, cols, dt, R, ns, want_t)
    xd = to_dev(x.reshape(rows, cols) if rows > 1 else x.reshape(-1))
    codes, codes_t, alpha, maxabs = L.luq_quantize_grad(xd, R=R, seed=seed, counter=counter, n_samples=ns,
                                                        codes=True, codes_t=want_t, pw2=True)
    rc, ra, rm = oluq.luq_quantize(x.ravel(), dtype=dt, R=R, seed=seed, counter=counter, n_samples=ns, pw2=True)
    assert _same(host(alpha)[0], ra), (host(alpha)[0], ra)
    assert _same(host(maxabs)[0], rm)
    nb = (rows * cols + 1) // 2
    hc = host(codes).reshape(ns, -1)
    for s in range(ns):
        assert_codes_equal(hc[s, :nb], rc[s], f"{what} plane {s}")
    if want_t:
        ht = host(codes_t).reshape(ns, -1)
        for s in range(ns):
            assert_codes_equal(ht[s, :nb], transpose_codes(rc[s], rows, cols), f"{what} transposed plane {s}")
    return ra


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n", [1, 7, 1001, 65537, (1 << 20) + 3])
def test_pw2_flat(L, n, dtype):
    x = synth.grad_1d(n, dtype, 0.3, seed=300 + n % 89)
    _check(L, x, 1, n, seed=n, counter=2, what="flat")


@pytest.mark.parametrize("shape", [(264, 200), (4104, 64), (1024, 392)])
@pytest.mark.parametrize("ns,R", [(1, 4), (2, 5), (1, 6)])
def test_pw2_tiles(L, shape, ns, R):
    r, c = shape
    x = synth.lognormal_grad((r, c), -10.0, 2.5, 0.3, [r, c, 7])
    _check(L, x, r, c, R=R, seed=r, counter=c, ns=ns, want_t=True, what="tile")


@pytest.mark.parametrize("top", [2.0 ** -7, 3.0e-3, 1e-30, 2.0 ** -126, 3.3e38, 2.0 ** 127])
def test_pw2_special_maxima(L, top):
    x = synth.grad_1d(70001, "f32", 0.2, seed=41)
    x = (x / np.abs(x).max()).astype(np.float32)
    x = (x.astype(np.float64) * top).astype(np.float32)
    ra = _check(L, x, 1, x.size, seed=3, what=f"max {top}")
    if top == 2.0 ** -7:   # a power-of-two maximum gives the plain alpha
        assert ra == oluq.luq_alpha(np.float32(np.abs(x).max()), 4)


def test_pw2_subnormal_and_zero_maxima(L):
    for vals in ([1e-40, -3e-41, 0.0, 7e-42] * 300, [0.0] * 64, [1.4e-45, 0.0] * 40):
        x = np.array(vals, np.float32)
        _check(L, x, 1, x.size, what=f"max {np.abs(x).max()}")


@pytest.mark.parametrize("frac", [0.3, 1.0, 1.6])
def test_pw2_hindsight(L, frac):
    x = synth.grad_1d(81920, "f32", 0.25, seed=42)
    m_hat = np.float32(np.abs(x).max() * frac)
    announce("pw2 hindsight", frac)
    state = torch.tensor([float(m_hat)], dtype=torch.float32, device="cuda:0")
    codes, _, alpha, maxabs = L.luq_quantize_grad_hindsight(to_dev(x), state, R=4, seed=6, counter=1, pw2=True)
    rc, ra, rm, rn = oluq.luq_quantize_hindsight(x, m_hat, R=4, seed=6, counter=1, pw2=True)
    assert _same(host(alpha)[0], ra) and _same(host(maxabs)[0], rm) and _same(host(state)[0], rn)
    assert_codes_equal(host(codes)[0, : rc.shape[1]], rc[0], f"hindsight pw2 x{frac}")

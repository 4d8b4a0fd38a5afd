"""GPU parity of the single-pass LUQ with the in-hindsight maximum
(luq_quantize_grad_hindsight) against the oracle: codes, alpha, the measured
maximum and the updated estimate bit-exact, over ragged and tiled shapes,
both dtypes, one and two SMP planes, estimates below, at and above the
tensor's maximum, degenerate estimates and non-finite elements (fp32 and bf16).
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


def _same_float(a, b):
    a, b = np.float32(a), np.float32(b)
    return (np.isnan(a) and np.isnan(b)) or a.tobytes() == b.tobytes()


def _check(L, x, rows, cols, m_hat, R=4, seed=0, counter=0, ns=1, eta=0.1, want_t=False, what=""):
    dt = "bf16" if x.dtype == np.uint16 else "f32"
    announce("hindsight", what, rows, cols, dt, float(m_hat), R, ns, eta, want_t)
    xd = to_dev(x.reshape(rows, cols) if rows > 1 else x.reshape(-1))
    state = torch.tensor([float(np.float32(m_hat))], dtype=torch.float32, device="cuda:0")
    codes, codes_t, alpha, maxabs = L.luq_quantize_grad_hindsight(
        xd, state, R=R, seed=seed, counter=counter, n_samples=ns, eta=eta, codes=True, codes_t=want_t)
    rc, ra, rm, rnext = oluq.luq_quantize_hindsight(x.ravel(), m_hat, dtype=dt, R=R, seed=seed, counter=counter,
                                                    n_samples=ns, eta=eta)
    assert _same_float(host(alpha)[0], ra), (host(alpha)[0], ra)
    assert _same_float(host(maxabs)[0], rm), (host(maxabs)[0], rm)
    assert _same_float(host(state)[0], rnext), (host(state)[0], rnext)
    n = rows * cols
    nb = (n + 1) // 2
    hc = host(codes).reshape(ns, -1)
    for s in range(ns):
        assert_codes_equal(hc[s, :nb], rc[s], f"{what} plane {s}")
    if want_t:
        ht = host(codes_t).reshape(ns, -1)
        for s in range(ns):
            assert_codes_equal(ht[s, :nb], transpose_codes(rc[s], rows, cols), f"{what} transposed plane {s}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n", [1, 7, 1001, 65537, (1 << 20) + 3])
@pytest.mark.parametrize("frac", [0.5, 1.0, 2.0])
def test_hindsight_flat(L, n, dtype, frac):
    x = synth.grad_1d(n, dtype, 0.25, seed=n % 97)
    xf = synth.bf16_bits_to_f32(x) if dtype == "bf16" else x
    m_hat = np.float32(np.abs(xf).max() * frac)
    _check(L, x, 1, n, m_hat, seed=n, counter=3, what=f"flat x{frac}")


@pytest.mark.parametrize("shape", [(264, 200), (4104, 64), (1024, 392), (8, 8)])
@pytest.mark.parametrize("ns", [1, 2])
def test_hindsight_tiles(L, shape, ns):
    r, c = shape
    x = synth.lognormal_grad((r, c), -10.0, 2.5, 0.3, [r, c])
    m_hat = np.float32(np.abs(x).max() * 0.7)
    _check(L, x, r, c, m_hat, R=5 if ns == 2 else 4, seed=r + c, counter=1, ns=ns, want_t=True, what="tile")


@pytest.mark.parametrize("shape", [(264, 200), (1024, 392)])
@pytest.mark.parametrize("ns", [1, 2])
@pytest.mark.parametrize("frac", [0.3, 1.0])
def test_hindsight_tiles_bf16(L, shape, ns, frac):
    """bf16 tiles (the packed 16-bit encoder with the top field capped): an
    estimate at 0.3 of the maximum clips every element above its top level."""
    r, c = shape
    x = synth.to_bf16_bits(synth.lognormal_grad((r, c), -10.0, 2.5, 0.3, [r, c, 7]))
    m_hat = np.float32(np.abs(synth.bf16_bits_to_f32(x)).max() * frac)
    _check(L, x, r, c, m_hat, R=5 if ns == 2 else 4, seed=r + c, counter=2, ns=ns, want_t=True,
           what=f"bf16 tile x{frac}")


@pytest.mark.parametrize("R", [4, 5, 6])
def test_hindsight_R_and_eta(L, R):
    x = synth.grad_1d(70001, "f32", 0.1, seed=R)
    _check(L, x, 1, x.size, np.float32(np.abs(x).max() * 0.9), R=R, eta=0.25, what=f"R={R}")


@pytest.mark.parametrize("m_hat", [0.0, -1.0, np.nan, np.inf, 1e-30, 3e38])
@pytest.mark.parametrize("n", [4096, 81920])
def test_hindsight_degenerate_estimates(L, m_hat, n):
    x = synth.grad_1d(n, "f32", 0.2, seed=8)
    _check(L, x, 1, n, np.float32(m_hat), seed=5, what=f"estimate {m_hat}")


def test_hindsight_nonfinite_elements(L):
    x = synth.grad_1d(70000, "f32", 0.2, seed=12)
    y = x.copy()
    y[123] = np.inf
    y[4567] = -np.inf
    _check(L, y, 1, y.size, np.float32(np.abs(x).max()), what="inf elements")
    y[999] = np.nan
    _check(L, y, 1, y.size, np.float32(np.abs(x).max()), what="nan element")


@pytest.mark.parametrize("R", [4, 6])
def test_hindsight_nonfinite_elements_bf16(L, R):
    """bf16 Inf, -Inf and NaN elements under an estimate: clipped to the top
    code with their sign, like every element above the top level."""
    x = synth.grad_1d(70000, "bf16", 0.2, seed=13)
    m_hat = np.float32(np.abs(synth.bf16_bits_to_f32(x)).max() * 0.5)
    y = x.copy()
    y[123], y[4567], y[999], y[1001] = 0x7F80, 0xFF80, 0x7FC0, 0xFFC1  # +Inf, -Inf, NaN, -NaN
    _check(L, y, 1, y.size, m_hat, R=R, what=f"bf16 non-finite R={R}")


def test_hindsight_empty_and_sequence(L):
    announce("hindsight empty")
    state = torch.tensor([2.0], dtype=torch.float32, device="cuda:0")
    x = torch.zeros(0, dtype=torch.float32, device="cuda:0")
    _, _, alpha, maxabs = L.luq_quantize_grad_hindsight(x, state)
    assert host(alpha)[0] == np.float32(0.125) and host(maxabs)[0] == 0
    assert host(state)[0] == oluq.hindsight_update(np.float32(0.0), np.float32(2.0), 0.1)
    # three steps carrying the estimate on the device
    announce("hindsight sequence")
    state = torch.tensor([1e-3], dtype=torch.float32, device="cuda:0")
    m = np.float32(1e-3)
    for t in range(3):
        x = synth.grad_1d(50000, "f32", 0.3, seed=200 + t)
        codes, _, alpha, _ = L.luq_quantize_grad_hindsight(to_dev(x), state, seed=1, counter=t)
        rc, ra, _, m = oluq.luq_quantize_hindsight(x, m, seed=1, counter=t)
        assert_codes_equal(host(codes)[0, : rc.shape[1]], rc[0], f"step {t}")
        assert _same_float(host(state)[0], m)

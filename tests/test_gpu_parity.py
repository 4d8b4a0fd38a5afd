"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Quantizer codes, alpha, maxabs and scales must be bit-exact; GEMM outputs
must lie within 1e-5 of sum_k |a_k b_k| of the exact float64 result and, in
addition, equal the fp32 epilogue applied to the exact integer sums.
Sizes span several tiles and ragged tails; edge cases cover empty, zero,
subnormal, huge and non-finite inputs.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import synth  # noqa: E402
from oracle import luq as oluq, int4 as oint4, gemm as ogemm, im2col as oim2col  # noqa: E402
from oracle.luq import unpack_nibbles  # noqa: E402
from gpu_util import (announce, to_dev, host, transpose_codes, assert_codes_equal,  # noqa: E402
                      assert_gemm_close, epilogue_replica)


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2112_10769_amd as lib
    return lib


def _dt(x):
    return "bf16" if x.dtype == np.uint16 else "f32"


def _check_luq(L, x, rows, cols, R=4, seed=0, counter=0, ns=1, want_t=False, want_rows=True, what=""):
    announce("luq", what, rows, cols, _dt(x), R, seed, counter, ns, want_t)
    xd = to_dev(x.reshape(rows, cols) if rows > 1 else x.reshape(-1))
    codes, codes_t, alpha, maxabs = L.luq_quantize_grad(xd, R=R, seed=seed, counter=counter, n_samples=ns,
                                                        codes=want_rows, codes_t=want_t)
    rc, ra, rm = oluq.luq_quantize(x.ravel(), dtype=_dt(x), R=R, seed=seed, counter=counter, n_samples=ns)
    a = host(alpha)[0]
    m = host(maxabs)[0]
    if np.isnan(ra):
        assert np.isnan(a)
    else:
        assert a.tobytes() == np.float32(ra).tobytes(), (a, ra)
    if np.isnan(rm):
        assert np.isnan(m)
    else:
        assert m.tobytes() == np.float32(rm).tobytes(), (m, rm)
    n = rows * cols
    nb = (n + 1) // 2
    if want_rows:
        hc = host(codes).reshape(ns, -1)
        for s in range(ns):
            assert_codes_equal(hc[s, :nb], rc[s], f"{what} plane {s}")
    if want_t:
        ht = host(codes_t).reshape(ns, -1)
        for s in range(ns):
            assert_codes_equal(ht[s, :nb], transpose_codes(rc[s], rows, cols), f"{what} transposed plane {s}")
    return rc, ra


@pytest.mark.parametrize("ns", [1, 2])
def test_luq_small_layer(L, ns):
    d = synth.small()
    _check_luq(L, d["g"], 256, 512, ns=ns, want_t=True, what="small layer")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n", [1, 2, 7, 8, 9, 15, 1001, 65537, (1 << 20) + 3])
def test_luq_flat_ragged(L, n, dtype):
    x = synth.grad_1d(n, dtype=dtype, zero_frac=0.3, seed=100 + n % 97)
    _check_luq(L, x, 1, n, seed=0xDEADBEEFCAFE0000 + n, counter=n, what="flat")


# includes narrow matrices whose transposing tiles shrink below 8192 words
@pytest.mark.parametrize("shape", [(8, 8), (264, 200), (136, 1032), (1024, 392), (40, 4096), (4104, 64),
                                   (2056, 16), (1000, 8)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_luq_tile_both_layouts(L, shape, dtype):
    r, c = shape
    x = synth.grad_1d(r * c, dtype=dtype, zero_frac=0.2, seed=200 + r)
    _check_luq(L, x, r, c, ns=2, seed=r * c, counter=7, want_t=True, what="tile")
    _check_luq(L, x, r, c, ns=1, seed=3, counter=1, want_t=True, want_rows=False, what="tile t-only")


@pytest.mark.parametrize("R", [5, 6])
def test_luq_other_R(L, R):
    x = synth.grad_1d(50003, seed=31, sigma=3.0)
    _check_luq(L, x, 1, x.size, R=R, seed=R, what=f"R={R}")
    if R == 5:
        _check_luq(L, x, 1, x.size, R=R, ns=2, what="R=5 smp")


def _edge_cases():
    rng = np.random.default_rng(5)
    base = synth.grad_1d(4096, seed=41)
    cases = {}
    cases["zeros"] = np.zeros(1000, np.float32)
    z = np.zeros(999, np.float32)
    z[500] = -3.5
    cases["single nonzero"] = z
    cases["tiny max (prescaled path)"] = (base * np.float32(2.0 ** -120)).astype(np.float32)
    cases["subnormal max"] = (base / np.abs(base).max() * np.float32(1e-39)).astype(np.float32)
    cases["max underflows alpha"] = np.array([1e-45, -1e-45, 0, 1e-45] * 4, np.float32)
    cases["huge max"] = (base / np.abs(base).max() * np.float32(3.0e38)).astype(np.float32)
    lv = np.array([16.0, 1.0, 2.0, 4.0, 8.0, -16.0, -1.0, 0.5, 0.25] * 100, np.float32)
    cases["on levels"] = lv
    inf = base.copy()
    inf[77] = np.inf
    cases["inf"] = inf
    nan = base.copy()
    nan[3] = np.nan
    cases["nan"] = nan
    neg0 = np.array([-0.0, 0.0, -0.0, 1.0] * 8, np.float32)
    cases["negative zero"] = neg0
    cases["all equal"] = np.full(777, -0.125, np.float32)
    cases["uniform mantissas"] = (rng.random(100000).astype(np.float32) * 2 - 1)
    return cases


def _big(x, at_least=70000, multiple=64):
    """x repeated to at least `at_least` elements (several max-pass and encode
    workgroups), cut to a multiple of `multiple` elements."""
    reps = -(-at_least // x.size)
    y = np.tile(x, reps)
    return y[: (y.size // multiple) * multiple] if y.size >= multiple else y


# each case as given (one or a few workgroups) and repeated to a larger size
@pytest.mark.parametrize("size", ["small", "large"])
@pytest.mark.parametrize("name", list(_edge_cases().keys()))
def test_luq_edge_values(L, name, size):
    x = _edge_cases()[name]
    if size == "large":
        x = _big(x)
    _check_luq(L, x, 1, x.size, seed=11, counter=2, what=f"{name} {size}")
    if x.size % 64 == 0:
        _check_luq(L, x, 8, x.size // 8, seed=11, counter=2, want_t=True, what=f"{name} {size} tile")


def test_luq_empty(L):
    announce("luq empty")
    x = torch.zeros(0, dtype=torch.float32, device="cuda:0")
    codes, _, alpha, maxabs = L.luq_quantize_grad(x)
    assert host(alpha)[0] == 0 and host(maxabs)[0] == 0


def test_luq_deterministic(L):
    x = synth.grad_1d(300000, seed=55)
    announce("luq determinism")
    outs = [host(L.luq_quantize_grad(to_dev(x), seed=9, counter=4)[0]) for _ in range(3)]
    assert all(np.array_equal(outs[0], o) for o in outs[1:])


# ------------------------------- INT4 ---------------------------------------

def _check_int4(L, x, rows, cols, signed, clip=0.0, want_t=False, what=""):
    announce("int4", what, rows, cols, _dt(x), signed, clip, want_t)
    xd = to_dev(x.reshape(rows, cols) if rows > 1 else x.reshape(-1))
    codes, codes_t, scale = L.int4_quantize(xd, is_signed=signed, clip=clip, codes=True, codes_t=want_t)
    rc, rs = oint4.int4_quantize(x.ravel(), dtype=_dt(x), is_signed=signed, clip=clip)
    s = host(scale)[0]
    if np.isnan(rs):
        assert np.isnan(s)
    else:
        assert s.tobytes() == np.float32(rs).tobytes(), (s, rs)
    assert_codes_equal(host(codes), rc, what)
    if want_t:
        assert_codes_equal(host(codes_t), transpose_codes(rc, rows, cols), what + " transposed")
    return rc, rs


@pytest.mark.parametrize("signed", [True, False])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(1, 1), (1, 13), (1, 100001), (264, 200), (136, 1032), (4104, 64)])
def test_int4_parity(L, signed, dtype, shape):
    r, c = shape
    x = synth.normal((r * c,), 1.3, [300, r, c])
    if dtype == "bf16":
        x = synth.to_bf16_bits(x)
    _check_int4(L, x, r, c, signed, want_t=(r % 8 == 0 and c % 8 == 0), what="int4")


@pytest.mark.parametrize("n", [4096, 81920])
def test_int4_clip_and_edges(L, n):
    x = synth.normal((n,), 1.0, [301])
    _check_int4(L, x, 1, n, True, clip=0.75, what="clip")
    _check_int4(L, x, 64, n // 64, False, clip=2.0, want_t=True, what="clip unsigned")
    _check_int4(L, np.zeros(100, np.float32), 1, 100, True, what="zeros")
    _check_int4(L, -np.abs(x), 1, n, False, what="all negative unsigned")
    y = x.copy()
    y[9] = np.nan
    _check_int4(L, y, 1, n, True, what="nan")
    y = x.copy()
    y[n - 9] = -np.inf
    _check_int4(L, y, 1, n, False, what="-inf unsigned")
    _check_int4(L, np.array([0.5, -0.5, 1.5, 2.5, -2.5, 7, -7, 3.5] * 8, np.float32), 1, 64, True, what="ties")
    _check_int4(L, (x * np.float32(2.0e-38)).astype(np.float32), 1, n, True, what="tiny max")


# ------------------------------- GEMMs --------------------------------------

def _gemm_case(L, M, N, K, ns, signed, seed):
    """dX = Q(g) Q(W): g [M, K], W [K, N]; compares with the oracle."""
    g = synth.lognormal_grad((M, K), -10.0, 2.5, 0.3, [seed, 1])
    w = synth.normal((K, N), 0.05, [seed, 2])
    if not signed:
        w = np.abs(w)
    gd, wd = to_dev(g), to_dev(w)
    announce("dgrad", M, N, K, ns, signed)
    gc, _, alpha, _ = L.luq_quantize_grad(gd, R=4, seed=seed, counter=1, n_samples=ns)
    _, wct, ws = L.int4_quantize(wd, is_signed=signed, codes=False, codes_t=True)
    dx = host(L.luq_gemm_dgrad(gc, alpha, wct, ws, signed, M, N, K, n_samples=ns))
    rc, ra, _ = oluq.luq_quantize(g, R=4, seed=seed, counter=1, n_samples=ns)
    wc, wsr = oint4.int4_quantize(w, is_signed=signed)
    ref, absref = ogemm.gemm_dgrad_ref(rc, ra, wc, wsr, signed, M, N, K)
    assert_gemm_close(dx, ref, absref, f"dgrad {M}x{N}x{K}")
    A = sum(oluq.luq_decode_int(rc[s], M * K).reshape(M, K) for s in range(ns))
    B = oint4.int4_decode_int(wc, K * N, signed).reshape(K, N)
    acc = (A.astype(np.float64) @ B.astype(np.float64)).astype(np.int64)
    assert np.array_equal(dx, epilogue_replica(acc, ra, ns, wsr)), "dgrad epilogue not bit-exact"


# shapes chosen to select each tile configuration (64x64 with and without
# split-K, 128x128, 256x256) with ragged edges in M, N and K
@pytest.mark.parametrize("M,N,K", [(256, 512, 512), (300, 200, 160), (37, 8, 32), (129, 136, 1056),
                                   (64, 64, 32768), (512, 384, 2048), (1500, 1400, 224),
                                   (4192, 4128, 288)])
@pytest.mark.parametrize("ns", [1, 2])
def test_dgrad_parity(L, M, N, K, ns):
    _gemm_case(L, M, N, K, ns, True, seed=M + N + K)


@pytest.mark.parametrize("M,N,K", [(200, 96, 256), (8, 8, 96)])
def test_dgrad_unsigned_weights(L, M, N, K):
    _gemm_case(L, M, N, K, 1, False, seed=7)


def _wgrad_case(L, T, Nout, Kin, ns, signed, seed):
    g = synth.lognormal_grad((T, Nout), -12.0, 2.5, 0.5, [seed, 1])
    a = synth.half_normal((T, Kin), [seed, 2]) if not signed else synth.normal((T, Kin), 1.0, [seed, 2])
    announce("wgrad", T, Nout, Kin, ns, signed)
    _, gct, alpha, _ = L.luq_quantize_grad(to_dev(g), R=4, seed=seed, counter=3, n_samples=ns,
                                           codes=False, codes_t=True)
    _, act, sa = L.int4_quantize(to_dev(a), is_signed=signed, codes=False, codes_t=True)
    dw = host(L.luq_gemm_wgrad(gct, alpha, act, sa, signed, T, Nout, Kin, n_samples=ns))
    rc, ra, _ = oluq.luq_quantize(g, R=4, seed=seed, counter=3, n_samples=ns)
    ac, sar = oint4.int4_quantize(a, is_signed=signed)
    ref, absref = ogemm.gemm_wgrad_ref(rc, ra, ac, sar, signed, T, Nout, Kin)
    assert_gemm_close(dw, ref, absref, f"wgrad {T}x{Nout}x{Kin}")
    G = sum(oluq.luq_decode_int(rc[s], T * Nout).reshape(T, Nout) for s in range(ns))
    X = oint4.int4_decode_int(ac, T * Kin, signed).reshape(T, Kin)
    acc = (G.T.astype(np.float64) @ X.astype(np.float64)).astype(np.int64)
    assert np.array_equal(dw, epilogue_replica(acc, ra, ns, sar)), "wgrad epilogue not bit-exact"


@pytest.mark.parametrize("T,Nout,Kin", [(256, 512, 512), (96, 40, 24), (4096, 64, 96), (8192, 8, 136),
                                         (160, 1544, 1416), (96, 4104, 4120)])
@pytest.mark.parametrize("ns", [1, 2])
def test_wgrad_parity(L, T, Nout, Kin, ns):
    _wgrad_case(L, T, Nout, Kin, ns, signed=False, seed=T + Nout)


def test_wgrad_signed_activations(L):
    _wgrad_case(L, 512, 64, 72, 1, signed=True, seed=9)


# few output rows, long reduction: the 64x192 split-K tile (ragged and
# 128-aligned reductions, ragged columns)
@pytest.mark.parametrize("T,Nout,Kin,ns", [(70048, 40, 200, 1), (66560, 64, 576, 1), (65696, 24, 392, 2)])
def test_wgrad_wide_tile(L, T, Nout, Kin, ns):
    _wgrad_case(L, T, Nout, Kin, ns, signed=False, seed=T % 1000 + Kin)


def test_gemm_long_reduction_exact_split(L):
    """K beyond the int32-exact chunk: chunk sums are combined in int64."""
    _wgrad_case(L, (1 << 18) + 4096, 8, 16, 1, signed=False, seed=13)


def _fwd_case(L, M, N, K, xsig, wsig, seed, dtype=np.float32):
    """y = Q(x) Q(W)^T: x [M, K] activations, W [N, K] weight; compares with the oracle."""
    x = synth.normal((M, K), 1.0, [seed, 1])
    if not xsig:
        x = np.maximum(x, 0)
    w = synth.normal((N, K), 0.05, [seed, 2])
    if not wsig:
        w = np.abs(w)
    announce("fwd", M, N, K, xsig, wsig)
    xc, _, sx = L.int4_quantize(to_dev(x), is_signed=xsig)
    wc, _, sw = L.int4_quantize(to_dev(w), is_signed=wsig)
    y = host(L.int4_gemm_fwd(xc, sx, xsig, wc, sw, wsig, M, N, K))
    rxc, rsx = oint4.int4_quantize(x, is_signed=xsig)
    rwc, rsw = oint4.int4_quantize(w, is_signed=wsig)
    assert host(sx)[0] == rsx and host(sw)[0] == rsw
    ref, absref = ogemm.gemm_fwd_ref(rxc, rsx, xsig, rwc, rsw, wsig, M, N, K)
    assert_gemm_close(y, ref, absref, f"fwd {M}x{N}x{K}")
    X = oint4.int4_decode_int(rxc, M * K, xsig).reshape(M, K)
    Wq = oint4.int4_decode_int(rwc, N * K, wsig).reshape(N, K)
    acc = (X.astype(np.float64) @ Wq.T.astype(np.float64)).astype(np.int64)
    assert np.array_equal(y, epilogue_replica(acc, rsx, 1, rsw)), "fwd epilogue not bit-exact"


# every tile configuration (64x64 with and without split-K, 128x128 with
# BK 64 and 128, 256x256, 64x192) with ragged M, N and K tails
@pytest.mark.parametrize("M,N,K", [(256, 512, 512), (300, 200, 160), (37, 8, 32), (129, 136, 1056),
                                   (64, 64, 32768), (512, 384, 2048), (1500, 1400, 224), (4192, 4128, 288),
                                   (2100, 1100, 64), (40, 200, 70048)])
def test_fwd_parity(L, M, N, K):
    _fwd_case(L, M, N, K, True, True, seed=M + 2 * N + K)


@pytest.mark.parametrize("xsig,wsig", [(False, True), (True, False), (False, False)])
@pytest.mark.parametrize("M,N,K", [(200, 96, 256), (2100, 2060, 1152)])
def test_fwd_code_signedness(L, M, N, K, xsig, wsig):
    _fwd_case(L, M, N, K, xsig, wsig, seed=11 + K)


def test_fwd_long_reduction_exact_split(L):
    """K beyond the int32-exact chunk of INT4 x INT4 (2^17): chunk sums are
    combined in int64, every output still equals the exact epilogue."""
    _fwd_case(L, 8, 24, (1 << 17) + 4096, True, True, seed=21)


def test_fwd_extreme_codes(L):
    """All codes at the end of the range: sums of 49 K (signed) and 225 K
    (unsigned) at K = 2^17, the longest unsplit reduction (4096 x 4096
    outputs fill the 256 x 256 tiles without a split), and the same with a
    split reduction (4 x 8 outputs)."""
    for (M, N), sig, byte, val in [((4096, 4096), True, 0x99, -7), ((4096, 4096), False, 0xFF, 15),
                                   ((4, 8), True, 0x99, -7), ((4, 8), False, 0xFF, 15)]:
        K = 1 << 17
        announce("fwd extreme codes", M, N, K, sig)
        xc = torch.full((M * K // 2,), byte, dtype=torch.uint8, device="cuda:0")
        wc = torch.full((N * K // 2,), byte, dtype=torch.uint8, device="cuda:0")
        one = torch.ones(1, dtype=torch.float32, device="cuda:0")
        y = host(L.int4_gemm_fwd(xc, one, sig, wc, one, sig, M, N, K))
        assert np.all(y == np.float32(val * val * K)), (sig, y[0, 0])


# ------------------------------- im2col -------------------------------------

# fast path (C and W multiples of 8) over several blocks and odd channel-group
# counts; generic path otherwise
@pytest.mark.parametrize("B,H,W,C", [(2, 6, 8, 16), (1, 5, 8, 6), (3, 7, 8, 64), (2, 4, 12, 8), (1, 1, 8, 8),
                                     (4, 30, 32, 24), (3, 20, 16, 64), (1, 3, 8, 512), (1, 3, 8, 520)])
def test_im2col_parity(L, B, H, W, C):
    act = synth.half_normal((B, H, W, C), [400, C])
    announce("im2col", B, H, W, C)
    ac, _, _ = L.int4_quantize(to_dev(act.reshape(B * H * W, C)), is_signed=False)
    col_t = host(L.int4_im2col3x3_t(ac, B, H, W, C))
    rac, _ = oint4.int4_quantize(act, is_signed=False)
    col = oim2col.im2col3x3_codes(rac, B, H, W, C)
    assert_codes_equal(col_t, transpose_codes(col, B * H * W, 9 * C), "im2col_t")


# ------------------------------- HIP graphs ---------------------------------

def test_graph_replays_match_eager(L):
    """The whole step captured in a HIP graph gives the eager results on every
    replay, with eager work and synchronisations between replays."""
    T, D, F = 256, 192, 320
    d = synth.mlp(seed=5, T=T, D=D, F=F)
    g, x, w = to_dev(d["g"]), to_dev(d["x"]), to_dev(d["W"])
    u8 = lambda n: torch.empty(int(n), dtype=torch.uint8, device="cuda:0")
    f1 = lambda: torch.empty(1, dtype=torch.float32, device="cuda:0")
    gc, gct, al, mx = u8(2 * L.plane_bytes(T * F)), u8(2 * L.plane_bytes(T * F)), f1(), f1()
    xct, sx, wct, sw = u8(T * D // 2), f1(), u8(F * D // 2), f1()
    dx = torch.empty(T, D, device="cuda:0")
    dw = torch.empty(F, D, device="cuda:0")
    wq = u8(L.workspace_size(L.OP_QUANTIZE_GRAD, T * F))
    wx = u8(L.workspace_size(L.OP_INT4_QUANTIZE, T * D))
    ww = u8(L.workspace_size(L.OP_INT4_QUANTIZE, F * D))
    wd = u8(max(L.workspace_size(L.OP_GEMM_DGRAD, T, D, F), 1))
    wg = u8(max(L.workspace_size(L.OP_GEMM_WGRAD, T, F, D), 1))

    def step():
        L.luq_quantize_grad(g, 4, 17, 5, 2, gc, gct, al, mx, wq)
        L.int4_quantize(x, True, 0.0, False, xct, sx, wx)
        L.int4_quantize(w, True, 0.0, False, wct, sw, ww)
        L.luq_gemm_dgrad(gc, al, wct, sw, True, T, D, F, 2, dx, wd)
        L.luq_gemm_wgrad(gct, al, xct, sx, True, T, F, D, 2, dw, wg)

    announce("graph eager reference")
    step()
    ref = [host(t).copy() for t in (gc, gct, al, xct, wct, dx, dw)]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for rep in range(4):
        for t in (gc, gct, xct, wct, dx, dw):
            t.zero_()
        torch.cuda.synchronize()
        announce("graph replay", rep)
        graph.replay()
        torch.cuda.synchronize()
        got = [host(t) for t in (gc, gct, al, xct, wct, dx, dw)]
        for a, b in zip(ref, got):
            assert np.array_equal(a, b), f"replay {rep} differs from eager"
        _ = (torch.ones(1024, device="cuda:0") * 2).sum().item()   # eager work between replays

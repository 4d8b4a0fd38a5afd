"""GPU parity of the 3x3 convolution activation gradient (luq_conv3x3_dgrad)
against the oracle (oracle/conv.py), through the C ABI.

Inputs: seeded synthetic gradients, activations' weights and codes from the
library's own quantizers (checked bit-exact against the oracle's on the way).
Every output is compared within 1e-5 of sum_k |a_k b_k| of the float64
result, and bit-for-bit with the fp32 epilogue fl32(fl32(acc) *
fl32(fl32(alpha / n) * s_W)) applied to the exact integer sums.

Shapes span: one and several 256-pixel tiles with a ragged tail, channel
counts that are not multiples of 64 (or of 4: scalar stores), Cout with a
half-filled 64-deep chunk and several chunks, images narrower than a tile
row and wider than 64 pixels (the wide-halo kernel), width and height 1, SMP
planes, unsigned weights, and the full ResNet-50 layer (batch 64, 56 x 56,
64 -> 64) on every pixel.  The row form (image rows of at most 64 pixels,
Cout 32 or 64, C a multiple of 32) gets its own shapes: one and two 32-pixel
tiles per row (ragged or full), one or two k-steps per tap, idle waves and
half-empty channel blocks, height and width 1, and row ranges of one row and
of a few rows crossing image borders.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import synth  # noqa: E402
from oracle import luq as oluq, int4 as oint4  # noqa: E402
from oracle.conv import conv3x3_dgrad_ref  # noqa: E402
from gpu_util import (announce, to_dev, host, transpose_codes, assert_codes_equal,  # noqa: E402
                      assert_gemm_close, epilogue_replica)


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2112_10769_amd as lib
    return lib


def _int_sums(planes, wc, wsig, B, H, W, C, Cout, pixels=None):
    """Exact integer sums: the oracle with unit scales, times the plane count."""
    ns = 1 if np.asarray(planes).ndim == 1 else np.asarray(planes).shape[0]
    s, _ = conv3x3_dgrad_ref(planes, np.float32(1), wc, np.float32(1), wsig, B, H, W, C, Cout, pixels=pixels)
    return np.rint(s * ns).astype(np.int64)


def _conv_case(L, B, H, W, C, Cout, ns=1, wsig=True, seed=0, zero_grad=False, use_codes_t=False):
    T = B * H * W
    g = synth.lognormal_grad((T, Cout), -12.0, 2.5, 0.5, [seed, 1])
    if zero_grad:
        g[:] = 0
    w = synth.normal((Cout, 9 * C), float(np.sqrt(2.0 / (9 * C))), [seed, 2])
    if not wsig:
        w = np.abs(w)
    announce("conv3x3_dgrad", dict(B=B, H=H, W=W, C=C, Cout=Cout, ns=ns, wsig=wsig, seed=seed))
    gc, _, alpha, _ = L.luq_quantize_grad(to_dev(g), R=4, seed=seed, counter=5, n_samples=ns)
    if use_codes_t:
        _, wct, sw = L.int4_quantize(to_dev(w), is_signed=wsig, codes=False, codes_t=True)
    else:
        wcg, _, sw = L.int4_quantize(to_dev(w), is_signed=wsig)
        wct = to_dev(transpose_codes(host(wcg), Cout, 9 * C))
    dact = host(L.luq_conv3x3_dgrad(gc, alpha, wct, sw, wsig, B, H, W, C, Cout, n_samples=ns))
    assert dact.shape == (T, C)

    rc, ra, _ = oluq.luq_quantize(g, R=4, seed=seed, counter=5, n_samples=ns)
    wc, wsr = oint4.int4_quantize(w, is_signed=wsig)
    assert host(alpha)[0].tobytes() == np.float32(ra).tobytes()
    assert host(sw)[0].tobytes() == np.float32(wsr).tobytes()
    gch = host(gc)
    for s in range(ns):
        assert_codes_equal(gch[s], rc[s], f"g codes plane {s}")
    assert_codes_equal(host(wct), transpose_codes(wc, Cout, 9 * C), "W codes_t")
    planes = rc if ns > 1 else rc[0]
    ref, absref = conv3x3_dgrad_ref(planes, ra, wc, wsr, wsig, B, H, W, C, Cout)
    assert_gemm_close(dact, ref, absref, f"conv dact {B}x{H}x{W}x{C}<-{Cout}")
    acc = _int_sums(planes, wc, wsig, B, H, W, C, Cout)
    assert np.array_equal(dact, epilogue_replica(acc, ra, ns, wsr)), "conv dact epilogue not bit-exact"
    return dact


@pytest.mark.parametrize("B,H,W,C,Cout", [
    (1, 4, 4, 64, 64),        # a single partial tile
    (4, 14, 14, 64, 64),      # 784 pixels: three tiles and a 16-pixel tail
    (2, 5, 7, 6, 32),         # C not a multiple of 4 (scalar stores), half chunk
    (3, 9, 11, 96, 96),       # two channel tiles (second partial), 1.5 chunks
    (2, 8, 8, 128, 256),      # four chunks, two full channel tiles
    (1, 3, 100, 8, 64),       # wider than 64: the wide-halo kernel
    (1, 2, 256, 4, 32),       # the widest image accepted
    (3, 1, 37, 16, 64),       # height 1
    (2, 45, 1, 16, 64),       # width 1
    (160, 32, 32, 8, 96),     # 640 tiles: workgroups walk two tiles, two Cout chunks each
    (8, 90, 100, 8, 96),      # wide-halo kernel with workgroups walking two tiles
    # row form (W <= 64, Cout 32 or 64, C a multiple of 32)
    (2, 9, 56, 64, 64),       # two pixel tiles per row, the second ragged
    (3, 5, 64, 96, 32),       # width 64, one k-step per tap, a half-empty second channel block
    (2, 7, 32, 128, 64),      # width 32: one pixel tile, four channel groups per workgroup
    (1, 6, 20, 32, 32),       # one active wave of four
    (3, 1, 40, 32, 64),       # height 1: both outer kernel rows off the image on every row
    (2, 45, 1, 32, 64),       # width 1
    (40, 3, 48, 64, 64),      # fewer rows than ranges: one row per workgroup
    (64, 40, 8, 32, 32),      # 2560 rows: ranges of 2-3 rows that cross image borders
    (256, 56, 8, 32, 32),     # 14336 rows in 1024 ranges: four workgroups per CU
    (16, 30, 40, 96, 64),     # 480 rows, two channel blocks
])
@pytest.mark.parametrize("ns", [1, 2])
def test_conv_dgrad_parity(L, B, H, W, C, Cout, ns):
    _conv_case(L, B, H, W, C, Cout, ns=ns, seed=B * 1000 + H * 100 + W + C + Cout)


@pytest.mark.parametrize("B,H,W,C,Cout", [(2, 7, 9, 24, 64), (1, 6, 70, 8, 96), (2, 9, 56, 64, 64),
                                          (3, 4, 30, 64, 32)])
def test_conv_dgrad_unsigned_weights(L, B, H, W, C, Cout):
    _conv_case(L, B, H, W, C, Cout, wsig=False, seed=17)


def test_conv_dgrad_weight_codes_from_transposed_quantizer(L):
    """The weight's codes_t output of int4_quantize is the operand layout."""
    _conv_case(L, 2, 12, 12, 64, 64, use_codes_t=True, seed=23)


def test_conv_dgrad_all_zero_gradient(L):
    dact = _conv_case(L, 1, 6, 6, 8, 32, zero_grad=True, seed=29)
    assert not np.any(dact)


def test_conv_dgrad_empty(L):
    announce("conv3x3_dgrad empty")
    gc = torch.zeros(256, dtype=torch.uint8, device="cuda")
    a = torch.ones(1, dtype=torch.float32, device="cuda")
    out = torch.full((1,), 7.0, device="cuda")
    L.luq_conv3x3_dgrad(gc, a, gc, a, True, 0, 5, 5, 8, 32, dact=out)
    L.luq_conv3x3_dgrad(gc, a, gc, a, True, 1, 5, 5, 0, 32, dact=out)
    assert host(out)[0] == 7.0


def test_conv_dgrad_resnet_layer_whole_output(L):
    """The ResNet-50 layer (batch 64, 56 x 56, 64 -> 64) in the benchmark's
    launch, every pixel against the oracle."""
    import bench
    announce("conv3x3_dgrad full ResNet layer")
    stages, _, d = bench.build_resnet(L, torch, torch.device("cuda:0"))
    for s in stages:
        if s.name in ("luq_quantize_grad", "int4_quantize(W)", "luq_conv3x3_dgrad"):
            announce("stage", s.name)
            s.fn()
    torch.cuda.synchronize()
    p = synth.RESNET
    B, H, W, C, Co = p["B"], p["H"], p["W"], p["C"], p["Cout"]
    dv = d["dev"]
    assert "dact" in dv, "the benchmark's conv workload computes the activation gradient"
    dact = host(dv["dact"])
    rc, ra, _ = oluq.luq_quantize(d["g"], R=4)
    wc, wsr = oint4.int4_quantize(d["W"], is_signed=True)
    assert_codes_equal(host(dv["gc"])[: rc[0].size], rc[0], "g codes")
    ref, absref = conv3x3_dgrad_ref(rc[0], ra, wc, wsr, True, B, H, W, C, Co)
    assert_gemm_close(dact, ref, absref, "resnet dact")
    acc = _int_sums(rc[0], wc, True, B, H, W, C, Co)
    assert np.array_equal(dact, epilogue_replica(acc, ra, 1, wsr)), "resnet dact epilogue not bit-exact"


# ----------------------------- weight gradient -----------------------------

from oracle.conv import conv3x3_wgrad_ref  # noqa: E402


def _wgrad_case(L, B, H, W, C, Cout, ns=1, asig=False, seed=0, R=4):
    T = B * H * W
    g = synth.lognormal_grad((T, Cout), -12.0, 2.5, 0.5, [seed, 1])
    a = synth.normal((T, C), 1.0, [seed, 2]) if asig else synth.half_normal((T, C), [seed, 2])
    announce("conv3x3_wgrad", dict(B=B, H=H, W=W, C=C, Cout=Cout, ns=ns, asig=asig, seed=seed, R=R))
    gd, ad = to_dev(g), to_dev(a)
    if T % 8 == 0 and Cout % 8 == 0 and C % 8 == 0:
        _, gct, alpha, _ = L.luq_quantize_grad(gd, R=R, seed=seed, counter=6, n_samples=ns, codes=False, codes_t=True)
        _, act, sa = L.int4_quantize(ad, is_signed=asig, codes=False, codes_t=True)
    else:  # row-major codes transposed on the host (the quantizers' codes_t needs multiples of 8)
        gc, _, alpha, _ = L.luq_quantize_grad(gd, R=R, seed=seed, counter=6, n_samples=ns)
        gch = host(gc)
        gct = to_dev(np.stack([transpose_codes(gch[s], T, Cout) for s in range(ns)]).reshape(ns, -1))
        ac, _, sa = L.int4_quantize(ad, is_signed=asig)
        act = to_dev(transpose_codes(host(ac), T, C))
    if ns == 2 and gct.dim() == 2 and gct.shape[1] != L.plane_bytes(T * Cout):
        pad = torch.zeros(2, L.plane_bytes(T * Cout), dtype=torch.uint8, device=gct.device)
        pad[:, : gct.shape[1]] = gct
        gct = pad
    dw = host(L.luq_conv3x3_wgrad(gct, alpha, act, sa, asig, B, H, W, C, Cout, n_samples=ns))
    assert dw.shape == (Cout, 9 * C)
    rc, ra, _ = oluq.luq_quantize(g, R=R, seed=seed, counter=6, n_samples=ns)
    rac, rsa = oint4.int4_quantize(a, is_signed=asig)
    assert host(alpha)[0].tobytes() == np.float32(ra).tobytes()
    assert host(sa)[0].tobytes() == np.float32(rsa).tobytes()
    planes = rc if ns > 1 else rc[0]
    ref, absref = conv3x3_wgrad_ref(planes, ra, rac, rsa, asig, B, H, W, C, Cout)
    assert_gemm_close(dw, ref, absref, f"conv dW {B}x{H}x{W}x{C}->{Cout}")
    s1, _ = conv3x3_wgrad_ref(planes, np.float32(1), rac, np.float32(1), asig, B, H, W, C, Cout)
    acc = np.rint(s1 * ns).astype(np.int64)
    assert np.array_equal(dw, epilogue_replica(acc, ra, ns, rsa)), "conv dW epilogue not bit-exact"
    return dw


@pytest.mark.parametrize("B,H,W,C,Cout", [
    (1, 4, 8, 64, 64),        # one stage, one split
    (4, 14, 16, 64, 64),      # 896 pixels, several stages, one split
    (2, 5, 16, 6, 32),        # C not a multiple of 4 (scalar stores), partial channel tiles
    (3, 9, 32, 96, 96),       # two channel tiles of each, partial second tiles
    (2, 8, 8, 128, 256),      # several output tiles
    (1, 2, 96, 8, 64),        # height 2: every row an image border
    (4, 1, 64, 16, 64),       # height 1
    (32, 32, 1, 16, 64),      # width 1
    (2, 3, 160, 8, 40),       # width above the 64-pixel window margin
    (16, 28, 28, 64, 64),     # several splits (split-K)
    (4, 256, 256, 8, 8),      # more pixel ranges than workgroups: some take two
    # row form (W <= 64, channels in multiples of 32)
    (2, 16, 7, 32, 32),       # odd width: every row starts at another nibble offset
    (1, 64, 1, 32, 32),       # width 1: both column edges in one code
    (8, 20, 36, 64, 64),      # row ranges of 2-3 rows that cross image borders
    (2, 10, 64, 32, 96),      # width 64: two full k-steps, no padding columns
    (3, 6, 48, 96, 32),       # the right edge column is the last code of a lane's 16
    (4, 70, 64, 256, 256),    # row ranges of 70 rows: two staged chunks (68 + 2, or 44 + 26 rows)
])
@pytest.mark.parametrize("ns", [1, 2])
def test_conv_wgrad_parity(L, B, H, W, C, Cout, ns):
    _wgrad_case(L, B, H, W, C, Cout, ns=ns, seed=B * 1000 + H * 100 + W + C + Cout)


@pytest.mark.parametrize("R,ns", [(6, 1), (5, 2)])
@pytest.mark.parametrize("B,H,W,C,Cout", [(4, 14, 16, 64, 64), (16, 28, 28, 64, 64)])
def test_conv_wgrad_parity_wide_levels(L, B, H, W, C, Cout, R, ns):
    """Codes whose values reach 2^6: R = 6, or the sum of two R = 5 samples."""
    _wgrad_case(L, B, H, W, C, Cout, ns=ns, R=R, seed=B * 7 + R)


@pytest.mark.parametrize("R,ns", [(6, 1), (5, 2)])
@pytest.mark.parametrize("B,H,W,C,Co", [(16, 256, 256, 384, 384), (32, 128, 64, 512, 512)])
def test_conv_wgrad_largest_terms_many_pixels(L, R, ns, B, H, W, C, Co):
    """Every term at its largest magnitude, 64 * 120 in carrier units (a
    constant gradient puts every element on the top LUQ level, 2^6 in units
    of alpha for R = 6 and for the sum of two R = 5 samples; a constant
    activation gives the top unsigned INT4 code 15, carried as 8 * 15), over
    2^20 pixels and 6 x 6 channel tiles, so that few workgroups each sum
    long pixel ranges (the second shape takes the row form, whose 2^18 pixels
    split into two row ranges of 2^17).  The exact result has a closed form:
    tap (kh, kw) gathers B (H - |kh - 1|) (W - |kw - 1|) products 2^6 * 15
    in value units."""
    T = B * H * W
    announce("conv3x3_wgrad largest terms", dict(T=T, C=C, Cout=Co, R=R, ns=ns))
    g = torch.full((T, Co), 1.0, dtype=torch.float32, device="cuda:0")
    _, gct, alpha, _ = L.luq_quantize_grad(g, R=R, n_samples=ns, codes=False, codes_t=True)
    del g
    a = torch.full((T, C), 0.75, dtype=torch.float32, device="cuda:0")
    _, act, sa = L.int4_quantize(a, is_signed=False, codes=False, codes_t=True)
    del a
    dw = host(L.luq_conv3x3_wgrad(gct, alpha, act, sa, False, B, H, W, C, Co, n_samples=ns))
    al, s_a = host(alpha)[0], host(sa)[0]
    assert al == np.float32(2.0 ** -R) and s_a == np.float32(np.float32(0.75) / np.float32(15))
    # the kernels' epilogue on the exact carrier sums: fl32(fl32(acc) * fl32(fl32(alpha / ns) * s_a) * 2^-3)
    sc = np.float32(np.float32(np.float32(al) * np.float32(1.0 / ns)) * s_a) * np.float32(0.125)
    for kh in range(3):
        for kw in range(3):
            count = B * (H - abs(kh - 1)) * (W - abs(kw - 1))
            acc = count * 64 * 120  # two samples of 2^5 add up to 2^6 per element as well
            want = np.float32(np.float32(acc) * sc)
            block = dw[:, (kh * 3 + kw) * C:(kh * 3 + kw + 1) * C]
            assert np.all(block == want), (kh, kw, np.unique(block)[:4], want)


def test_conv_wgrad_signed_activations(L):
    _wgrad_case(L, 2, 12, 12, 64, 64, asig=True, seed=31)


def test_conv_wgrad_equals_lowered_gemm(L):
    """The implicit weight gradient equals luq_gemm_wgrad on the im2col lowering, bit for bit."""
    B, H, W, C, Co = 8, 14, 14, 64, 64
    T = B * H * W
    g = synth.lognormal_grad((T, Co), -12.0, 2.5, 0.5, [33, 1])
    a = synth.half_normal((T, C), [33, 2])
    announce("conv wgrad vs lowered")
    _, gct, alpha, _ = L.luq_quantize_grad(to_dev(g), R=4, seed=1, counter=1, codes=False, codes_t=True)
    ac, act, sa = L.int4_quantize(to_dev(a), is_signed=False, codes=True, codes_t=True)
    colt = L.int4_im2col3x3_t(ac, B, H, W, C)
    low = host(L.luq_gemm_wgrad(gct, alpha, colt, sa, False, T, Co, 9 * C))
    imp = host(L.luq_conv3x3_wgrad(gct, alpha, act, sa, False, B, H, W, C, Co))
    assert np.array_equal(low, imp)


def test_conv_wgrad_resnet_layer_whole_output(L):
    """The ResNet-50 layer (batch 64, 56 x 56, 64 -> 64) in the benchmark's
    launch, the whole dW [64, 576] over 200704 pixels against the oracle."""
    import bench
    announce("conv3x3_wgrad full ResNet layer")
    stages, _, d = bench.build_resnet(L, torch, torch.device("cuda:0"))
    for s in stages:
        if s.name in ("luq_quantize_grad", "int4_quantize(act)", "luq_conv3x3_wgrad"):
            announce("stage", s.name)
            s.fn()
    torch.cuda.synchronize()
    p = synth.RESNET
    B, H, W, C, Co = p["B"], p["H"], p["W"], p["C"], p["Cout"]
    dv = d["dev"]
    dw = host(dv["dw"])
    rc, ra, _ = oluq.luq_quantize(d["g"], R=4)
    rac, rsa = oint4.int4_quantize(d["act"].reshape(-1, C), is_signed=False)
    ref, absref = conv3x3_wgrad_ref(rc[0], ra, rac, rsa, False, B, H, W, C, Co)
    assert_gemm_close(dw, ref, absref, "resnet dW")
    s1, _ = conv3x3_wgrad_ref(rc[0], np.float32(1), rac, np.float32(1), False, B, H, W, C, Co)
    assert np.array_equal(dw, epilogue_replica(np.rint(s1).astype(np.int64), ra, 1, rsa)), "resnet dW epilogue"

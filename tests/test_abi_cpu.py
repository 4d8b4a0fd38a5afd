"""The C-ABI library loads without a GPU, exports every function include/luq.h
declares, and rejects invalid arguments on the host before any launch.

Every call below is built to fail validation, so nothing is enqueued; the
pointers are never dereferenced.
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "luq.h")

luq = pytest.importorskip("paper_2112_10769_amd")
LIB = luq.LIB

P = ctypes.c_void_p(0x10000)      # 16-byte aligned, never dereferenced
P2 = ctypes.c_void_p(0x20000)
P3 = ctypes.c_void_p(0x30000)
PMIS = ctypes.c_void_p(0x10004)   # misaligned
NUL = None
WS = 1 << 20


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^[a-z_][\w \*]*?\b((?:luq|int4)_\w+)\s*\(", text, flags=re.M)))


def test_every_declared_function_is_exported():
    names = _declared()
    assert len(names) == 16, names
    for n in names:
        assert hasattr(LIB, n), n
    assert set(names) == set(luq.EXPORTS)


def test_version_and_strings():
    v = int(re.search(r"#define LUQ_ABI_VERSION (\d+)", open(HEADER).read()).group(1))
    assert LIB.luq_abi_version() == v
    for s in range(9):
        assert LIB.luq_status_string(s)
    assert b"non-finite" in LIB.luq_status_string(8)
    assert LIB.luq_status_string(99) == b"unknown status"


def test_plane_and_workspace_sizes():
    assert luq.plane_bytes(0) == 0
    assert luq.plane_bytes(1) == 256
    assert luq.plane_bytes(512) == 256
    assert luq.plane_bytes(514) == 512
    assert luq.plane_bytes(256 * 512) == 65536
    assert luq.workspace_size(luq.OP_QUANTIZE_GRAD, 1000) >= 4096
    assert luq.workspace_size(luq.OP_INT4_QUANTIZE, 0) == 0
    # a long, thin reduction is split along K and needs partial sums
    assert luq.workspace_size(luq.OP_GEMM_WGRAD, 200704, 64, 576) > 0
    assert luq.workspace_size(luq.OP_GEMM_DGRAD, 8192, 4096, 16384) == 0
    # the forward product of INT4 x INT4 (|A|, |B| <= 120 after expansion)
    # is int32-exact only up to K = 2^17: a longer reduction is split
    assert luq.workspace_size(luq.OP_GEMM_FWD, 8192, 4096, 1 << 18) > 0
    assert luq.workspace_size(luq.OP_GEMM_DGRAD, 8192, 4096, 1 << 18) == 0
    assert luq.workspace_size(luq.OP_GEMM_FWD, 8192, 16384, 4096) == 0
    assert luq.workspace_size(99, 1, 1, 1) == 0


def _qg(**kw):
    a = dict(g=P, dt=0, rows=4, cols=8, R=4, seed=0, counter=0, ns=1, codes=P2, codes_t=NUL,
             alpha=P3, maxabs=NUL, ws=P, ws_bytes=WS)
    a.update(kw)
    return LIB.luq_quantize_grad(a["g"], a["dt"], a["rows"], a["cols"], a["R"], a["seed"], a["counter"],
                                 a["ns"], a["codes"], a["codes_t"], a["alpha"], a["maxabs"], a["ws"],
                                 a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(dt=2), 3),
    (dict(rows=-1), 2),
    (dict(rows=3, cols=7), 2),
    (dict(rows=12, cols=8, codes_t=P2), 2),
    (dict(rows=16, cols=12, codes_t=P2), 2),
    (dict(rows=2**40, cols=2**40), 2),
    (dict(R=3), 4), (dict(R=7), 4),
    (dict(R=3 | 0x100), 4), (dict(R=4 | 0x200), 4), (dict(R=0x105, ns=2, g=PMIS), 6),
    (dict(ns=3), 4), (dict(ns=0), 4),
    (dict(ns=2, R=6), 4), (dict(ns=2, R=6 | 0x100), 4),
    (dict(alpha=NUL), 1),
    (dict(R=0x104, alpha=NUL), 1),
    (dict(g=NUL), 1),
    (dict(codes=NUL, codes_t=NUL), 1),
    (dict(ws=NUL), 5),
    (dict(ws_bytes=16), 5),
    (dict(g=PMIS), 6),
    (dict(codes=PMIS), 6),
    (dict(alpha=ctypes.c_void_p(0x10001)), 6),
])
def test_quantize_grad_validation(kw, status):
    assert _qg(**kw) == status
    assert LIB.luq_last_error()


def _hs(**kw):
    a = dict(g=P, dt=0, rows=4, cols=8, R=4, seed=0, counter=0, ns=1, eta=0.1, codes=P2, codes_t=NUL,
             state=P3, alpha=P3, maxabs=NUL, ws=P, ws_bytes=WS)
    a.update(kw)
    return LIB.luq_quantize_grad_hindsight(a["g"], a["dt"], a["rows"], a["cols"], a["R"], a["seed"],
                                           a["counter"], a["ns"], a["eta"], a["codes"], a["codes_t"], a["state"],
                                           a["alpha"], a["maxabs"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(dt=2), 3), (dict(rows=3, cols=7), 2), (dict(rows=12, cols=8, codes_t=P2), 2),
    (dict(R=7), 4), (dict(ns=2, R=6), 4),
    (dict(eta=-0.1), 4), (dict(eta=1.5), 4), (dict(eta=float("nan")), 4),
    (dict(state=NUL), 1), (dict(alpha=NUL), 1), (dict(g=NUL), 1), (dict(codes=NUL, codes_t=NUL), 1),
    (dict(ws=NUL), 5), (dict(ws_bytes=16), 5), (dict(g=PMIS), 6),
    (dict(state=ctypes.c_void_p(0x10002)), 6),
])
def test_quantize_grad_hindsight_validation(kw, status):
    assert _hs(**kw) == status
    assert LIB.luq_last_error()


def _i4(**kw):
    a = dict(x=P, dt=0, rows=4, cols=8, signed=1, clip=0.0, codes=P2, codes_t=NUL, scale=P3, ws=P, ws_bytes=WS)
    a.update(kw)
    return LIB.int4_quantize(a["x"], a["dt"], a["rows"], a["cols"], a["signed"], a["clip"], a["codes"],
                             a["codes_t"], a["scale"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(dt=5), 3), (dict(cols=-2), 2), (dict(rows=8, cols=4, codes_t=P2), 2),
    (dict(clip=float("nan")), 4), (dict(clip=float("inf")), 4),
    (dict(scale=NUL), 1), (dict(x=NUL), 1), (dict(codes=NUL), 1),
    (dict(ws=NUL), 5), (dict(ws_bytes=8), 5), (dict(x=PMIS), 6),
])
def test_int4_validation(kw, status):
    assert _i4(**kw) == status


def _dg(**kw):
    a = dict(g=P, alpha=P3, ns=1, w=P2, ws_=P3, wsig=1, M=64, N=64, K=64, dx=P, ws=P, wsb=WS)
    a.update(kw)
    return LIB.luq_gemm_dgrad(a["g"], a["alpha"], a["ns"], a["w"], a["ws_"], a["wsig"], a["M"], a["N"],
                              a["K"], a["dx"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(g=NUL), 1), (dict(alpha=NUL), 1), (dict(w=NUL), 1), (dict(ws_=NUL), 1), (dict(dx=NUL), 1),
    (dict(ns=3), 4),
    (dict(M=0), 2), (dict(N=-1), 2), (dict(K=48), 2), (dict(K=0), 2), (dict(M=2**31), 2),
    (dict(g=PMIS), 6), (dict(w=PMIS), 6),
    (dict(M=64, N=64, K=1 << 19, ws=NUL), 5),
])
def test_dgrad_validation(kw, status):
    assert _dg(**kw) == status


def test_wgrad_validation():
    args = [P, P3, 1, P2, P3, 0]
    assert LIB.luq_gemm_wgrad(*args, 40, 64, 64, P, P, WS, None) == 2          # T not a multiple of 32
    assert LIB.luq_gemm_wgrad(*args, 200704, 64, 576, P, NUL, 0, None) == 5    # split-K needs ws
    assert LIB.luq_gemm_wgrad(NUL, P3, 1, P2, P3, 0, 64, 8, 8, P, P, WS, None) == 1


def _fw(**kw):
    a = dict(x=P, xs=P3, xsig=1, w=P2, ws_=P3, wsig=1, M=64, N=64, K=64, y=P, ws=P, wsb=WS)
    a.update(kw)
    return LIB.int4_gemm_fwd(a["x"], a["xs"], a["xsig"], a["w"], a["ws_"], a["wsig"], a["M"], a["N"], a["K"],
                             a["y"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(x=NUL), 1), (dict(xs=NUL), 1), (dict(w=NUL), 1), (dict(ws_=NUL), 1), (dict(y=NUL), 1),
    (dict(M=0), 2), (dict(N=-1), 2), (dict(K=48), 2), (dict(K=16), 2), (dict(N=2**31), 2),
    (dict(x=PMIS), 6), (dict(w=PMIS), 6), (dict(y=ctypes.c_void_p(0x10002)), 6),
    (dict(M=8192, N=4096, K=1 << 18, ws=NUL), 5),
    (dict(M=8192, N=4096, K=1 << 18, wsb=1024), 5),
])
def test_fwd_validation(kw, status):
    assert _fw(**kw) == status


def test_im2col_validation():
    assert LIB.int4_im2col3x3_t(P, 1, 3, 3, 3, P2, None) == 2       # odd C
    assert LIB.int4_im2col3x3_t(P, 1, 3, 3, 2, P2, None) == 2       # T = 9 not a multiple of 8
    assert LIB.int4_im2col3x3_t(NUL, 1, 2, 4, 2, P2, None) == 1
    assert LIB.int4_im2col3x3_t(PMIS, 1, 2, 4, 2, P2, None) == 6
    assert LIB.int4_im2col3x3_t(P, -1, 2, 4, 2, P2, None) == 2
    assert LIB.int4_im2col3x3_t(P, 0, 2, 4, 2, P2, None) == 0       # empty: nothing to do


def _cv(**kw):
    a = dict(g=P, alpha=P3, ns=1, w=P2, ws_=P3, wsig=1, B=2, H=8, W=8, C=64, Co=64, out=P)
    a.update(kw)
    return LIB.luq_conv3x3_dgrad(a["g"], a["alpha"], a["ns"], a["w"], a["ws_"], a["wsig"], a["B"], a["H"],
                                 a["W"], a["C"], a["Co"], a["out"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(g=NUL), 1), (dict(alpha=NUL), 1), (dict(w=NUL), 1), (dict(ws_=NUL), 1), (dict(out=NUL), 1),
    (dict(ns=0), 4), (dict(ns=3), 4),
    (dict(B=-1), 2), (dict(Co=48), 2), (dict(Co=0), 2), (dict(Co=16), 2), (dict(Co=32768), 2),
    (dict(W=257), 2), (dict(B=4096, H=256, W=256, Co=64), 2), (dict(B=1, H=1, W=1, C=(1 << 20) + 1, Co=32), 2),
    (dict(g=PMIS), 6), (dict(w=PMIS), 6), (dict(out=ctypes.c_void_p(0x10002)), 6),
    (dict(B=0), 0), (dict(C=0), 0), (dict(B=0, g=NUL, out=NUL), 0),
])
def test_conv_dgrad_validation(kw, status):
    assert _cv(**kw) == status


def test_smp_sum_sample_counts():
    """n_samples accepts 1, 2 and LUQ_SMP_SUM | 2; two samples need R <= 5;
    the convolution takes sample planes only."""
    SUM2 = luq.SMP_SUM | 2
    args = lambda ns, R: (P, 0, 8, 8, R, 0, 0, ns, P2, NUL, P3, NUL, P, WS, None)
    assert LIB.luq_quantize_grad(*args(SUM2, 6)) == 4
    assert LIB.luq_quantize_grad(*args(0x11, 4)) == 4
    assert LIB.luq_quantize_grad(*args(0x10, 4)) == 4
    assert LIB.luq_quantize_grad(*args(3, 4)) == 4
    assert LIB.luq_quantize_grad(P, 0, 8, 8, 4, 0, 0, SUM2, NUL, NUL, P3, NUL, P, WS, None) == 1  # no output
    assert _dg(ns=SUM2, g=NUL) == 1
    assert _dg(ns=0x11) == 4
    assert _dg(ns=SUM2, K=48) == 2
    # an int8 operand of 2^31 bytes: M * K reaches the 32-bit offset limit
    assert _dg(ns=SUM2, M=1 << 17, K=1 << 14) == 2
    assert _cv(ns=SUM2) == 4


def _cw(**kw):
    a = dict(g=P, alpha=P3, ns=1, a=P2, as_=P3, asig=0, B=2, H=8, W=8, C=64, Co=64, dw=P, ws=P, wsb=WS << 6)
    a.update(kw)
    return LIB.luq_conv3x3_wgrad(a["g"], a["alpha"], a["ns"], a["a"], a["as_"], a["asig"], a["B"], a["H"], a["W"],
                                 a["C"], a["Co"], a["dw"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(g=NUL), 1), (dict(alpha=NUL), 1), (dict(a=NUL), 1), (dict(as_=NUL), 1), (dict(dw=NUL), 1),
    (dict(ns=0), 4), (dict(ns=0x12), 4),
    (dict(B=-1), 2), (dict(C=0), 2), (dict(Co=0), 2), (dict(B=0), 2), (dict(H=3, W=3), 2),
    (dict(B=1 << 14, H=256, W=256), 2), (dict(B=17, H=1 << 15, W=1 << 10, C=1, Co=1), 2),
    (dict(g=PMIS), 6), (dict(a=PMIS), 6), (dict(dw=ctypes.c_void_p(0x10002)), 6),
    (dict(B=64, H=56, W=56, ws=NUL), 5), (dict(B=64, H=56, W=56, wsb=1024), 5),
    (dict(B=64, H=56, W=56, ws=PMIS), 6),
])
def test_conv_wgrad_validation(kw, status):
    assert _cw(**kw) == status


def test_conv_wgrad_workspace():
    assert luq.workspace_size(luq.OP_CONV_WGRAD, 64 * 56 * 56, 64, 64) > 0
    assert luq.workspace_size(luq.OP_CONV_WGRAD, 0, 64, 64) == 0


def test_query_status_rejects_bad_workspace_on_the_host():
    """Null and misaligned workspaces are refused before any HIP call."""
    assert LIB.luq_query_status(NUL, None) == 1
    assert LIB.luq_query_status(PMIS, None) == 6
    assert luq.LUQ_ERR_NONFINITE == 8


def test_quantizer_workspace_holds_the_status_word():
    """The status word sits after the 16384 partials and their fold."""
    assert luq.workspace_size(luq.OP_QUANTIZE_GRAD, 1) == (16384 + 2) * 4
    assert luq.workspace_size(luq.OP_INT4_QUANTIZE, 1 << 30) == (16384 + 2) * 4


@pytest.mark.parametrize("T,C,Cout", [
    (200704, 64, 64),            # the ResNet-50 layer
    (1 << 20, 384, 384),         # many channel tiles, few splits
    (1 << 20, 64, 64),
    (1 << 22, 64, 64),
    (1 << 24, 256, 512),
    (1 << 29, 8, 8),
    (1 << 29, 32, 32),           # row form: ranges forced by the int32 bound
    (3 << 18, 512, 512),         # row form: one block set per range, several ranges
])
def test_conv_wgrad_plan_keeps_int32_sums_exact(T, C, Cout):
    """The weight gradient's workgroups sum their pixel ranges in int32: for
    the largest terms (LUQ 2^6 -- R = 6, or two R = 5 samples -- times the
    INT4 carrier 8 * 15) the pixels one workgroup sums must stay below
    2^31 / 7680.  The split count comes from the workspace the plan asks for
    (one [Cout][9C] int32 slab per split); a workgroup then sums at most
    ceil(ranges / splits) ranges of 2 * lg <= 2560 pixels, i.e. fewer than
    T / splits + 2 * 2560 pixels.  The row form (W <= 64, channels in
    multiples of 32) asks for one slab per row range and its ranges differ by
    at most one row of <= 64 pixels, which the same bound covers."""
    ws = luq.workspace_size(luq.OP_CONV_WGRAD, T, C, Cout)
    slab = Cout * 9 * C * 4
    assert ws % slab == 0
    nsplit = max(ws // slab, 1)
    worst_pixels = T / nsplit + 2 * 2560
    assert worst_pixels * 64 * 120 < 2 ** 31, (nsplit, worst_pixels)


def _qn(**kw):
    a = dict(g=P, dt=0, rows=4, cols=8, R=4, seed=0, counter=0, ns=1, codes=P2, codes_t=NUL, alpha=P3, maxabs=NUL)
    a.update(kw)
    return LIB.luq_quantize_grad_noalloc(a["g"], a["dt"], a["rows"], a["cols"], a["R"], a["seed"], a["counter"],
                                         a["ns"], a["codes"], a["codes_t"], a["alpha"], a["maxabs"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(dt=2), 3),
    (dict(rows=-1), 2),
    (dict(rows=3, cols=7), 2),
    (dict(rows=4, cols=12, codes_t=P), 2),
    (dict(R=7), 4),
    (dict(R=6, ns=2), 4),
    (dict(ns=3), 4),
    (dict(alpha=NUL), 1),
    (dict(g=NUL), 1),
    (dict(codes=NUL), 1),
    (dict(g=PMIS), 6),
    (dict(codes=PMIS), 6),
])
def test_noalloc_quantizer_rejects_bad_arguments_on_the_host(kw, status):
    """The allocation-free LUQ entry point validates like luq_quantize_grad
    (no workspace argument) and launches nothing on error."""
    assert _qn(**kw) == status
    assert LIB.luq_last_error()


def test_fp6_carrier_workspace_sizes():
    """The FP6 carrier's workspace holds both operands as FP6 blocks (3/4 byte
    per code, rows padded to 32, K to 64) plus split sums when it splits."""
    M, N, K = 8192, 4096, 16384
    assert luq.workspace_size(luq.OP_GEMM_DGRAD_FP6, M, N, K) == (M + N) * K * 3 // 4
    assert luq.workspace_size(luq.OP_GEMM_WGRAD_FP6, 8192, 16384, 4096) == (16384 + 4096) * 8192 * 3 // 4
    # ragged rows and k: 37 rows pad to 64, K = 96 to 128
    assert luq.workspace_size(luq.OP_GEMM_DGRAD_FP6, 37, 8, 96) >= (64 + 32) * 128 * 3 // 4
    # a reduction above 16384 is split: split sums come on top
    assert luq.workspace_size(luq.OP_GEMM_DGRAD_FP6, 64, 64, 32768) > (64 + 64) * 32768 * 3 // 4


def test_fp6_carrier_rejects_on_the_host():
    def dg(ns, ws_bytes=WS, K=64):
        return LIB.luq_gemm_dgrad(P, P3, ns, P2, P3, 1, 8, 8, K, P, P, ws_bytes, None)
    assert dg(luq.CARRIER_FP6 | 2) == 4
    assert dg(luq.CARRIER_FP6 | luq.SMP_SUM | 2) == 4
    assert dg(luq.CARRIER_FP6 | 1, ws_bytes=16) == 5
    assert dg(luq.CARRIER_FP6 | 1, K=48) == 2

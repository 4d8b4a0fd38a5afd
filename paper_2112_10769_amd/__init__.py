"""Python binding of libluq (the LUQ 4-bit backward hot path on MI355X).

Argument marshalling only: torch tensors supply device memory and the
current HIP stream; every step runs in the HIP kernels of libluq.so.  The
functions carry the names of the C ABI in include/luq.h.  Outputs that are
not passed in are allocated with torch on the input's device.

The library must have been built (``python -m paper_2112_10769_amd._build``
or ``__graft_entry__.build()``); importing the binding without it raises.
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libluq.so")

LUQ_OK = 0
LUQ_ERR_NONFINITE = 8
LUQ_F32, LUQ_BF16 = 0, 1
ALPHA_PW2 = 0x100  # or-ed into R: power-of-two alpha
SMP_SUM = 0x10     # or-ed into n_samples = 2: the two samples as int8 sums
CARRIER_FP6 = 0x40  # or-ed into n_samples = 1 of the backward GEMMs: FP6 MFMA carrier
OP_QUANTIZE_GRAD, OP_INT4_QUANTIZE, OP_GEMM_DGRAD, OP_GEMM_WGRAD, OP_GEMM_FWD, OP_CONV_WGRAD = 0, 1, 2, 3, 4, 5
OP_GEMM_DGRAD_FP6, OP_GEMM_WGRAD_FP6 = 6, 7

EXPORTS = (
    "luq_abi_version", "luq_status_string", "luq_last_error", "luq_plane_bytes",
    "luq_workspace_size", "luq_query_status", "luq_quantize_grad", "luq_quantize_grad_noalloc", "luq_quantize_grad_hindsight", "int4_quantize",
    "luq_gemm_dgrad", "luq_gemm_wgrad", "int4_gemm_fwd", "int4_im2col3x3_t", "luq_conv3x3_dgrad",
    "luq_conv3x3_wgrad",
)


class LuqError(RuntimeError):
    def __init__(self, status, where, detail):
        super().__init__(f"{where}: status {status} ({detail})")
        self.status = status


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"libluq.so not built at {LIB_PATH}; run __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i64, u64, u32, i32, f32, sz = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64,
                                       ctypes.c_uint32, ctypes.c_int, ctypes.c_float, ctypes.c_size_t)
    lib.luq_abi_version.restype = i32
    lib.luq_status_string.restype = ctypes.c_char_p
    lib.luq_status_string.argtypes = [i32]
    lib.luq_last_error.restype = ctypes.c_char_p
    lib.luq_plane_bytes.restype = sz
    lib.luq_plane_bytes.argtypes = [i64]
    lib.luq_workspace_size.restype = sz
    lib.luq_workspace_size.argtypes = [i32, i64, i64, i64]
    lib.luq_query_status.restype = i32
    lib.luq_query_status.argtypes = [vp, vp]
    lib.luq_quantize_grad.restype = i32
    lib.luq_quantize_grad.argtypes = [vp, i32, i64, i64, i32, u64, u32, i32, vp, vp, vp, vp, vp, sz, vp]
    lib.luq_quantize_grad_noalloc.restype = i32
    lib.luq_quantize_grad_noalloc.argtypes = [vp, i32, i64, i64, i32, u64, u32, i32, vp, vp, vp, vp, vp]
    lib.luq_quantize_grad_hindsight.restype = i32
    lib.luq_quantize_grad_hindsight.argtypes = [vp, i32, i64, i64, i32, u64, u32, i32, f32, vp, vp, vp, vp, vp, vp,
                                                sz, vp]
    lib.int4_quantize.restype = i32
    lib.int4_quantize.argtypes = [vp, i32, i64, i64, i32, f32, vp, vp, vp, vp, sz, vp]
    lib.luq_gemm_dgrad.restype = i32
    lib.luq_gemm_dgrad.argtypes = [vp, vp, i32, vp, vp, i32, i64, i64, i64, vp, vp, sz, vp]
    lib.luq_gemm_wgrad.restype = i32
    lib.luq_gemm_wgrad.argtypes = [vp, vp, i32, vp, vp, i32, i64, i64, i64, vp, vp, sz, vp]
    lib.int4_gemm_fwd.restype = i32
    lib.int4_gemm_fwd.argtypes = [vp, vp, i32, vp, vp, i32, i64, i64, i64, vp, vp, sz, vp]
    lib.int4_im2col3x3_t.restype = i32
    lib.int4_im2col3x3_t.argtypes = [vp, i64, i64, i64, i64, vp, vp]
    lib.luq_conv3x3_dgrad.restype = i32
    lib.luq_conv3x3_dgrad.argtypes = [vp, vp, i32, vp, vp, i32, i64, i64, i64, i64, i64, vp, vp]
    lib.luq_conv3x3_wgrad.restype = i32
    lib.luq_conv3x3_wgrad.argtypes = [vp, vp, i32, vp, vp, i32, i64, i64, i64, i64, i64, vp, vp, sz, vp]
    return lib


LIB = _load()


def _check(status, where):
    if status != LUQ_OK:
        detail = LIB.luq_last_error().decode() or LIB.luq_status_string(status).decode()
        raise LuqError(status, where, detail)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(dev):
    return ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)


def _dtype(t):
    if t.dtype == torch.float32:
        return LUQ_F32
    if t.dtype == torch.bfloat16:
        return LUQ_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def abi_version():
    return LIB.luq_abi_version()


def plane_bytes(n):
    return int(LIB.luq_plane_bytes(n))


def workspace_size(op, d0, d1=0, d2=0):
    return int(LIB.luq_workspace_size(op, d0, d1, d2))


def query_status(ws):
    """Status of the last quantizer call that used the workspace tensor ws
    (synchronizes torch's current stream): LUQ_OK or LUQ_ERR_NONFINITE;
    raises LuqError for anything else."""
    st = LIB.luq_query_status(_ptr(ws), _stream(ws.device))
    if st not in (LUQ_OK, LUQ_ERR_NONFINITE):
        _check(st, "luq_query_status")
    return st


def _bytes(n, dev):
    return torch.empty(max(int(n), 1), dtype=torch.uint8, device=dev)


def _shape2d(x):
    if x.dim() == 1:
        return 1, x.shape[0]
    return x.shape[0], x.numel() // max(x.shape[0], 1)


def _code_buffer(n, n_samples, dev):
    """n_samples planes of codes, or with SMP_SUM one int8 byte per element."""
    if not n:
        return _bytes(1, dev)
    if n_samples & SMP_SUM:
        return torch.empty(n, dtype=torch.int8, device=dev)
    return _bytes(n_samples * plane_bytes(n), dev).view(n_samples, -1)


def luq_quantize_grad(g, R=4, seed=0, counter=0, n_samples=1, codes=True, codes_t=False,
                      alpha=None, maxabs=None, ws=None, pw2=False):
    """LUQ codes of g (2-D [rows, cols] or 1-D).  codes / codes_t: True to
    allocate, a uint8 tensor to write into, or False; pw2 for the
    power-of-two alpha; n_samples = 2 | SMP_SUM for the summed samples.
    Returns (codes, codes_t, alpha, maxabs) with codes of shape
    [n_samples, plane] (an int8 vector of the sums with SMP_SUM)."""
    rows, cols = _shape2d(g)
    n = rows * cols
    dev = g.device
    if codes is True:
        codes = _code_buffer(n, n_samples, dev)
    if codes_t is True:
        codes_t = _code_buffer(n, n_samples, dev)
    codes = codes if codes is not False else None
    codes_t = codes_t if codes_t is not False else None
    alpha = torch.empty(1, dtype=torch.float32, device=dev) if alpha is None else alpha
    maxabs = torch.empty(1, dtype=torch.float32, device=dev) if maxabs is None else maxabs
    wsb = workspace_size(OP_QUANTIZE_GRAD, n)
    ws = _bytes(wsb, dev) if ws is None else ws
    g = g.contiguous()
    st = LIB.luq_quantize_grad(_ptr(g) if n else None, _dtype(g), rows, cols, R | (ALPHA_PW2 if pw2 else 0),
                               seed & (2**64 - 1), counter & 0xFFFFFFFF, n_samples,
                               _ptr(codes), _ptr(codes_t), _ptr(alpha), _ptr(maxabs), _ptr(ws),
                               ws.numel(), _stream(dev))
    _check(st, "luq_quantize_grad")
    return codes, codes_t, alpha, maxabs


def luq_quantize_grad_noalloc(g, codes, codes_t, alpha, maxabs=None, R=4, seed=0, counter=0, n_samples=1,
                              pw2=False):
    """luq_quantize_grad with the library's static scratch instead of a
    workspace: the caller passes every output buffer (codes / codes_t may be
    None), and nothing is allocated.  Returns (codes, codes_t, alpha, maxabs)."""
    rows, cols = _shape2d(g)
    n = rows * cols
    st = LIB.luq_quantize_grad_noalloc(_ptr(g) if n else None, _dtype(g), rows, cols, R | (ALPHA_PW2 if pw2 else 0),
                                       seed & (2**64 - 1), counter & 0xFFFFFFFF, n_samples, _ptr(codes),
                                       _ptr(codes_t), _ptr(alpha), _ptr(maxabs), _stream(g.device))
    _check(st, "luq_quantize_grad_noalloc")
    return codes, codes_t, alpha, maxabs


def luq_quantize_grad_hindsight(g, state, R=4, seed=0, counter=0, n_samples=1, eta=0.1, codes=True,
                                codes_t=False, alpha=None, maxabs=None, ws=None, pw2=False):
    """Single-pass LUQ with the in-hindsight maximum: alpha from the estimate
    in `state` (a 1-element float32 device tensor, updated in place to the
    next estimate); pw2 for the power-of-two alpha of the estimate.  Returns
    (codes, codes_t, alpha, maxabs)."""
    rows, cols = _shape2d(g)
    n = rows * cols
    dev = g.device
    if codes is True:
        codes = _code_buffer(n, n_samples, dev)
    if codes_t is True:
        codes_t = _code_buffer(n, n_samples, dev)
    codes = codes if codes is not False else None
    codes_t = codes_t if codes_t is not False else None
    alpha = torch.empty(1, dtype=torch.float32, device=dev) if alpha is None else alpha
    maxabs = torch.empty(1, dtype=torch.float32, device=dev) if maxabs is None else maxabs
    wsb = workspace_size(OP_QUANTIZE_GRAD, n)
    ws = _bytes(wsb, dev) if ws is None else ws
    g = g.contiguous()
    st = LIB.luq_quantize_grad_hindsight(_ptr(g) if n else None, _dtype(g), rows, cols,
                                         R | (ALPHA_PW2 if pw2 else 0),
                                         seed & (2**64 - 1), counter & 0xFFFFFFFF, n_samples, float(eta),
                                         _ptr(codes), _ptr(codes_t), _ptr(state), _ptr(alpha), _ptr(maxabs),
                                         _ptr(ws), ws.numel(), _stream(dev))
    _check(st, "luq_quantize_grad_hindsight")
    return codes, codes_t, alpha, maxabs


def int4_quantize(x, is_signed=True, clip=0.0, codes=True, codes_t=False, scale=None, ws=None):
    """INT4 codes of x.  Returns (codes, codes_t, scale)."""
    rows, cols = _shape2d(x)
    n = rows * cols
    dev = x.device
    nb = (n + 1) // 2
    if codes is True:
        codes = _bytes(nb, dev)
    if codes_t is True:
        codes_t = _bytes(nb, dev)
    codes = codes if codes is not False else None
    codes_t = codes_t if codes_t is not False else None
    scale = torch.empty(1, dtype=torch.float32, device=dev) if scale is None else scale
    wsb = workspace_size(OP_INT4_QUANTIZE, n)
    ws = _bytes(wsb, dev) if ws is None else ws
    x = x.contiguous()
    st = LIB.int4_quantize(_ptr(x) if n else None, _dtype(x), rows, cols,
                           1 if is_signed else 0, float(clip), _ptr(codes), _ptr(codes_t),
                           _ptr(scale), _ptr(ws), ws.numel(), _stream(dev))
    _check(st, "int4_quantize")
    return codes, codes_t, scale


def luq_gemm_dgrad(g_codes, alpha, w_codes_t, w_scale, w_signed, M, N, K, n_samples=1, dx=None, ws=None):
    """dX [M, N] = Q(g) Q(W) from g codes [M, K] and transposed W codes [N, K]."""
    dev = g_codes.device
    dx = torch.empty(M, N, dtype=torch.float32, device=dev) if dx is None else dx
    wsb = workspace_size(OP_GEMM_DGRAD_FP6 if n_samples & CARRIER_FP6 else OP_GEMM_DGRAD, M, N, K)
    ws = _bytes(wsb, dev) if ws is None else ws
    st = LIB.luq_gemm_dgrad(_ptr(g_codes), _ptr(alpha), n_samples, _ptr(w_codes_t), _ptr(w_scale),
                            1 if w_signed else 0, M, N, K, _ptr(dx), _ptr(ws), ws.numel(), _stream(dev))
    _check(st, "luq_gemm_dgrad")
    return dx


def luq_gemm_wgrad(g_codes_t, alpha, a_codes_t, a_scale, a_signed, T, Nout, Kin, n_samples=1, dw=None, ws=None):
    """dW [Nout, Kin] = Q(g)^T Q(a) from transposed codes g^T [Nout, T] and a^T [Kin, T]."""
    dev = g_codes_t.device
    dw = torch.empty(Nout, Kin, dtype=torch.float32, device=dev) if dw is None else dw
    wsb = workspace_size(OP_GEMM_WGRAD_FP6 if n_samples & CARRIER_FP6 else OP_GEMM_WGRAD, T, Nout, Kin)
    ws = _bytes(wsb, dev) if ws is None else ws
    st = LIB.luq_gemm_wgrad(_ptr(g_codes_t), _ptr(alpha), n_samples, _ptr(a_codes_t), _ptr(a_scale),
                            1 if a_signed else 0, T, Nout, Kin, _ptr(dw), _ptr(ws), ws.numel(), _stream(dev))
    _check(st, "luq_gemm_wgrad")
    return dw


def int4_gemm_fwd(x_codes, x_scale, x_signed, w_codes, w_scale, w_signed, M, N, K, y=None, ws=None):
    """y [M, N] = Q(x) Q(W)^T from x codes [M, K] and W codes [N, K] (row-major)."""
    dev = x_codes.device
    y = torch.empty(M, N, dtype=torch.float32, device=dev) if y is None else y
    wsb = workspace_size(OP_GEMM_FWD, M, N, K)
    ws = _bytes(wsb, dev) if ws is None else ws
    st = LIB.int4_gemm_fwd(_ptr(x_codes), _ptr(x_scale), 1 if x_signed else 0, _ptr(w_codes), _ptr(w_scale),
                           1 if w_signed else 0, M, N, K, _ptr(y), _ptr(ws), ws.numel(), _stream(dev))
    _check(st, "int4_gemm_fwd")
    return y


def int4_im2col3x3_t(act_codes, B, H, W, C, col_t=None):
    """Transposed 3x3 im2col of NHWC INT4 codes: [9*C, B*H*W] packed along tokens."""
    dev = act_codes.device
    T = B * H * W
    col_t = _bytes(9 * C * T // 2, dev) if col_t is None else col_t
    st = LIB.int4_im2col3x3_t(_ptr(act_codes), B, H, W, C, _ptr(col_t), _stream(dev))
    _check(st, "int4_im2col3x3_t")
    return col_t


def luq_conv3x3_dgrad(g_codes, alpha, w_codes_t, w_scale, w_signed, B, H, W, C, Cout, n_samples=1, dact=None):
    """Activation gradient [B*H*W, C] of a 3x3 / stride 1 / pad 1 convolution
    from LUQ codes of g [B*H*W, Cout] and transposed weight codes [9*C, Cout]."""
    dev = g_codes.device
    dact = torch.empty(B * H * W, C, dtype=torch.float32, device=dev) if dact is None else dact
    st = LIB.luq_conv3x3_dgrad(_ptr(g_codes), _ptr(alpha), n_samples, _ptr(w_codes_t), _ptr(w_scale),
                               1 if w_signed else 0, B, H, W, C, Cout, _ptr(dact), _stream(dev))
    _check(st, "luq_conv3x3_dgrad")
    return dact


def luq_conv3x3_wgrad(g_codes_t, alpha, a_codes_t, a_scale, a_signed, B, H, W, C, Cout, n_samples=1, dw=None,
                      ws=None):
    """Weight gradient [Cout, 9*C] of a 3x3 / stride 1 / pad 1 convolution from
    transposed LUQ codes of g [Cout, B*H*W] and transposed activation codes
    [C, B*H*W]."""
    dev = g_codes_t.device
    dw = torch.empty(Cout, 9 * C, dtype=torch.float32, device=dev) if dw is None else dw
    wsb = workspace_size(OP_CONV_WGRAD, B * H * W, C, Cout)
    ws = _bytes(wsb, dev) if ws is None else ws
    st = LIB.luq_conv3x3_wgrad(_ptr(g_codes_t), _ptr(alpha), n_samples, _ptr(a_codes_t), _ptr(a_scale),
                               1 if a_signed else 0, B, H, W, C, Cout, _ptr(dw), _ptr(ws), ws.numel(), _stream(dev))
    _check(st, "luq_conv3x3_wgrad")
    return dw

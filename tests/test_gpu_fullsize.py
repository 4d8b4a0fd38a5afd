"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times: the buffers and calls are the benchmark's own (its stage
builders), run once in stage order.

Where the oracle finishes in seconds the whole output is compared (the conv
workload's quantizers, im2col and weight gradient); otherwise outputs are
sampled -- code ranges and single elements computed one by one by the
oracle from their flat indices, GEMM rows and whole 256-row tile bands
computed from exactly the codes they need -- and properties that hold at any
size are checked on the whole output (maxabs, alpha, the transposed layout
against the row-major one, valid code set).
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import synth  # noqa: E402
from oracle import luq as oluq, int4 as oint4, gemm as ogemm, im2col as oim2col  # noqa: E402
from oracle.luq import unpack_nibbles, pack_nibbles  # noqa: E402
from gpu_util import (announce, to_dev, host, transpose_codes, assert_codes_equal,  # noqa: E402
                      assert_gemm_close, epilogue_replica)

DEV = torch.device("cuda:0") if torch.cuda.is_available() else None


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2112_10769_amd as lib
    return lib


def _run(stages, what):
    for s in stages:
        announce(what, "stage", s.name)
        s.fn()
        torch.cuda.synchronize()


def _check_max_alpha(gmax, alpha, xf, R=4):
    m = np.float32(np.abs(xf).max())
    assert host(gmax)[0].tobytes() == m.tobytes()
    assert host(alpha)[0].tobytes() == np.float32(oluq.luq_alpha(m, R)).tobytes()
    return m


def _valid_code_set(nib, R=4):
    """Field <= R+1 and no negative zero, over the whole array."""
    e = nib & 7
    assert int(e.max(initial=0)) <= R + 1
    assert not np.any((e == 0) & (nib >= 8)), "negative zero code"


def _sampled_ranges(n, count, length, seed):
    rng = np.random.default_rng(seed)
    starts = [0, max(0, n - length)] + list(rng.integers(0, n - length, size=count))
    return [(int(s), int(min(n, s + length))) for s in starts]


# --------------------------- conv workload ----------------------------------

@pytest.fixture(scope="module")
def conv(L):
    import bench
    announce("full-size conv workload: inputs and stages")
    stages, _, d = bench.build_resnet(L, torch, DEV, lowered=True)
    _run(stages, "conv")
    p = synth.RESNET
    d.update(B=p["B"], H=p["H"], Wd=p["W"], C=p["C"], Co=p["Cout"])
    d["T"] = p["B"] * p["H"] * p["W"]
    d["luq"] = oluq.luq_quantize(d["g"], R=4)             # the whole tensor
    d["act_q"] = oint4.int4_quantize(d["act"], is_signed=False)
    d["w_q"] = oint4.int4_quantize(d["W"], is_signed=True)
    return d


def test_conv_luq_codes_whole_tensor(conv):
    T, Co, dv = conv["T"], conv["Co"], conv["dev"]
    rc, ra, rm = conv["luq"]
    assert host(dv["alpha"])[0].tobytes() == np.float32(ra).tobytes()
    assert host(dv["gmax"])[0].tobytes() == np.float32(rm).tobytes()
    assert_codes_equal(host(dv["gc"])[: rc[0].size], rc[0], "conv g codes")
    assert_codes_equal(host(dv["gct"])[: rc[0].size], transpose_codes(rc[0], T, Co), "conv g codes_t")


def test_conv_activation_int4_and_im2col_whole_tensor(conv):
    B, H, W, C, T, dv = conv["B"], conv["H"], conv["Wd"], conv["C"], conv["T"], conv["dev"]
    rac, rsa = conv["act_q"]
    assert host(dv["sa"])[0].tobytes() == np.float32(rsa).tobytes()
    assert_codes_equal(host(dv["ac"]), rac, "conv act codes")
    col = oim2col.im2col3x3_codes(rac, B, H, W, C)
    assert_codes_equal(host(dv["colt"]), transpose_codes(col, T, 9 * C), "conv im2col_t")


def test_conv_weight_int4(conv):
    Co, C, dv = conv["Co"], conv["C"], conv["dev"]
    rwc, rsw = conv["w_q"]
    assert host(dv["sw"])[0].tobytes() == np.float32(rsw).tobytes()
    assert_codes_equal(host(dv["wct"]), transpose_codes(rwc, Co, 9 * C), "conv W codes_t")


def test_conv_dgrad_sampled_rows(conv):
    """dX [200704, 576]: 40 rows (image corners, edges, random) against the oracle."""
    T, Co, C, dv = conv["T"], conv["Co"], conv["C"], conv["dev"]
    rc, ra, _ = conv["luq"]
    rwc, rsw = conv["w_q"]
    H, W = conv["H"], conv["Wd"]
    rng = np.random.default_rng(11)
    rows = np.unique(np.concatenate([[0, W - 1, H * W - 1, H * W, T - 1],
                                     rng.integers(0, T, size=35)])).astype(np.int64)
    dx = host(dv["dx"])[rows]
    ref, absref = ogemm.gemm_dgrad_ref(rc, ra, rwc, rsw, True, T, 9 * C, Co, rows=rows)
    assert_gemm_close(dx, ref, absref, "conv dX rows")
    A = oluq.luq_decode_int(rc[0], T * Co).reshape(T, Co)[rows]
    Bm = oint4.int4_decode_int(rwc, Co * 9 * C, True).reshape(Co, 9 * C)
    acc = (A.astype(np.float64) @ Bm.astype(np.float64)).astype(np.int64)
    assert np.array_equal(dx, epilogue_replica(acc, ra, 1, rsw)), "conv dX epilogue not bit-exact"


def test_conv_wgrad_whole_output(conv):
    """dW [64, 576] over the full reduction of 200704 positions (split-K)."""
    B, H, W, C, T, Co, dv = conv["B"], conv["H"], conv["Wd"], conv["C"], conv["T"], conv["Co"], conv["dev"]
    rc, ra, _ = conv["luq"]
    rac, rsa = conv["act_q"]
    col = oim2col.im2col3x3_codes(rac, B, H, W, C)
    dw = host(dv["dw"])
    ref, absref = ogemm.gemm_wgrad_ref(rc, ra, col, rsa, False, T, Co, 9 * C)
    assert_gemm_close(dw, ref, absref, "conv dW")
    G = oluq.luq_decode_int(rc[0], T * Co).reshape(T, Co)
    X = oint4.int4_decode_int(col, T * 9 * C, False).reshape(T, 9 * C)
    acc = (G.T.astype(np.float64) @ X.astype(np.float64)).astype(np.int64)
    assert np.array_equal(dw, epilogue_replica(acc, ra, 1, rsa)), "conv dW epilogue not bit-exact"


# --------------------------- transformer MLP --------------------------------

@pytest.fixture(scope="module")
def mlp_data():
    announce("full-size MLP workload: inputs")
    d = synth.mlp()
    d["gf"] = synth.bf16_bits_to_f32(d["g"])
    d["xq"] = oint4.int4_quantize(d["x"], dtype="bf16", is_signed=True)
    d["wq"] = oint4.int4_quantize(d["W"], is_signed=True)
    return d


@pytest.fixture(scope="module", params=[1, 2, 0x12], ids=["ns1", "smp2", "smp2sum"])
def mlp(L, mlp_data, request):
    import bench
    ns = request.param
    stages, _, d = bench.build_mlp(L, torch, DEV, ns=ns, d={k: mlp_data[k] for k in ("g", "x", "W")})
    _run(stages, f"mlp ns={ns}")
    out = {"ns": ns & 0xF, "summed": bool(ns & L.SMP_SUM), "dev": d["dev"]}
    yield out
    d["dev"].clear()
    torch.cuda.empty_cache()


def _g_nibbles_at(data, idx, alpha, s):
    return oluq.luq_nibbles_at(data["gf"].ravel()[idx], idx, alpha, 4, 0, 0, s)


def test_mlp_luq_sampled_codes_and_layouts(mlp, mlp_data):
    T, F = mlp_data["g"].shape
    n, ns, dv = T * F, mlp["ns"], mlp["dev"]
    alpha = np.float32(oluq.luq_alpha(_check_max_alpha(dv["gmax"], dv["alpha"], mlp_data["gf"]), 4))
    pb = (n + 1) // 2
    pb_pad = (pb + 255) // 256 * 256
    gc, gct = host(dv["gc"]), host(dv["gct"])
    if mlp["summed"]:
        sums = gc[:n].view(np.int8)
        for a, b in _sampled_ranges(n, 24, 4096, 100):
            planes = np.stack([pack_nibbles(oluq.luq_nibbles_range(mlp_data["gf"].ravel()[a:b], a, alpha, 4, 0, 0, s))
                               for s in range(2)])
            assert np.array_equal(sums[a:b], oluq.luq_smp_sum(planes, b - a)), f"sums [{a}, {b})"
        assert np.array_equal(gct[:n].view(np.int8).reshape(F, T), sums.reshape(T, F).T), "sums transposed layout"
        return
    for s in range(ns):
        plane = unpack_nibbles(gc[s * pb_pad:s * pb_pad + pb], n)
        _valid_code_set(plane)
        for a, b in _sampled_ranges(n, 24, 4096, 100 + s):
            ref = oluq.luq_nibbles_range(mlp_data["gf"].ravel()[a:b], a, alpha, 4, 0, 0, s)
            assert np.array_equal(plane[a:b], ref), f"plane {s} codes [{a}, {b})"
        # the transposed plane holds the same codes: whole-array layout check
        tplane = unpack_nibbles(gct[s * pb_pad:s * pb_pad + pb], n).reshape(F, T)
        assert np.array_equal(tplane, plane.reshape(T, F).T), f"plane {s} transposed layout"


def test_mlp_int4_whole_tensors(mlp, mlp_data):
    T, D = mlp_data["x"].shape
    F = mlp_data["W"].shape[0]
    dv = mlp["dev"]
    xc, xs = mlp_data["xq"]
    wc, ws = mlp_data["wq"]
    assert host(dv["sx"])[0].tobytes() == np.float32(xs).tobytes()
    assert host(dv["sw"])[0].tobytes() == np.float32(ws).tobytes()
    assert_codes_equal(host(dv["xct"]), transpose_codes(xc, T, D), "mlp x codes_t")
    assert_codes_equal(host(dv["wct"]), transpose_codes(wc, F, D), "mlp W codes_t")


def test_mlp_dgrad_sampled_rows(mlp, mlp_data):
    """dX [8192, 4096] = Q(g) [8192, 16384] Q(W) [16384, 4096]: 8 rows."""
    T, F = mlp_data["g"].shape
    D = mlp_data["x"].shape[1]
    ns, dv = mlp["ns"], mlp["dev"]
    alpha = np.float32(oluq.luq_alpha(np.float32(np.abs(mlp_data["gf"]).max()), 4))
    wc, ws = mlp_data["wq"]
    rows = np.array([0, 1, 4095, 4096, 5000, 7777, 8190, 8191], dtype=np.int64)
    idx = (rows[:, None] * F + np.arange(F)[None, :]).ravel()
    planes = np.stack([pack_nibbles(_g_nibbles_at(mlp_data, idx, alpha, s)) for s in range(ns)])
    dx = host(dv["dx"])[rows]
    ref, absref = ogemm.gemm_dgrad_ref(planes, alpha, wc, ws, True, len(rows), D, F)
    assert_gemm_close(dx, ref, absref, f"mlp dX rows ns={ns}")
    A = sum(oluq.luq_decode_int(planes[s], len(rows) * F).reshape(len(rows), F) for s in range(ns))
    Bm = oint4.int4_decode_int(wc, F * D, True).reshape(F, D)
    acc = (A.astype(np.float64) @ Bm.astype(np.float64)).astype(np.int64)
    assert np.array_equal(dx, epilogue_replica(acc, alpha, ns, ws)), "mlp dX epilogue not bit-exact"


def test_mlp_wgrad_sampled_rows(mlp, mlp_data):
    """dW [16384, 4096] = Q(g)^T Q(x) over 8192 tokens: 8 rows (output features)."""
    T, F = mlp_data["g"].shape
    D = mlp_data["x"].shape[1]
    ns, dv = mlp["ns"], mlp["dev"]
    alpha = np.float32(oluq.luq_alpha(np.float32(np.abs(mlp_data["gf"]).max()), 4))
    xc, xs = mlp_data["xq"]
    outs = np.array([0, 1, 2, 3, 8191, 8192, 16382, 16383], dtype=np.int64)
    idx = (np.arange(T)[:, None] * F + outs[None, :]).ravel()      # g[:, outs], token-major
    planes = np.stack([pack_nibbles(_g_nibbles_at(mlp_data, idx, alpha, s)) for s in range(ns)])
    dw = host(dv["dw"])[outs]
    ref, absref = ogemm.gemm_wgrad_ref(planes, alpha, xc, xs, True, T, len(outs), D)
    assert_gemm_close(dw, ref, absref, f"mlp dW rows ns={ns}")
    G = sum(oluq.luq_decode_int(planes[s], T * len(outs)).reshape(T, len(outs)) for s in range(ns))
    X = oint4.int4_decode_int(xc, T * D, True).reshape(T, D)
    acc = (G.T.astype(np.float64) @ X.astype(np.float64)).astype(np.int64)
    assert np.array_equal(dw, epilogue_replica(acc, alpha, ns, xs)), "mlp dW epilogue not bit-exact"


def test_mlp_dgrad_full_row_band(mlp, mlp_data):
    """dX rows 4096..4351: one whole 256-row tile band across all 4096 columns
    (every column tile of the 256 x 256 kernel)."""
    T, F = mlp_data["g"].shape
    D = mlp_data["x"].shape[1]
    ns, dv = mlp["ns"], mlp["dev"]
    alpha = np.float32(oluq.luq_alpha(np.float32(np.abs(mlp_data["gf"]).max()), 4))
    wc, ws = mlp_data["wq"]
    r0, nr = 4096, 256
    idx = np.arange(r0 * F, (r0 + nr) * F, dtype=np.int64)
    planes = np.stack([pack_nibbles(_g_nibbles_at(mlp_data, idx, alpha, s)) for s in range(ns)])
    dx = host(dv["dx"])[r0:r0 + nr]
    A = sum(oluq.luq_decode_int(planes[s], nr * F).reshape(nr, F) for s in range(ns))
    Bm = oint4.int4_decode_int(wc, F * D, True).reshape(F, D)
    acc = (A.astype(np.float64) @ Bm.astype(np.float64)).astype(np.int64)
    absacc = np.abs(A).astype(np.float64) @ np.abs(Bm).astype(np.float64)
    sc = np.float64(alpha) / ns * np.float64(ws)
    assert_gemm_close(dx, acc * sc, absacc * sc, f"mlp dX band ns={ns}")
    assert np.array_equal(dx, epilogue_replica(acc, alpha, ns, ws)), "mlp dX band epilogue not bit-exact"


def test_mlp_wgrad_full_row_band(mlp, mlp_data):
    """dW rows (output features) 8192..8447: one whole 256-row tile band
    across all 4096 columns, over the 8192 tokens."""
    T, F = mlp_data["g"].shape
    D = mlp_data["x"].shape[1]
    ns, dv = mlp["ns"], mlp["dev"]
    alpha = np.float32(oluq.luq_alpha(np.float32(np.abs(mlp_data["gf"]).max()), 4))
    xc, xs = mlp_data["xq"]
    o0, no = 8192, 256
    outs = np.arange(o0, o0 + no, dtype=np.int64)
    idx = (np.arange(T)[:, None] * F + outs[None, :]).ravel()      # g[:, outs], token-major
    planes = np.stack([pack_nibbles(_g_nibbles_at(mlp_data, idx, alpha, s)) for s in range(ns)])
    dw = host(dv["dw"])[o0:o0 + no]
    G = sum(oluq.luq_decode_int(planes[s], T * no).reshape(T, no) for s in range(ns))
    X = oint4.int4_decode_int(xc, T * D, True).reshape(T, D)
    acc = (G.T.astype(np.float64) @ X.astype(np.float64)).astype(np.int64)
    absacc = np.abs(G.T).astype(np.float64) @ np.abs(X).astype(np.float64)
    sc = np.float64(alpha) / ns * np.float64(xs)
    assert_gemm_close(dw, acc * sc, absacc * sc, f"mlp dW band ns={ns}")
    assert np.array_equal(dw, epilogue_replica(acc, alpha, ns, xs)), "mlp dW band epilogue not bit-exact"


@pytest.fixture(scope="module")
def mlp_fwd(L, mlp_data):
    import bench
    stages, _, d = bench.build_mlp_fwd(L, torch, DEV, d={k: mlp_data[k] for k in ("g", "x", "W")})
    _run(stages, "mlp fwd")
    yield d["dev"]
    d["dev"].clear()
    torch.cuda.empty_cache()


def test_mlp_fwd_int4_whole_tensors(mlp_fwd, mlp_data):
    xc, xs = mlp_data["xq"]
    wc, ws = mlp_data["wq"]
    assert host(mlp_fwd["sx"])[0].tobytes() == np.float32(xs).tobytes()
    assert host(mlp_fwd["sw"])[0].tobytes() == np.float32(ws).tobytes()
    assert_codes_equal(host(mlp_fwd["xc"]), xc, "mlp fwd x codes")
    assert_codes_equal(host(mlp_fwd["wc"]), wc, "mlp fwd W codes")


def test_mlp_fwd_sampled_rows(mlp_fwd, mlp_data):
    """y [8192, 16384] = Q(x) [8192, 4096] Q(W)^T [4096, 16384]: 8 rows."""
    T, D = mlp_data["x"].shape
    F = mlp_data["W"].shape[0]
    xc, xs = mlp_data["xq"]
    wc, ws = mlp_data["wq"]
    rows = np.array([0, 1, 255, 256, 4100, 6001, 8190, 8191], dtype=np.int64)
    y = host(mlp_fwd["y"])[rows]
    ref, absref = ogemm.gemm_fwd_ref(xc, xs, True, wc, ws, True, T, F, D, rows=rows)
    assert_gemm_close(y, ref, absref, "mlp fwd rows")
    X = oint4.int4_decode_int(xc, T * D, True).reshape(T, D)[rows]
    Wm = oint4.int4_decode_int(wc, F * D, True).reshape(F, D)
    acc = (X.astype(np.float64) @ Wm.T.astype(np.float64)).astype(np.int64)
    assert np.array_equal(y, epilogue_replica(acc, xs, 1, ws)), "mlp fwd epilogue not bit-exact"


# --------------------------- 1-D quantizer sweep ----------------------------

def _sweep_case(L, g, dtype, what):
    n = g.size
    announce("sweep", what, n, dtype)
    gd = to_dev(g)
    codes, _, alpha, gmax = L.luq_quantize_grad(gd, R=4)
    gf = synth.bf16_bits_to_f32(g) if dtype == "bf16" else g
    m = _check_max_alpha(gmax, alpha, gf)
    a = np.float32(oluq.luq_alpha(m, 4))
    nib = unpack_nibbles(host(codes), n)
    _valid_code_set(nib)
    for s0, s1 in _sampled_ranges(n, 24, 2048, n % 9973):
        ref = oluq.luq_nibbles_range(gf[s0:s1], s0, a, 4, 0, 0, 0)
        assert np.array_equal(nib[s0:s1], ref), f"{what}: codes [{s0}, {s1})"


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_sweep_2pow28(L, dtype):
    _sweep_case(L, synth.sweep(28, dtype), dtype, "2^28")


def _tiled_draw(k, dtype, seed):
    """2^k elements that repeat one 2^24-element lognormal(-10, 3) draw (25%
    zeros) with a different sign pattern per copy: the marginal distribution
    of the sweep, cheap to build at 2^29 and 2^30."""
    base = synth.lognormal_grad((1 << 24,), -10.0, 3.0, 0.25, [4, seed])
    copies = 1 << (k - 24)
    flips = np.random.default_rng(seed).random(copies) < 0.5
    if dtype == "bf16":
        b = synth.to_bf16_bits(base)
        sign = np.where(flips, np.uint16(0x8000), np.uint16(0))
        return (b[None, :] ^ sign[:, None]).ravel()
    return (base[None, :] * np.where(flips, -1.0, 1.0).astype(np.float32)[:, None]).ravel()


@pytest.mark.parametrize("k,dtype", [(29, "bf16"), (30, "bf16"), (29, "f32")])
def test_sweep_large_streamed(L, k, dtype):
    """The streamed quantizer paths at the sweep's largest bf16 sizes and
    fp32 2^29 (sampled code ranges, whole-tensor max, alpha and code set)."""
    g = _tiled_draw(k, dtype, 100 + k)
    _sweep_case(L, g, dtype, f"2^{k}")
    torch.cuda.empty_cache()


def test_sweep_2pow30_fp32_beyond_4GiB(L):
    """2^30 fp32 elements (4 GiB in, 512 MiB of codes): byte offsets past
    2^32.  The input repeats one 2^24-element lognormal draw with a different
    sign pattern per copy (same marginal distribution, cheap to build)."""
    base = synth.lognormal_grad((1 << 24,), -10.0, 3.0, 0.25, [4, 30])
    flips = np.where(np.random.default_rng(30).random(64) < 0.5, -1.0, 1.0).astype(np.float32)
    g = (base[None, :] * flips[:, None]).ravel()
    del base
    _sweep_case(L, g, "f32", "2^30")

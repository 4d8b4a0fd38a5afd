"""Benchmark of the LUQ 4-bit backward hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W]
                    [--workload mlp|mlp_smp|mlp_smp_planes|mlp_fwd|resnet|resnet_lowered|small|luq_sweep]

A step is one pass of the whole hot path over one batch of synthetic input,
inputs resident in HBM:
  LUQ of the neural gradient (row-major codes for dX, transposed for dW),
  INT4 of the activations (+ 3x3 im2col on codes for the lowered conv),
  INT4 of the weights (transposed codes), the dX GEMM and the dW GEMM.
The default workload is the largest: the backward of a Transformer MLP
linear layer, 8192 tokens x 4096 -> 16384 (bf16 gradients and activations;
dX 8192x4096 over K = 16384, dW 16384x4096 over K = 8192).  `resnet` is the
ResNet-50 3x3 conv (batch 64, 56x56, 64->64) whose gradients are
implicit-GEMM convolutions on the codes (dact [T, C], dW [Cout, 9C]);
`--workload resnet_lowered` lowers the activation codes by im2col and runs
both as GEMMs on the lowered layout instead (dcol [T, 9C], which a col2im
would still have to fold).  `small` is one linear layer, 256 tokens x
512 -> 512, on fp32 gradients lognormal(-10, 2) with 50% zeros, half-normal
activations (unsigned INT4) and He weights.
`--workload mlp_smp` is the MLP layer with two SMP samples stored as int8
sums (the bytes of two 4-bit planes); `mlp_smp_planes` keeps two planes;
`mlp_fp6` runs both GEMMs on the FP6 carrier (priced against its 10.1 PF
peak instead of INT8's 5.0 POPS).

Prints one JSON line.  `value` is roofline-normalised throughput: the sum,
over the step's kernels, of each kernel's roofline time (algorithmic HBM
bytes / 8 TB/s, or int8 MACs / 5 POPS, whichever is larger) divided by the
measured step time, in percent.  Per-kernel GB/s and TOPS are listed too.
`roofline` describes the dominant kernel, timed with HIP events on the
stream it runs on; `cpu_baseline` times the CPU oracle on a bounded sample
of the same workload (before the GPU is touched), and `paper_context`
carries the only timing the paper reports for this path (its appendix's
stochastic- versus nearest-rounding quantizer times on one A40), as context.

`--workload mlp_fwd` measures the forward pass of the same MLP layer instead:
INT4 of the activations and of the weight (row-major codes) and the forward
GEMM y = Q(x) Q(W)^T (Eq. forward).

`--workload luq_sweep` measures the LUQ quantizer alone on 1-D gradients of
2^20..2^30 elements (fp32 and bf16, lognormal magnitudes exp(N(-10, 3)),
random sign, 25% zeros; 0% and 50% zeros at 2^28): `value` is then the
quantizer's mean fraction of the HBM roofline over the sizes >= 2^27, and
`sweep` lists every size, with the single-pass in-hindsight variant
(roofline N * s_in + N/2 bytes) and the power-of-two alpha beside it.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK = 8.0e12      # bytes/s
I8_PEAK = 5.0e15       # int8 dense ops/s
FP6_PEAK = 10.1e15     # fp6 / fp4 dense ops/s (the FP6 carrier's MFMA)
METRIC = "LUQ quantize GB/s + 4-bit bwd GEMM TFLOP/s (as % of roofline), 1 MI355X"
METRIC_FWD = "INT4 quantize GB/s + 4-bit fwd GEMM TFLOP/s (as % of roofline), 1 MI355X"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    # the GPU's clock climbs for about 0.1 s of sustained load (the MLP step
    # times 1.177 ms after 5 warmup steps, 1.127 ms after 100): the default
    # warmup reaches the steady state a training run works in
    p.add_argument("--warmup", type=int, default=200)
    p.add_argument("--workload", default="mlp", choices=["mlp", "mlp_fp6", "mlp_smp", "mlp_smp_planes", "mlp_fwd", "resnet",
                                                         "resnet_lowered", "small", "luq_sweep"])
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    p.add_argument("--sweep-log2", default=None,
                   help="comma-separated log2 sizes for luq_sweep (default: 20,22,24,26..30)")
    p.add_argument("--calibrate-copy", action="store_true",
                   help="only run a plain 512 MiB device-to-device copy (HBM counter calibration)")
    return p.parse_args()


class Stage:
    """One launch of the step; `peak` is the dense MFMA peak of the carrier its
    MACs run on (INT8, or FP6 for the FP6 carrier)."""

    def __init__(self, name, fn, bytes_, ops=0.0, peak=I8_PEAK):
        self.name, self.fn, self.bytes, self.ops, self.peak = name, fn, float(bytes_), float(ops), peak

    def roofline_s(self):
        return max(self.bytes / HBM_PEAK, self.ops / self.peak)

    def bound(self):
        return "hbm" if self.bytes / HBM_PEAK >= self.ops / self.peak else "mfma"


def build_resnet(L, torch, dev, lowered=False, d=None):
    """The 3x3 conv layer's backward.  By default both gradients come from the
    implicit-GEMM convolution kernels: dact [T, C] (M = T, K = 9 * Cout,
    N = C) and dW [Cout, 9C] (M = Cout, N = 9C, K = T) read the codes of g and
    of the activations directly.  With lowered, the activation codes are
    lowered by im2col (58 MB of column codes) and both gradients are GEMMs on
    the lowered layout: dcol [T, 9C] (which a col2im would still have to
    fold) and dW."""
    import synth
    p = synth.RESNET
    B, H, W, C, Co = p["B"], p["H"], p["W"], p["C"], p["Cout"]
    T, Ki = B * H * W, 9 * C
    d = dict(d) if d is not None else synth.resnet()
    g = torch.from_numpy(d["g"]).to(dev)                              # [T, Cout]
    act = torch.from_numpy(d["act"].reshape(T, C)).to(dev)            # NHWC as [T, C]
    w = torch.from_numpy(d["W"]).to(dev)                              # [Cout, 9C]
    u8 = lambda n: torch.empty(int(n), dtype=torch.uint8, device=dev)
    f32 = lambda *s: torch.empty(*s, dtype=torch.float32, device=dev)
    gc, gct, alpha, gmax = u8(L.plane_bytes(T * Co)), u8(L.plane_bytes(T * Co)), f32(1), f32(1)
    ac, sa = u8(T * C // 2), f32(1)                                   # row-major (lowered) or transposed codes
    wct, sw = u8(Co * Ki // 2), f32(1)
    dw = f32(Co, Ki)
    wsq = u8(L.workspace_size(L.OP_QUANTIZE_GRAD, T * Co))
    wsa = u8(L.workspace_size(L.OP_INT4_QUANTIZE, T * C))
    wsw = u8(L.workspace_size(L.OP_INT4_QUANTIZE, Co * Ki))
    n_g, n_a, n_w = T * Co, T * C, Co * Ki
    dv = dict(g=g, act=act, w=w, gc=gc, gct=gct, alpha=alpha, gmax=gmax, ac=ac, sa=sa, wct=wct, sw=sw, dw=dw)
    stages = [
        Stage("luq_quantize_grad", lambda: L.luq_quantize_grad(g, 4, 0, 0, 1, gc, gct, alpha, gmax, wsq),
              2 * 4 * n_g + 2 * n_g / 2),
    ]
    if lowered:
        colt = u8(Ki * T // 2)
        dx = f32(T, Ki)
        wsd = u8(max(L.workspace_size(L.OP_GEMM_DGRAD, T, Ki, Co), 1))
        wsg = u8(max(L.workspace_size(L.OP_GEMM_WGRAD, T, Co, Ki), 1))
        dv.update(colt=colt, dx=dx)
        stages += [
            Stage("int4_quantize(act)", lambda: L.int4_quantize(act, False, 0.0, ac, False, sa, wsa),
                  2 * 4 * n_a + n_a / 2),
            Stage("int4_im2col3x3_t", lambda: L.int4_im2col3x3_t(ac, B, H, W, C, colt), n_a / 2 + Ki * T / 2),
            Stage("int4_quantize(W)", lambda: L.int4_quantize(w, True, 0.0, False, wct, sw, wsw),
                  2 * 4 * n_w + n_w / 2),
            # dW right after im2col, while its 58 MB of column codes may still be
            # in the last-level cache; the dX GEMM's 462 MB of output would evict them
            Stage("luq_gemm_wgrad", lambda: L.luq_gemm_wgrad(gct, alpha, colt, sa, False, T, Co, Ki, 1, dw, wsg),
                  Co * T / 2 + Ki * T / 2 + 4 * Co * Ki, 2.0 * T * Ki * Co),
            Stage("luq_gemm_dgrad", lambda: L.luq_gemm_dgrad(gc, alpha, wct, sw, True, T, Ki, Co, 1, dx, wsd),
                  T * Co / 2 + Ki * Co / 2 + 4 * T * Ki, 2.0 * T * Ki * Co),
        ]
    else:
        dact = f32(T, C)
        wsc = u8(max(L.workspace_size(L.OP_CONV_WGRAD, T, C, Co), 1))
        dv.update(dact=dact)
        stages += [
            Stage("int4_quantize(act)", lambda: L.int4_quantize(act, False, 0.0, False, ac, sa, wsa),
                  2 * 4 * n_a + n_a / 2),
            Stage("int4_quantize(W)", lambda: L.int4_quantize(w, True, 0.0, False, wct, sw, wsw),
                  2 * 4 * n_w + n_w / 2),
            # g^T and activation codes once each
            Stage("luq_conv3x3_wgrad",
                  lambda: L.luq_conv3x3_wgrad(gct, alpha, ac, sa, False, B, H, W, C, Co, 1, dw, wsc),
                  Co * T / 2 + C * T / 2 + 4 * Co * Ki, 2.0 * T * Ki * Co),
            # g codes, W codes and dact once each
            Stage("luq_conv3x3_dgrad",
                  lambda: L.luq_conv3x3_dgrad(gc, alpha, wct, sw, True, B, H, W, C, Co, 1, dact),
                  T * Co / 2 + Ki * Co / 2 + 4 * T * C, 2.0 * T * C * Ki),
        ]
    d["dev"] = dv
    cfg = {"workload": "resnet50_conv3x3_bwd_lowered" if lowered else "resnet50_conv3x3_bwd",
           "batch": B, "hw": [H, W], "cin": C, "cout": Co,
           "gradients": ("GEMMs on the im2col lowering: dcol [T, 9C] and dW" if lowered else
                         "implicit-GEMM convolution: dact [T, C] and dW [Cout, 9C]"),
           "gemm_dgrad_MNK": [T, Ki, Co] if lowered else [T, C, Ki], "gemm_wgrad_MNK": [Co, Ki, T],
           "grad": "lognormal(-12,2.5) fp32, 50% zeros", "R": 4, "n_samples": 1}
    return stages, cfg, d


def build_mlp(L, torch, dev, ns=1, T=None, D=None, F=None, d=None):
    """Backward of the MLP up-projection.  ns: 1, 2 (two SMP sample planes),
    L.SMP_SUM | 2 (the two samples as int8 sums, same bytes as two planes) or
    L.CARRIER_FP6 | 1 (one sample, both GEMMs on the FP6 carrier; their
    workspaces hold the operands converted to FP6 blocks)."""
    import synth
    T = T or synth.MLP["T"]
    D = D or synth.MLP["D"]
    F = F or synth.MLP["F"]
    d = dict(d) if d is not None else synth.mlp(T=T, D=D, F=F)
    bf = lambda a: torch.from_numpy(a.view("int16")).to(dev).view(torch.bfloat16)
    g, x = bf(d["g"]), bf(d["x"])                                     # [T, F], [T, D]
    w = torch.from_numpy(d["W"]).to(dev)                              # [F, D]
    u8 = lambda n: torch.empty(int(n), dtype=torch.uint8, device=dev)
    f32 = lambda *s: torch.empty(*s, dtype=torch.float32, device=dev)
    summed = bool(ns & L.SMP_SUM)
    fp6 = bool(ns & L.CARRIER_FP6)
    nsamp = ns & 0xF
    gbytes = T * F if summed else nsamp * L.plane_bytes(T * F)
    gc, gct, alpha, gmax = u8(gbytes), u8(gbytes), f32(1), f32(1)
    xct, sx = u8(T * D // 2), f32(1)
    wct, sw = u8(F * D // 2), f32(1)
    dx, dw = f32(T, D), f32(F, D)
    wsq = u8(L.workspace_size(L.OP_QUANTIZE_GRAD, T * F))
    wsx = u8(L.workspace_size(L.OP_INT4_QUANTIZE, T * D))
    wsw = u8(L.workspace_size(L.OP_INT4_QUANTIZE, F * D))
    wsd = u8(max(L.workspace_size(L.OP_GEMM_DGRAD_FP6 if fp6 else L.OP_GEMM_DGRAD, T, D, F), 1))
    wsg = u8(max(L.workspace_size(L.OP_GEMM_WGRAD_FP6 if fp6 else L.OP_GEMM_WGRAD, T, F, D), 1))
    n_g, n_x, n_w = T * F, T * D, F * D
    peak = FP6_PEAK if fp6 else I8_PEAK
    stages = [
        Stage("luq_quantize_grad", lambda: L.luq_quantize_grad(g, 4, 0, 0, ns & ~L.CARRIER_FP6, gc, gct, alpha, gmax,
                                                               wsq),
              2 * 2 * n_g + 2 * nsamp * n_g / 2),
        Stage("int4_quantize(x)", lambda: L.int4_quantize(x, True, 0.0, False, xct, sx, wsx), 2 * 2 * n_x + n_x / 2),
        Stage("int4_quantize(W)", lambda: L.int4_quantize(w, True, 0.0, False, wct, sw, wsw), 2 * 4 * n_w + n_w / 2),
        Stage("luq_gemm_dgrad", lambda: L.luq_gemm_dgrad(gc, alpha, wct, sw, True, T, D, F, ns, dx, wsd),
              nsamp * T * F / 2 + D * F / 2 + 4 * T * D, 2.0 * T * D * F, peak),
        Stage("luq_gemm_wgrad", lambda: L.luq_gemm_wgrad(gct, alpha, xct, sx, True, T, F, D, ns, dw, wsg),
              nsamp * F * T / 2 + D * T / 2 + 4 * F * D, 2.0 * T * D * F, peak),
    ]
    d["dev"] = dict(g=g, x=x, w=w, gc=gc, gct=gct, alpha=alpha, gmax=gmax, xct=xct, sx=sx, wct=wct, sw=sw,
                    dx=dx, dw=dw)
    cfg = {"workload": "transformer_mlp_bwd" + ("_smp2" if nsamp == 2 else "") + ("_planes" if ns == 2 else "")
           + ("_fp6" if fp6 else ""),
           "tokens": T, "d_model": D, "hidden": F, "grad": "lognormal(-14,3) bf16", "R": 4, "n_samples": nsamp,
           "gemm_carrier": "fp6 e3m2 x e2m3 (10.1 PF peak)" if fp6 else "int8 (5.0 POPS peak)"}
    if nsamp == 2:
        cfg["smp_operand"] = "int8 sums of the two samples" if summed else "two 4-bit planes"
    return stages, cfg, d


def build_mlp_fwd(L, torch, dev, T=None, D=None, F=None, d=None):
    """Forward of the MLP up-projection: y [T, F] = Q(x) Q(W)^T, x [T, D], W [F, D]."""
    import synth
    T = T or synth.MLP["T"]
    D = D or synth.MLP["D"]
    F = F or synth.MLP["F"]
    d = dict(d) if d is not None else synth.mlp(T=T, D=D, F=F)
    x = torch.from_numpy(d["x"].view("int16")).to(dev).view(torch.bfloat16)
    w = torch.from_numpy(d["W"]).to(dev)
    u8 = lambda n: torch.empty(int(n), dtype=torch.uint8, device=dev)
    f32 = lambda *s: torch.empty(*s, dtype=torch.float32, device=dev)
    xc, sx, wc, sw, y = u8(T * D // 2), f32(1), u8(F * D // 2), f32(1), f32(T, F)
    wsx = u8(L.workspace_size(L.OP_INT4_QUANTIZE, T * D))
    wsw = u8(L.workspace_size(L.OP_INT4_QUANTIZE, F * D))
    wsf = u8(max(L.workspace_size(L.OP_GEMM_FWD, T, F, D), 1))
    n_x, n_w = T * D, F * D
    stages = [
        Stage("int4_quantize(x)", lambda: L.int4_quantize(x, True, 0.0, xc, False, sx, wsx), 2 * 2 * n_x + n_x / 2),
        Stage("int4_quantize(W)", lambda: L.int4_quantize(w, True, 0.0, wc, False, sw, wsw), 2 * 4 * n_w + n_w / 2),
        Stage("int4_gemm_fwd", lambda: L.int4_gemm_fwd(xc, sx, True, wc, sw, True, T, F, D, y, wsf),
              T * D / 2 + F * D / 2 + 4 * T * F, 2.0 * T * D * F),
    ]
    d["dev"] = dict(x=x, w=w, xc=xc, sx=sx, wc=wc, sw=sw, y=y)
    cfg = {"workload": "transformer_mlp_fwd", "tokens": T, "d_model": D, "hidden": F,
           "gemm_fwd_MNK": [T, F, D], "x": "N(0,1) bf16", "W": "N(0,0.02^2) fp32"}
    return stages, cfg, d


def build_small(L, torch, dev, d=None):
    """One linear layer backward, 256 tokens x 512 -> 512, on the small
    parity workload's own inputs: g fp32 lognormal(-10, 2) with 50% zeros,
    activations half-normal (unsigned INT4), W [512 out, 512 in] He (signed)."""
    import synth
    T, D, F = 256, 512, 512
    d = dict(d) if d is not None else synth.small()
    g = torch.from_numpy(d["g"]).to(dev)                              # [T, F]
    a = torch.from_numpy(d["a"]).to(dev)                              # [T, D]
    w = torch.from_numpy(d["W"]).to(dev)                              # [F, D]
    u8 = lambda n: torch.empty(int(n), dtype=torch.uint8, device=dev)
    f32 = lambda *s: torch.empty(*s, dtype=torch.float32, device=dev)
    gc, gct, alpha, gmax = u8(L.plane_bytes(T * F)), u8(L.plane_bytes(T * F)), f32(1), f32(1)
    act, sa, wct, sw = u8(T * D // 2), f32(1), u8(F * D // 2), f32(1)
    dx, dw = f32(T, D), f32(F, D)
    wsq = u8(L.workspace_size(L.OP_QUANTIZE_GRAD, T * F))
    wsa = u8(L.workspace_size(L.OP_INT4_QUANTIZE, T * D))
    wsw = u8(L.workspace_size(L.OP_INT4_QUANTIZE, F * D))
    wsd = u8(max(L.workspace_size(L.OP_GEMM_DGRAD, T, D, F), 1))
    wsg = u8(max(L.workspace_size(L.OP_GEMM_WGRAD, T, F, D), 1))
    n_g, n_a, n_w = T * F, T * D, F * D
    stages = [
        Stage("luq_quantize_grad", lambda: L.luq_quantize_grad(g, 4, 0, 0, 1, gc, gct, alpha, gmax, wsq),
              2 * 4 * n_g + 2 * n_g / 2),
        Stage("int4_quantize(a)", lambda: L.int4_quantize(a, False, 0.0, False, act, sa, wsa), 2 * 4 * n_a + n_a / 2),
        Stage("int4_quantize(W)", lambda: L.int4_quantize(w, True, 0.0, False, wct, sw, wsw), 2 * 4 * n_w + n_w / 2),
        Stage("luq_gemm_dgrad", lambda: L.luq_gemm_dgrad(gc, alpha, wct, sw, True, T, D, F, 1, dx, wsd),
              T * F / 2 + D * F / 2 + 4 * T * D, 2.0 * T * D * F),
        Stage("luq_gemm_wgrad", lambda: L.luq_gemm_wgrad(gct, alpha, act, sa, False, T, F, D, 1, dw, wsg),
              F * T / 2 + D * T / 2 + 4 * F * D, 2.0 * T * D * F),
    ]
    d["dev"] = dict(g=g, a=a, w=w, gc=gc, gct=gct, alpha=alpha, gmax=gmax, act=act, sa=sa, wct=wct, sw=sw,
                    dx=dx, dw=dw)
    cfg = {"workload": "linear_256x512x512_bwd", "tokens": T, "d_in": D, "d_out": F,
           "grad": "lognormal(-10,2) fp32, 50% zeros", "a": "half-normal fp32 (unsigned INT4)",
           "W": "He fp32 (signed INT4)", "R": 4, "n_samples": 1}
    return stages, cfg, d


SWEEP_LOG2 = (20, 22, 24, 26, 27, 28, 29, 30)


def device_lognormal(torch, n, mu, sigma, zero_frac, seed, dtype):
    """Gradient-like tensor drawn on the device: |g| = exp(N(mu, sigma)),
    random sign, a fraction of exact zeros (inputs only; no method arithmetic)."""
    gen = torch.Generator(device="cuda:0")
    gen.manual_seed(seed)
    g = torch.randn(n, generator=gen, device="cuda:0")
    g.mul_(sigma).add_(mu).exp_()
    sign = torch.rand(n, generator=gen, device="cuda:0") < 0.5
    g[sign] = -g[sign]
    del sign
    if zero_frac > 0:
        g[torch.rand(n, generator=gen, device="cuda:0") < zero_frac] = 0.0
    return g if dtype == "f32" else g.to(torch.bfloat16)


def run_sweep(L, torch, steps, sizes=None):
    dev = torch.device("cuda:0")
    sizes = sizes or SWEEP_LOG2
    cases = [(k, dt, 0.25) for dt in ("f32", "bf16") for k in sizes]
    if sizes == SWEEP_LOG2:
        cases += [(28, dt, z) for dt in ("f32", "bf16") for z in (0.0, 0.5)]
    rows = []
    for k, dt, z in cases:
        n = 1 << k
        g = device_lognormal(torch, n, -10.0, 3.0, z, 4000 + 10 * k + (dt == "bf16"), dt)
        s_in = 4 if dt == "f32" else 2
        codes = torch.empty(L.plane_bytes(n), dtype=torch.uint8, device=dev)
        alpha = torch.empty(1, dtype=torch.float32, device=dev)
        gmax = torch.empty(1, dtype=torch.float32, device=dev)
        ws = torch.empty(L.workspace_size(L.OP_QUANTIZE_GRAD, n), dtype=torch.uint8, device=dev)
        fn = lambda: L.luq_quantize_grad(g, 4, 0, 0, 1, codes, False, alpha, gmax, ws)
        per_graph = 10 if k >= 26 else 50
        gr = capture(torch, [fn] * per_graph)
        gr.replay()
        t = time_graph(torch, gr, max(3, steps // 4)) / per_graph
        alg = 2 * n * s_in + n / 2
        # power-of-two alpha (same passes, same bytes)
        fp = lambda: L.luq_quantize_grad(g, 4 | L.ALPHA_PW2, 0, 0, 1, codes, False, alpha, gmax, ws)
        grp = capture(torch, [fp] * per_graph)
        grp.replay()
        tp = time_graph(torch, grp, max(3, steps // 4)) / per_graph
        # single pass with the in-hindsight maximum (the estimate starts at
        # this tensor's maximum, so every replay sees the same estimate)
        state = gmax.clone()
        hs = lambda: L.luq_quantize_grad_hindsight(g, state, 4, 0, 0, 1, 0.0, codes, False, alpha, None, ws)
        grh = capture(torch, [hs] * per_graph)
        grh.replay()
        th = time_graph(torch, grh, max(3, steps // 4)) / per_graph
        alg1 = n * s_in + n / 2
        rows.append({"log2_n": k, "dtype": dt, "zeros": z, "us": round(t * 1e6, 2),
                     "GB/s": round(alg / t / 1e9, 1), "frac": round(alg / t / HBM_PEAK, 4),
                     "single_read_GB/s": round((n * s_in + n / 2) / t / 1e9, 1),
                     "hindsight_us": round(th * 1e6, 2), "hindsight_GB/s": round(alg1 / th / 1e9, 1),
                     "hindsight_frac": round(alg1 / th / HBM_PEAK, 4),
                     "pw2_us": round(tp * 1e6, 2), "pw2_frac": round(alg / tp / HBM_PEAK, 4)})
        del g, codes, ws, gr, grh, grp
        torch.cuda.empty_cache()
    big = [r["frac"] for r in rows if r["log2_n"] >= min(27, max(sizes)) and r["zeros"] == 0.25]
    top = max((r for r in rows if r["zeros"] == 0.25 and r["dtype"] == "f32"), key=lambda r: r["log2_n"])
    n = 1 << top["log2_n"]
    roof = {"kernel": "luq_quantize_grad (max pass + encode)", "bound": "hbm",
            "achieved": top["GB/s"], "peak": 8000.0, "unit": "GB/s", "frac": top["frac"],
            "traffic": None, "algorithmic_bytes": 2 * n * 4 + n / 2, "launch_us": top["us"]}
    cfg = {"workload": "luq_quantizer_sweep", "sizes": [f"2^{k}" for k in sizes],
           "dtypes": ["f32", "bf16"], "grad": "lognormal(-10,3), random sign, 25% zeros", "R": 4,
           "n_samples": 1}
    return rows, 100.0 * sum(big) / len(big), roof, cfg


def cpu_sweep_baseline():
    """The oracle's LUQ of 2^26 fp32 elements over a process pool, and of 2^24
    on one core, each repeated until at least 5 s."""
    from oracle import luq as oluq
    import synth
    info = cpu_info()
    procs = max(1, min(POOL_MAX_PROCS, info["cores_available"]))
    n = 1 << 26
    g = synth.grad_1d(n, "f32", 0.25, seed=4)
    tp, reps_p = 0.0, 0
    while tp < 5.0:
        tp += pool_quantizers(g, "f32", procs, int4=False)[0]
        reps_p += 1
    n1 = 1 << 24
    t1, reps_1 = 0.0, 0
    while t1 < 5.0:
        t0 = time.perf_counter()
        oluq.luq_quantize(g[:n1], R=4)
        t1 += time.perf_counter() - t0
        reps_1 += 1
    alg = (2 * n * 4 + n / 2) * reps_p
    alg1 = (2 * n1 * 4 + n1 / 2) * reps_1
    legs = [{"leg": f"luq {n} fp32 elements, pool", "reps": reps_p, "s": round(tp, 3), "cores": procs,
             "GB/s": round(alg / tp / 1e9, 4)},
            {"leg": f"luq {n1} fp32 elements, one core", "reps": reps_1, "s": round(t1, 3), "cores": 1,
             "GB/s": round(alg1 / t1 / 1e9, 4)}]
    return {"value": round(100.0 * alg / tp / HBM_PEAK, 6), "unit": "% of MI355X HBM roofline",
            "cores": procs, "kind": "oracle", "GB/s": round(alg / tp / 1e9, 4),
            "sample": f"LUQ (max pass, then encode) of 2^26 fp32 elements over {procs} processes, {reps_p} times",
            "legs": legs, **info}


def capture(torch, fns):
    """A HIP graph that replays the given launches (no host work per replay)."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for f in fns:
            f()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for f in fns:
            f()
    torch.cuda.synchronize()
    return g


def time_graph(torch, g, reps):
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record()
    for _ in range(reps):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / 1e3 / reps


def time_stages(torch, stages, steps, warmup):
    """Step time (the whole hot path replayed as one graph) and per-stage times
    measured inside the step: right after the timed replays, the same steps
    run once more with HIP events recorded on the stream between the stages,
    so every stage is timed on the inputs its predecessors just wrote and at
    the clock the step runs at (a kernel repeated on its own keeps its inputs
    in the last-level cache and runs at a higher clock)."""
    step = capture(torch, [s.fn for s in stages])
    for _ in range(warmup):
        step.replay()
    step_s = time_graph(torch, step, steps)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(stages) + 1)] for _ in range(steps)]
    torch.cuda.synchronize()
    # short steps: a spin kernel holds the GPU while the host enqueues every
    # eager step, so the stages then run back to back (their kernels finish
    # faster than the host could feed them one by one).  Long steps keep the
    # GPU ahead of the host anyway and run right after the timed replays, in
    # the same clock state.
    if step_s < 3e-4:
        torch.cuda._sleep(50_000_000)
    for e in ev:
        e[0].record()
        for i, s in enumerate(stages):
            s.fn()
            e[i + 1].record()
    torch.cuda.synchronize()
    per = {s.name: sum(e[i].elapsed_time(e[i + 1]) for e in ev) / 1e3 / steps for i, s in enumerate(stages)}
    return step_s, per


# ---------------------------------------------------------------------------
# CPU baseline: the oracle as it stands, on the host's cores.

POOL_CHUNK = 1 << 22        # elements per pool task (the oracle's Philox is counter-based)
POOL_MAX_PROCS = 16         # the host share that goes with one GPU

# Paper context: the appendix's stochastic-rounding overhead table, the only
# timing the paper gives for this path (one A40, the authors' CUDA kernel,
# mean of 100 runs per size).  Another machine's numbers: context, not a target.
PAPER_SR_TABLE = {
    "source": "appendix, stochastic rounding overhead (SR vs round-to-nearest quantizer times)",
    "hardware": "1x NVIDIA A40, the authors' CUDA quantizer kernel (described as not optimised), mean of 100 runs",
    "tensor_elements": [1e3, 1e4, 1e5, 1e6, 1e7, 1e8],
    "sr_us": [2.64, 2.64, 3.94, 4.07, 6.89, 9.83],
    "rdn_us": [2.55, 2.60, 3.89, 4.01, 6.78, 9.77],
}


def paper_context():
    t = dict(PAPER_SR_TABLE)
    t["sr_overhead_pct"] = [round(100.0 * (a / b - 1.0), 2) for a, b in zip(t["sr_us"], t["rdn_us"])]
    t["note"] = ("the paper simulates 4-bit GEMMs and publishes no GEMM throughput; its SR quantizer costs "
                 "0.6-3.5% over round-to-nearest on the A40. Here the stochastic LUQ encode and the INT4 "
                 "round-to-nearest encode are timed in the same step (kernels.luq_quantize_grad vs "
                 "kernels.int4_quantize(x))")
    return t


def cpu_info():
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas = None
    return {"cpu_model": model, "cores_available": len(os.sched_getaffinity(0)), "blas_threads": blas}


_POOL_VIEW = {}


def _pool_view(name, n, dt):
    """A worker's view of the shared input (attached once per process)."""
    if name not in _POOL_VIEW:
        import numpy as np
        from multiprocessing import shared_memory
        shm = shared_memory.SharedMemory(name=name)
        _POOL_VIEW[name] = (shm, np.ndarray((n,), dtype=np.uint16 if dt == "bf16" else np.float32, buffer=shm.buf))
    return _POOL_VIEW[name][1]


def _pool_task(job):
    """One 2^22-element chunk of an oracle pass: the max key, or the LUQ / INT4
    codes given the tensor-wide alpha / range (which is what makes the
    passes independent per chunk)."""
    import numpy as np
    from oracle import luq as oluq, int4 as oint4
    kind, name, n, dt, c0, c1, arg = job
    x = _pool_view(name, n, dt)[c0:c1]
    xf = oluq.to_float32(x, dt)
    if kind == "maxabs":
        return float(np.abs(xf.astype(np.float64)).max())
    if kind == "luq":
        alpha, R = arg
        return int(oluq.pack_nibbles(oluq.luq_nibbles_range(xf, c0, np.float32(alpha), R, 0, 0, 0)).size)
    if kind == "int4":
        codes, _ = oint4.int4_quantize(x, dtype=dt, is_signed=True, clip=arg)
        return int(codes.size)
    raise ValueError(kind)


def _pool_warm(_):
    from oracle import luq, int4  # noqa: F401  (import cost outside the timed region)
    return 0


def pool_quantizers(x, dt, procs, int4=True):
    """The oracle's LUQ and INT4 (signed, max-abs) of the whole tensor x over
    a pool of `procs` processes: a max pass, then the encode, each split into
    2^22-element tasks.  Returns (seconds LUQ, seconds INT4 or None)."""
    import multiprocessing as mp
    from multiprocessing import shared_memory
    import numpy as np
    n = x.size
    shm = shared_memory.SharedMemory(create=True, size=x.nbytes)
    try:
        np.ndarray(x.shape, dtype=x.dtype, buffer=shm.buf)[...] = x
        chunks = [(c, min(n, c + POOL_CHUNK)) for c in range(0, n, POOL_CHUNK)]
        ctx = mp.get_context("spawn")  # fresh interpreters: nothing of this process is inherited
        with ctx.Pool(procs) as pool:
            # a bounded wait: a pool whose workers cannot start would otherwise
            # replace them forever
            run = lambda fn, jobs: pool.map_async(fn, jobs).get(timeout=300)
            run(_pool_warm, range(procs))
            run(_pool_task, [("maxabs", shm.name, n, dt, c0, c0 + 8, None) for c0, _ in chunks[:procs]])
            t0 = time.perf_counter()
            m = max(run(_pool_task, [("maxabs", shm.name, n, dt, c0, c1, None) for c0, c1 in chunks]))
            alpha = float(np.float32(m * 2.0 ** -4))
            run(_pool_task, [("luq", shm.name, n, dt, c0, c1, (alpha, 4)) for c0, c1 in chunks])
            t_luq = time.perf_counter() - t0
            t_int4 = None
            if int4:
                t0 = time.perf_counter()
                m = max(run(_pool_task, [("maxabs", shm.name, n, dt, c0, c1, None) for c0, c1 in chunks]))
                run(_pool_task, [("int4", shm.name, n, dt, c0, c1, float(np.float32(m))) for c0, c1 in chunks])
                t_int4 = time.perf_counter() - t0
    finally:
        shm.close()
        shm.unlink()
    return t_luq, t_int4


def cpu_baseline(workload, d):
    """The oracle on a bounded sample of the workload (10-30 s of CPU work).
    `value` is the sample's roofline-normalised throughput (the same measure
    as the GPU line); `legs` gives every timed piece with the cores it used."""
    import numpy as np
    from oracle import luq as oluq, int4 as oint4, gemm as ogemm, im2col as oim2col, conv as oconv
    import synth
    info = cpu_info()
    blas = info["blas_threads"] or 1
    legs = []
    t_roof, t_cpu = 0.0, 0.0

    def timed(label, fn, bytes_, ops=0.0, cores=1, value=True):
        nonlocal t_roof, t_cpu
        t0 = time.perf_counter()
        fn()
        dt = time.perf_counter() - t0
        roof = max(bytes_ / HBM_PEAK, ops / I8_PEAK)
        legs.append({"leg": label, "s": dt, "cores": cores, "roof_s": roof})
        if value:
            t_roof += roof
            t_cpu += dt
        return dt

    if workload in ("resnet", "resnet_lowered"):
        # the whole step, repeated until at least 10 s of CPU work
        p = synth.RESNET
        B, H, W, C, Co = p["B"], p["H"], p["W"], p["C"], p["Cout"]
        T, K9 = B * H * W, 9 * C
        n_g, n_a, n_w = T * Co, T * C, Co * K9
        reps = 0
        while t_cpu < 10.0:
            out = {}
            legs.clear()

            def luq():
                out["g"] = oluq.luq_quantize(d["g"], R=4)

            def act():
                out["a"] = oint4.int4_quantize(d["act"], is_signed=False)

            def col():
                out["col"] = oim2col.im2col3x3_codes(out["a"][0], B, H, W, C)

            def wq():
                out["w"] = oint4.int4_quantize(d["W"], is_signed=True)

            timed("luq", luq, 2 * 4 * n_g + 2 * n_g / 2)
            timed("int4(act)", act, 2 * 4 * n_a + n_a / 2)
            timed("int4(W)", wq, 2 * 4 * n_w + n_w / 2)
            gc, ga, _ = out["g"]
            if workload == "resnet_lowered":
                timed("im2col", col, n_a / 2 + K9 * T / 2)
                timed("dW", lambda: ogemm.gemm_wgrad_ref(gc, ga, out["col"], out["a"][1], False, T, Co, K9),
                      Co * T / 2 + K9 * T / 2 + 4 * Co * K9, 2.0 * T * K9 * Co, cores=blas)
                timed("dX", lambda: ogemm.gemm_dgrad_ref(gc, ga, out["w"][0], out["w"][1], True, T, K9, Co),
                      T * Co / 2 + K9 * Co / 2 + 4 * T * K9, 2.0 * T * K9 * Co, cores=blas)
            else:
                timed("dW", lambda: oconv.conv3x3_wgrad_ref(gc, ga, out["a"][0], out["a"][1], False,
                                                            B, H, W, C, Co),
                      Co * T / 2 + C * T / 2 + 4 * Co * K9, 2.0 * T * K9 * Co, cores=blas)
                timed("dact", lambda: oconv.conv3x3_dgrad_ref(gc, ga, out["w"][0], out["w"][1], True,
                                                              B, H, W, C, Co),
                      T * Co / 2 + K9 * Co / 2 + 4 * T * C, 2.0 * T * K9 * Co, cores=blas)
            reps += 1
        sample = f"the whole conv step, {reps} times (legs of the last)"
    elif workload == "small":
        # the whole layer step, repeated until at least 10 s of CPU work
        T, D, F = 256, 512, 512
        reps = 0
        while t_cpu < 10.0:
            legs.clear()
            out = {}
            timed("luq", lambda: out.update(g=oluq.luq_quantize(d["g"], R=4)), 2 * 4 * T * F + 2 * T * F / 2)
            timed("int4(a)", lambda: out.update(a=oint4.int4_quantize(d["a"], is_signed=False)),
                  2 * 4 * T * D + T * D / 2)
            timed("int4(W)", lambda: out.update(w=oint4.int4_quantize(d["W"], is_signed=True)),
                  2 * 4 * F * D + F * D / 2)
            gc, ga, _ = out["g"]
            timed("dX", lambda: ogemm.gemm_dgrad_ref(gc, ga, out["w"][0], out["w"][1], True, T, D, F),
                  T * F / 2 + D * F / 2 + 4 * T * D, 2.0 * T * D * F, cores=blas)
            timed("dW", lambda: ogemm.gemm_wgrad_ref(gc, ga, out["a"][0], out["a"][1], False, T, F, D),
                  F * T / 2 + D * T / 2 + 4 * F * D, 2.0 * T * D * F, cores=blas)
            reps += 1
        sample = f"the whole 256x512x512 layer step, {reps} times (legs of the last)"
    elif workload == "mlp_fwd":
        # INT4 of the whole activation over a process pool, and the forward
        # GEMM on 64 token rows with BLAS threads
        procs = max(1, min(POOL_MAX_PROCS, info["cores_available"]))
        x = d["x"].reshape(-1)
        F, D = d["W"].shape
        rows = 64
        xc, sx = oint4.int4_quantize(d["x"][:rows], dtype="bf16")
        wc, ws = oint4.int4_quantize(d["W"], is_signed=True)             # [F, D] = [N, K]
        _, t_int4 = pool_quantizers(x[: 8 * POOL_CHUNK], "bf16", procs)
        n = min(x.size, 8 * POOL_CHUNK)
        legs.append({"leg": f"int4 {n} bf16 elements, pool", "s": t_int4, "cores": procs,
                     "roof_s": (2 * 2 * n + n / 2) / HBM_PEAK})
        t_roof += (2 * 2 * n + n / 2) / HBM_PEAK
        t_cpu += t_int4
        while t_cpu < 10.0:
            timed(f"fwd {rows} rows", lambda: ogemm.gemm_fwd_ref(xc, sx, True, wc, ws, True, rows, F, D),
                  rows * D / 2 + 4 * rows * F, 2.0 * rows * D * F, cores=blas)
        sample = f"INT4 of {n} activation elements over a pool, then the forward GEMM on {rows} token rows"
    else:
        # the MLP backward: LUQ and INT4 of the whole 8192 x 16384 gradient
        # over a process pool (max pass, then encode, in 2^22-element tasks),
        # the same on one core for 2^20 elements, and dX on 64 token rows with
        # BLAS threads
        procs = max(1, min(POOL_MAX_PROCS, info["cores_available"]))
        g = d["g"].reshape(-1)
        n = g.size
        t_luq, t_int4 = pool_quantizers(g, "bf16", procs)
        for label, t, b in ((f"luq {n} bf16 elements, pool", t_luq, 2 * 2 * n + n / 2),
                            (f"int4 {n} bf16 elements, pool", t_int4, 2 * 2 * n + n / 2)):
            legs.append({"leg": label, "s": t, "cores": procs, "roof_s": b / HBM_PEAK})
            t_roof += b / HBM_PEAK
            t_cpu += t
        n1 = 1 << 20
        timed("luq 2^20 bf16, one core", lambda: oluq.luq_quantize(g[:n1], dtype="bf16", R=4),
              2 * 2 * n1 + n1 / 2, value=False)
        F = d["g"].shape[1]
        D = d["x"].shape[1]
        rows = 64
        gcodes, alpha, _ = oluq.luq_quantize(d["g"][:rows], dtype="bf16", R=4)
        wc, ws = oint4.int4_quantize(d["W"], is_signed=True)             # [F, D] = [K, N]
        while t_cpu < 12.0:
            timed(f"dgrad {rows} rows", lambda: ogemm.gemm_dgrad_ref(gcodes, alpha, wc, ws, True, rows, D, F),
                  rows * F / 2 + 4 * rows * D, 2.0 * rows * D * F, cores=blas)
        sample = (f"LUQ and INT4 of the whole {n}-element gradient over {procs} processes, "
                  f"LUQ of 2^20 elements on one core, dX on {rows} token rows")
    merged = {}
    for leg in legs:  # repeats of one leg are reported once, with their count
        m = merged.setdefault(leg["leg"], {"leg": leg["leg"], "s": 0.0, "roof_s": 0.0, "reps": 0,
                                           "cores": leg["cores"]})
        m["s"] += leg["s"]
        m["roof_s"] += leg["roof_s"]
        m["reps"] += 1
    legs = []
    for m in merged.values():
        legs.append({"leg": m["leg"], "reps": m["reps"], "s": round(m["s"], 3), "cores": m["cores"],
                     "pct_of_gpu_roofline": float(f"{100.0 * m['roof_s'] / m['s']:.3g}")})
    return {"value": 100.0 * t_roof / t_cpu, "unit": "% of MI355X roofline",
            "cores": max(leg["cores"] for leg in legs), "kind": "oracle", "sample": sample,
            "cpu_seconds": round(t_cpu, 3), "legs": legs, **info}


PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = {"luq_gemm_dgrad": "gemm_kernel.hpp", "luq_gemm_wgrad": "gemm_kernel.hpp",
                  "luq_conv3x3_dgrad": "conv.hip", "luq_conv3x3_wgrad": "conv.hip",
                  "int4_gemm_fwd": "gemm_kernel.hpp",
                  "luq_quantize_grad": "quant.hip", "int4_im2col3x3_t": "im2col.hip"}


def measured_traffic(kernel, workload):
    """HBM bytes per launch from the committed counter summary, if it was taken
    on the current kernel source (else None)."""
    import hashlib
    path = os.path.join(PROFILES, f"{kernel}_{workload}_traffic.md")
    src = KERNEL_SOURCES.get(kernel)
    if not src or not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line and line.strip().startswith("- "):
            k, v = line.strip()[2:].split(":", 1)
            fields[k.strip()] = v.strip().strip("`")
    h = hashlib.sha256(open(os.path.join(ROOT, "paper_2112_10769_amd", "csrc", src), "rb").read()).hexdigest()
    if fields.get("source_sha256") != h or "hbm_bytes_per_launch" not in fields:
        return None
    return float(fields["hbm_bytes_per_launch"])


def calibrate_copy(torch):
    n = 512 << 20
    src = torch.empty(n // 4, dtype=torch.float32, device="cuda:0").fill_(1.0)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibration": "device copy", "bytes_read": n, "bytes_written": n, "launches": 3}), flush=True)


def host_data(workload):
    """The workload's synthetic inputs on the host (seeded NumPy draws)."""
    import synth
    if workload in ("resnet", "resnet_lowered"):
        return synth.resnet()
    if workload == "small":
        return synth.small()
    return synth.mlp()


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build measures one GPU only; --gpus must be 1"}))
        sys.exit(2)
    # the CPU oracle runs first, before this process touches the GPU (its
    # worker processes are spawned fresh and use no GPU)
    if args.workload == "luq_sweep":
        cpu = None if args.no_cpu or args.calibrate_copy else cpu_sweep_baseline()
    elif not args.calibrate_copy:
        d = host_data(args.workload)
        cpu = None if args.no_cpu else cpu_baseline(
            args.workload if args.workload in ("resnet", "resnet_lowered", "mlp_fwd", "small") else "mlp", d)
    import torch
    if args.calibrate_copy:
        calibrate_copy(torch)
        return
    import paper_2112_10769_amd as L
    dev = torch.device("cuda:0")
    if args.workload == "luq_sweep":
        sizes = tuple(int(k) for k in args.sweep_log2.split(",")) if args.sweep_log2 else None
        rows, value, roof, cfg = run_sweep(L, torch, args.steps, sizes)
        out = {"metric": METRIC, "value": round(value, 2), "unit": "% of roofline", "n_gpus": 1,
               "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(roof["launch_us"] / 1e3, 4), "higher_is_better": True,
               "scaling": "weak", "vs_baseline": None, "dtype": "f32",
               "data": "synthetic", "config": cfg, "roofline": roof, "sweep": rows}
        if cpu:
            out["cpu_baseline"] = cpu
        out["paper_context"] = paper_context()
        print(json.dumps(out), flush=True)
        return
    if args.workload in ("resnet", "resnet_lowered"):
        stages, cfg, d = build_resnet(L, torch, dev, lowered=args.workload == "resnet_lowered", d=d)
    elif args.workload == "mlp_fwd":
        stages, cfg, d = build_mlp_fwd(L, torch, dev, d=d)
    elif args.workload == "small":
        stages, cfg, d = build_small(L, torch, dev, d=d)
    else:
        ns = {"mlp_smp": L.SMP_SUM | 2, "mlp_smp_planes": 2, "mlp_fp6": L.CARRIER_FP6 | 1}.get(args.workload, 1)
        stages, cfg, d = build_mlp(L, torch, dev, ns, d=d)
    step_s, per = time_stages(torch, stages, args.steps, args.warmup)
    roof_total = sum(s.roofline_s() for s in stages)
    kernels = {}
    for s in stages:
        t = per[s.name]
        kernels[s.name] = {"us": round(t * 1e6, 2), "GB/s": round(s.bytes / t / 1e9, 1),
                           "TOPS": round(s.ops / t / 1e12, 1) if s.ops else None,
                           "bound": s.bound(), "frac": round(s.roofline_s() / t, 4)}
    dom = max(stages, key=lambda s: per[s.name])
    t = per[dom.name]
    traffic = measured_traffic(dom.name, cfg["workload"])
    if dom.bound() == "hbm":
        roof = {"kernel": dom.name, "bound": "hbm", "achieved": round(dom.bytes / t / 1e9, 1), "peak": 8000.0,
                "unit": "GB/s", "frac": round(dom.bytes / t / HBM_PEAK, 4), "traffic": traffic}
    else:
        roof = {"kernel": dom.name, "bound": "mfma", "achieved": round(dom.ops / t / 1e12, 1),
                "peak": round(dom.peak / 1e12, 1), "unit": "TFLOP/s", "frac": round(dom.ops / t / dom.peak, 4),
                "traffic": traffic}
    roof["algorithmic_bytes"] = dom.bytes
    roof["launch_us"] = round(t * 1e6, 2)
    out = {
        "metric": METRIC_FWD if args.workload == "mlp_fwd" else METRIC,
        "value": round(100.0 * roof_total / step_s, 2), "unit": "% of roofline",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(step_s * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "i8",
        "data": "synthetic", "config": cfg, "roofline": roof, "kernels": kernels,
        "roofline_step_us": round(roof_total * 1e6, 2),
    }
    if cpu:
        out["cpu_baseline"] = cpu
    out["paper_context"] = paper_context()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

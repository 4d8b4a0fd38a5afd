"""Test-side helpers for the GPU parity tests (no method arithmetic here)."""
import sys

import numpy as np
import torch

from oracle.luq import unpack_nibbles, pack_nibbles

DEV = torch.device("cuda:0")


def announce(*what):
    """Names the case on stdout before a GPU step (flushed)."""
    print("[gpu case]", *what, flush=True)
    sys.stdout.flush()


def to_dev(a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:  # bfloat16 bit patterns
        return torch.from_numpy(a.view(np.int16)).to(DEV).view(torch.bfloat16)
    return torch.from_numpy(a).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def transpose_codes(codes, rows, cols):
    """Packed [rows][cols] nibbles -> packed [cols][rows] nibbles."""
    nib = unpack_nibbles(codes, rows * cols).reshape(rows, cols)
    return pack_nibbles(np.ascontiguousarray(nib.T).ravel())


def assert_codes_equal(gpu_bytes, ref_bytes, what=""):
    gpu_bytes = np.asarray(gpu_bytes, dtype=np.uint8).ravel()[: ref_bytes.size]
    ref_bytes = np.asarray(ref_bytes, dtype=np.uint8).ravel()
    bad = np.nonzero(gpu_bytes != ref_bytes)[0]
    assert bad.size == 0, f"{what}: {bad.size} bytes differ, first at {bad[:8]}: gpu {gpu_bytes[bad[:8]]} ref {ref_bytes[bad[:8]]}"


def assert_gemm_close(gpu, ref, absref, what=""):
    """|gpu - ref| <= 1e-5 * sum_k |a_k b_k| per output, exact zero where that sum is 0."""
    gpu = np.asarray(gpu, dtype=np.float64)
    err = np.abs(gpu - ref)
    tol = 1e-5 * absref
    bad = err > tol
    assert not bad.any(), f"{what}: {bad.sum()} outputs out of tolerance; worst rel {np.max(err / np.maximum(absref, 1e-300))}"
    assert np.all(gpu[absref == 0] == 0), f"{what}: nonzero output where every product is 0"


def epilogue_replica(acc_int, alpha, n_samples, scale):
    """fl32(fl32(acc) * fl32(fl32(alpha / n) * s)) from exact integer sums."""
    sc = np.float32(np.float32(np.float32(alpha) * np.float32(1.0 / n_samples)) * np.float32(scale))
    return (acc_int.astype(np.float64).astype(np.float32) * sc).astype(np.float32)

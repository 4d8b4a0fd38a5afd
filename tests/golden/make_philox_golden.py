"""Writes philox_rocrand.txt: Philox4x32-10 blocks from rocRAND (host build).

Run from the repository root:  python tests/golden/make_philox_golden.py
Needs hipcc and the rocRAND headers of a ROCm install.  The file pins the
oracle's generator; nothing in it comes from the oracle or the HIP library.
"""
import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))


def build(outdir):
    exe = os.path.join(outdir, "philox_rocrand_pin")
    subprocess.run(["hipcc", "-O1", "-x", "hip", "--offload-arch=gfx950",
                    "-I/opt/rocm/include", os.path.join(HERE, "philox_rocrand_pin.cpp"),
                    "-o", exe], check=True)
    return exe


def cases():
    # rocRAND takes the block index as offset = 4*blk in 64 bits, so blk < 2^62
    out = [(0, 0, 0, 0), (0, 1, 0, 0), (0xFFFFFFFFFFFFFFFF, (1 << 62) - 1, 0xFFFFFFFF, 0xFFFFFFFF)]
    x = 0x243F6A8885A308D3  # digits of pi, as a fixed pseudo-random walk
    for _ in range(61):
        x = (x * 6364136223846793005 + 1442695040888963407) & 0xFFFFFFFFFFFFFFFF
        seed = x
        x = (x * 6364136223846793005 + 1442695040888963407) & 0xFFFFFFFFFFFFFFFF
        blk = (x >> (x & 31)) & ((1 << 62) - 1)
        s = (x >> 8) & 1
        c = (x >> 16) & 0xFFFFFFFF
        out.append((seed, blk, s, c))
    return out


def run(exe, items):
    inp = "".join("%x %x %x %x\n" % c for c in items)
    res = subprocess.run([exe], input=inp, capture_output=True, text=True, check=True)
    return res.stdout


if __name__ == "__main__":
    with tempfile.TemporaryDirectory() as d:
        txt = run(build(d), cases())
    with open(os.path.join(HERE, "philox_rocrand.txt"), "w") as f:
        f.write("# Philox4x32-10 (rocRAND header engine, host build): seed blk s c -> y0 y1 y2 y3\n")
        f.write(txt)
    sys.exit(0)

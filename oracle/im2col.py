"""3x3 convolution lowering (im2col) on packed 4-bit codes -- oracle.

Test infrastructure only.  The ResNet-style workload writes the weight
gradient of a 3x3 convolution (stride 1, zero padding 1) as the update GEMM
of Eq. update: dW[Cout, 9*Cin] = Q(g)^T Q(a_col), with a_col the lowered
activations.  Rows of a_col are output pixels (b, y, x) in row-major order;
columns are (kh, kw, c) in that order.  Out-of-image taps are zero, which is
code 0 for both INT4 code sets.  Plain loops over the nine taps.
"""

import numpy as np

from .luq import unpack_nibbles, pack_nibbles


def im2col3x3_codes(codes, B, H, W, C):
    """codes: packed NHWC [B, H, W, C] nibbles -> packed [B*H*W, 9*C] nibbles."""
    nib = unpack_nibbles(codes, B * H * W * C).reshape(B, H, W, C)
    padded = np.zeros((B, H + 2, W + 2, C), dtype=np.uint8)
    padded[:, 1:H + 1, 1:W + 1, :] = nib
    out = np.zeros((B, H, W, 3, 3, C), dtype=np.uint8)
    for kh in range(3):
        for kw in range(3):
            out[:, :, :, kh, kw, :] = padded[:, kh:kh + H, kw:kw + W, :]
    return pack_nibbles(out.reshape(B * H * W, 9 * C).ravel())

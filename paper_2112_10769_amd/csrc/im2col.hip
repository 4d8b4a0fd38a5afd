// 3x3 / stride 1 / zero-pad 1 convolution lowering on packed INT4 codes,
// written transposed ([9*C][T], tokens innermost) so that the update GEMM
// dW = Q(g)^T Q(a_col) (Eq. update) reads both operands K-major.
//
// General path: one lane produces one output word, 8 consecutive tokens t of
// one column (kh, kw, c), gathered nibble by nibble from the NHWC codes.
#include "luq_device.hpp"
#include "luq_launch.hpp"

namespace luq {

__global__ __launch_bounds__(256) void im2col3x3_t_kernel(const uint8_t* __restrict__ act, int B,
                                                         int H, int W, int C,
                                                         uint8_t* __restrict__ col_t) {
  const int64_t T = (int64_t)B * H * W;
  const int64_t words_per_row = T >> 3;
  const int64_t total = words_per_row * 9 * C;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t krow = idx / words_per_row;
    const int64_t t0 = (idx - krow * words_per_row) * 8;
    const int c = (int)(krow % C);
    const int tap = (int)(krow / C);
    const int dy = tap / 3 - 1, dx = tap % 3 - 1;
    uint32_t word = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int64_t t = t0 + e;
      const int x = (int)(t % W);
      const int64_t by = t / W;
      const int y = (int)(by % H);
      const int b = (int)(by / H);
      const int ys = y + dy, xs = x + dx;
      uint32_t nib = 0;
      if (ys >= 0 && ys < H && xs >= 0 && xs < W) {
        const int64_t src = (((int64_t)b * H + ys) * W + xs) * C + c;
        nib = (act[src >> 1] >> ((src & 1) * 4)) & 0xFu;
      }
      word |= nib << (4 * e);
    }
    *reinterpret_cast<uint32_t*>(col_t + krow * (T >> 1) + (t0 >> 1)) = word;
  }
}

// Fast path for C % 8 == 0 and W % 8 == 0: a lane loads the 8 channels
// (one word) of 8 consecutive pixels of a row for one tap, transposes the 8x8
// nibble block in registers and writes 8 words, one per channel row of
// col_t.  Lanes of a wave take consecutive pixel groups, so each store
// instruction writes contiguous bytes of one row.
__global__ __launch_bounds__(256) void im2col3x3_t_fast_kernel(const uint8_t* __restrict__ act, int B,
                                                              int H, int W, int C,
                                                              uint8_t* __restrict__ col_t) {
  const int64_t T = (int64_t)B * H * W;
  const int64_t groups = T >> 3;  // pixel groups of 8 along x
  const int cg = C >> 3;          // channel groups of 8
  const int64_t total = groups * 9 * cg;
  const int W8 = W >> 3;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t grp = idx % groups;
    const int64_t rest = idx / groups;
    const int c8 = (int)(rest % cg);
    const int tap = (int)(rest / cg);
    const int dy = tap / 3 - 1, dx = tap % 3 - 1;
    const int x0 = (int)(grp % W8) * 8;
    const int64_t by = grp / W8;
    const int y = (int)(by % H);
    const int b = (int)(by / H);
    const int ys = y + dy;
    uint32_t r[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int xs = x0 + e + dx;
      r[e] = 0;
      if (ys >= 0 && ys < H && xs >= 0 && xs < W)
        r[e] = *reinterpret_cast<const uint32_t*>(act + ((((int64_t)b * H + ys) * W + xs) * C >> 1) + c8 * 4);
    }
    transpose8x8_nibbles(r);
    const int64_t t0 = ((int64_t)b * H + y) * W + x0;
    uint8_t* dst = col_t + ((int64_t)tap * C + c8 * 8) * (T >> 1) + (t0 >> 1);
#pragma unroll
    for (int c = 0; c < 8; ++c) *reinterpret_cast<uint32_t*>(dst + c * (T >> 1)) = r[c];
  }
}

hipError_t launch_im2col3x3_t(const uint8_t* act, int64_t B, int64_t H, int64_t W, int64_t C,
                              uint8_t* col_t, hipStream_t st) {
  const int64_t total = (B * H * W / 8) * 9 * C;
  if (total == 0) return hipSuccess;
  if ((C & 7) == 0 && (W & 7) == 0) {
    const int64_t lanes = total / 8;
    int64_t nb = (lanes + 255) / 256;
    if (nb > 65536) nb = 65536;
    hipLaunchKernelGGL(im2col3x3_t_fast_kernel, dim3((unsigned)nb), dim3(256), 0, st, act, (int)B,
                       (int)H, (int)W, (int)C, col_t);
    return hipGetLastError();
  }
  int64_t nb = (total + 255) / 256;
  if (nb > 16384) nb = 16384;
  hipLaunchKernelGGL(im2col3x3_t_kernel, dim3((unsigned)nb), dim3(256), 0, st, act, (int)B, (int)H,
                     (int)W, (int)C, col_t);
  return hipGetLastError();
}

}  // namespace luq

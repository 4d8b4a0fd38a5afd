// 3x3 / stride 1 / zero-pad 1 convolution lowering on packed INT4 codes,
// written transposed ([9*C][T], tokens innermost) so that the update GEMM
// dW = Q(g)^T Q(a_col) (Eq. update) reads both operands K-major.
//
// One lane produces one output word: 8 consecutive tokens t of one column
// (kh, kw, c).  Tokens are gathered nibble by nibble from the NHWC codes,
// which stay cache resident (the codes are 1/8 the size of the float input).
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

hipError_t launch_im2col3x3_t(const uint8_t* act, int64_t B, int64_t H, int64_t W, int64_t C,
                              uint8_t* col_t, hipStream_t st) {
  const int64_t total = (B * H * W / 8) * 9 * C;
  if (total == 0) return hipSuccess;
  int64_t nb = (total + 255) / 256;
  if (nb > 16384) nb = 16384;
  hipLaunchKernelGGL(im2col3x3_t_kernel, dim3((unsigned)nb), dim3(256), 0, st, act, (int)B, (int)H,
                     (int)W, (int)C, col_t);
  return hipGetLastError();
}

}  // namespace luq

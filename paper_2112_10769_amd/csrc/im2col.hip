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

// Fast path for C % 8 == 0 and W % 8 == 0.  A lane owns one channel group
// (8 channels, one code word per pixel) of 8 consecutive pixels of one image
// row, for the three taps of one kernel row dy: it loads the 10 words of
// input row y + dy that the taps read (x0-1 .. x0+8; words outside the image
// read as zero codes), and for each dx transposes the 8x8 nibble block
// (pixel x channel) into 8 column words, one per channel row of col_t.
// Consecutive lanes take consecutive channel groups of a pixel group, so a
// load instruction reads whole 32-byte pixels and a store instruction writes
// 32 contiguous bytes into each of 8 rows.  Integer index math is 32-bit and
// done once per lane.
__global__ __launch_bounds__(256) void im2col3x3_t_fast_kernel(const uint8_t* __restrict__ act,
                                                              int B, int H, int W, int C,
                                                              uint8_t* __restrict__ col_t) {
  const int cg = C >> 3, W8 = W >> 3;
  const uint32_t lanes = (uint32_t)B * H * W8 * cg;
  const uint32_t i = blockIdx.x * 256u + threadIdx.x;
  if (i >= lanes) return;
  const int dy = (int)blockIdx.y - 1;
  const uint32_t grp = i / cg;
  const int c8 = (int)(i - grp * cg);
  const uint32_t by = grp / W8;
  const int x0 = (int)(grp - by * W8) * 8;
  const int y = (int)(by % H);
  const int ys = y + dy;
  const bool row_ok = ys >= 0 && ys < H;
  const int64_t T = (int64_t)B * H * W;
  // word index of pixel (b, ys, x0 - 1), channel group c8: the pixel index is
  // b * H * W + ys * W + x0 - 1 = (by + dy) * W + x0 - 1 (all below 2^31 / cg)
  const int base = (((int)by + dy) * W + x0 - 1) * cg + c8;
  const uint32_t* src = reinterpret_cast<const uint32_t*>(act);
  uint32_t v[10];
#pragma unroll
  for (int k = 0; k < 10; ++k) {
    const int xs = x0 - 1 + k;
    const bool ok = row_ok && xs >= 0 && xs < W;
    const uint32_t w = src[ok ? base + k * cg : 0];  // a valid address even where the value is unused
    v[k] = ok ? w : 0u;
  }
  const int64_t t0 = by * (int64_t)W + x0;
#pragma unroll
  for (int dx = 0; dx < 3; ++dx) {
    uint32_t r[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) r[e] = v[e + dx];
    transpose8x8_nibbles(r);
    const int tap = (dy + 1) * 3 + dx;
    uint8_t* dst = col_t + ((int64_t)tap * C + c8 * 8) * (T >> 1) + (t0 >> 1);
#pragma unroll
    for (int c = 0; c < 8; ++c) *reinterpret_cast<uint32_t*>(dst + c * (T >> 1)) = r[c];
  }
}

hipError_t launch_im2col3x3_t(const uint8_t* act, int64_t B, int64_t H, int64_t W, int64_t C,
                              uint8_t* col_t, hipStream_t st) {
  const int64_t total = (B * H * W / 8) * 9 * C;
  if (total == 0) return hipSuccess;
  // the fast kernel indexes input words in 32 bits
  if ((C & 7) == 0 && (W & 7) == 0 && B * H * W * (C >> 3) < (1LL << 31)) {
    const int64_t lanes = B * H * (W >> 3) * (C >> 3);
    const int64_t nb = (lanes + 255) / 256;
    hipLaunchKernelGGL(im2col3x3_t_fast_kernel, dim3((unsigned)nb, 3), dim3(256), 0, st, act, (int)B,
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

// Internal launchers behind the C ABI (host side).  Arguments are already
// validated by the ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace luq {

// Sample-count argument meaning two SMP samples stored as one int8 sum per
// element (LUQ_SMP_SUM | 2 in the C ABI).
constexpr int kSmpSum = 0x12;

// ceil(n/2) rounded up to 256 bytes: the distance between SMP planes.
inline size_t plane_bytes(int64_t n) {
  const size_t b = (size_t)((n + 1) / 2);
  return (b + 255) & ~(size_t)255;
}

size_t quant_workspace_bytes(int64_t n);
// Byte offset, in a quantizer's workspace, of the status word of its last
// call: kStatusTag | luq_status, so that a word no quantizer wrote is told
// apart.
size_t quant_status_offset();
constexpr uint32_t kStatusTag = 0x4C510000u;
constexpr uint32_t kStatusTagMask = 0xFFFF0000u;

hipError_t launch_luq_quantize(const void* g, int bf16, int64_t rows, int64_t cols, int R, int pw2,
                               uint64_t seed, uint32_t counter, int ns, uint8_t* codes,
                               uint8_t* codes_t, float* alpha, float* maxabs, void* ws,
                               hipStream_t st);

// luq_quantize_grad with its workspace in the library's per-device static
// scratch array (no allocation); noalloc_scratch_bytes() is that array's size.
size_t noalloc_scratch_bytes();
hipError_t launch_luq_quantize_noalloc(const void* g, int bf16, int64_t rows, int64_t cols, int R, int pw2,
                                       uint64_t seed, uint32_t counter, int ns, uint8_t* codes, uint8_t* codes_t,
                                       float* alpha, float* maxabs, hipStream_t st);

hipError_t launch_luq_quantize_hindsight(const void* g, int bf16, int64_t rows, int64_t cols, int R, int pw2,
                                         uint64_t seed, uint32_t counter, int ns, float eta, uint8_t* codes,
                                         uint8_t* codes_t, float* state, float* alpha, float* maxabs, void* ws,
                                         hipStream_t st);

hipError_t launch_int4_quantize(const void* x, int bf16, int64_t rows, int64_t cols, int is_signed,
                                float clip, uint8_t* codes, uint8_t* codes_t, float* scale,
                                void* ws, hipStream_t st);

// C[m][n] = (alpha / ns) * bscale * sum_k A[m][k] * B[n][k] with A LUQ codes
// (ns planes, plane stride a_plane) and B INT4 codes, both K-major.
size_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K, int ns);
hipError_t launch_gemm_luq_int4(const uint8_t* A, int64_t a_plane, int ns, const float* alpha,
                                const uint8_t* B, const float* bscale, int b_signed, int64_t M,
                                int64_t N, int64_t K, float* C, void* ws, size_t ws_bytes,
                                hipStream_t st);

// The same product on the FP6 carrier (one sample): the codes are converted
// once into fragment-major FP6 blocks in the workspace, then multiplied with
// the scaled f8f6f4 MFMA; bit-identical to launch_gemm_luq_int4.
constexpr int kCarrierFp6 = 0x40;
size_t gemm_fp6_workspace_bytes(int64_t M, int64_t N, int64_t K);
bool gemm_fp6_fits(int64_t M, int64_t N, int64_t K);
hipError_t launch_gemm_luq_int4_fp6(const uint8_t* A, const float* alpha, const uint8_t* B, const float* bscale,
                                    int b_signed, int64_t M, int64_t N, int64_t K, float* C, void* ws,
                                    hipStream_t st);

// y[m][n] = x_scale * w_scale * sum_k X[m][k] * W[n][k], INT4 codes, K-major.
size_t gemm_fwd_workspace_bytes(int64_t M, int64_t N, int64_t K);
hipError_t launch_gemm_int4_fwd(const uint8_t* X, const float* x_scale, int x_signed, const uint8_t* W,
                                const float* w_scale, int w_signed, int64_t M, int64_t N, int64_t K, float* Y,
                                void* ws, hipStream_t st);

// dact[t][c] of a 3x3 / stride 1 / pad 1 convolution from LUQ codes of g
// [T][Cout] (ns planes) and INT4 codes of W transposed [9*C][Cout].
int conv3x3_max_width();
hipError_t launch_conv3x3_dgrad(const uint8_t* g, int64_t g_plane, int ns, const float* alpha, const uint8_t* w,
                                const float* wscale, int w_signed, int64_t B, int64_t H, int64_t W, int64_t C,
                                int64_t Cout, float* dact, hipStream_t st);

// dW [Cout][9*C] of the same convolution from LUQ codes of g transposed
// [Cout][T] (ns planes) and INT4 codes of the activations transposed [C][T].
size_t conv3x3_wgrad_workspace_bytes(int64_t T, int64_t C, int64_t Cout);
int64_t conv3x3_wgrad_blocks(int64_t T, int64_t C, int64_t Cout);
hipError_t launch_conv3x3_wgrad(const uint8_t* g, int64_t g_plane, int ns, const float* alpha, const uint8_t* act,
                                const float* ascale, int a_signed, int64_t B, int64_t H, int64_t W, int64_t C,
                                int64_t Cout, float* dw, void* ws, hipStream_t st);

hipError_t launch_im2col3x3_t(const uint8_t* act, int64_t B, int64_t H, int64_t W, int64_t C,
                              uint8_t* col_t, hipStream_t st);

}  // namespace luq

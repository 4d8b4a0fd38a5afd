// extern "C" entry points of libluq: argument validation on the host, then
// launches on the caller's stream.  Nothing is enqueued when validation
// fails.  See include/luq.h for the contract of every function.
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "../../include/luq.h"
#include "luq_launch.hpp"

static_assert(LUQ_CARRIER_FP6 == luq::kCarrierFp6, "carrier flag");

namespace {

thread_local char g_last_error[256] = "";

luq_status fail(luq_status st, const char* fmt, const char* what) {
  snprintf(g_last_error, sizeof(g_last_error), fmt, what);
  return st;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
bool aligned4(const void* p) { return ((uintptr_t)p & 3u) == 0; }

luq_status hip_status(hipError_t e) {
  if (e == hipSuccess) return LUQ_OK;
  return fail(LUQ_ERR_HIP, "HIP launch failed: %s", hipGetErrorString(e));
}

bool mul_overflows(int64_t a, int64_t b) { return a > 0 && b > INT64_MAX / a; }

luq_status check_matrix(int64_t rows, int64_t cols, bool transposed, const char* name) {
  if (rows < 0 || cols < 0) return fail(LUQ_ERR_SHAPE, "%s: negative size", name);
  if (mul_overflows(rows, cols)) return fail(LUQ_ERR_SHAPE, "%s: size overflows", name);
  if (rows > 1 && (cols & 1)) return fail(LUQ_ERR_SHAPE, "%s: cols must be even when rows > 1", name);
  if (transposed && ((rows & 7) || (cols & 7)))
    return fail(LUQ_ERR_SHAPE, "%s: the transposed layout needs rows and cols multiples of 8", name);
  return LUQ_OK;
}

// n_samples of the LUQ entry points: 1, 2, or LUQ_SMP_SUM | 2 (the two
// samples stored as int8 sums); two samples need R <= 5.
luq_status check_samples(int n_samples, int R, const char* name) {
  if (n_samples != 1 && n_samples != 2 && n_samples != (LUQ_SMP_SUM | 2))
    return fail(LUQ_ERR_PARAM, "%s: n_samples must be 1, 2 or LUQ_SMP_SUM | 2", name);
  if (n_samples != 1 && R > 5) return fail(LUQ_ERR_PARAM, "%s: two samples need R <= 5", name);
  return LUQ_OK;
}

}  // namespace

extern "C" {

int luq_abi_version(void) { return LUQ_ABI_VERSION; }

const char* luq_status_string(luq_status s) {
  switch (s) {
    case LUQ_OK: return "ok";
    case LUQ_ERR_NULL: return "required pointer is NULL";
    case LUQ_ERR_SHAPE: return "invalid shape";
    case LUQ_ERR_DTYPE: return "unknown dtype";
    case LUQ_ERR_PARAM: return "parameter out of range";
    case LUQ_ERR_WORKSPACE: return "workspace missing or too small";
    case LUQ_ERR_ALIGN: return "pointer not 16-byte aligned";
    case LUQ_ERR_HIP: return "HIP runtime error";
    case LUQ_ERR_NONFINITE: return "input tensor has a non-finite element";
    default: return "unknown status";
  }
}

const char* luq_last_error(void) { return g_last_error; }

luq_status luq_query_status(const void* ws, void* stream) {
  g_last_error[0] = 0;
  if (!ws) return fail(LUQ_ERR_NULL, "%s: ws is NULL", "luq_query_status");
  if (!aligned16(ws)) return fail(LUQ_ERR_ALIGN, "%s: ws must be 16-byte aligned", "luq_query_status");
  const hipStream_t st = static_cast<hipStream_t>(stream);
  uint32_t word = 0;
  hipError_t e = hipMemcpyAsync(&word, static_cast<const uint8_t*>(ws) + luq::quant_status_offset(),
                                sizeof(word), hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_status(e);
  if ((word & luq::kStatusTagMask) != luq::kStatusTag)
    return fail(LUQ_ERR_WORKSPACE, "%s: the workspace holds no quantizer status", "luq_query_status");
  const luq_status s = (luq_status)(word & 0xFFFFu);
  if (s == LUQ_ERR_NONFINITE) return fail(LUQ_ERR_NONFINITE, "%s: the last quantized tensor was not finite",
                                          "luq_query_status");
  return s;
}

size_t luq_plane_bytes(int64_t n) { return n <= 0 ? 0 : luq::plane_bytes(n); }

size_t luq_workspace_size(int op, int64_t d0, int64_t d1, int64_t d2) {
  switch (op) {
    case LUQ_OP_QUANTIZE_GRAD:
    case LUQ_OP_INT4_QUANTIZE:
      return d0 > 0 ? luq::quant_workspace_bytes(d0) : 0;
    case LUQ_OP_GEMM_DGRAD:
      return (d0 > 0 && d1 > 0 && d2 > 0) ? luq::gemm_workspace_bytes(d0, d1, d2, 1) : 0;
    case LUQ_OP_GEMM_WGRAD:
      return (d0 > 0 && d1 > 0 && d2 > 0) ? luq::gemm_workspace_bytes(d1, d2, d0, 1) : 0;
    case LUQ_OP_GEMM_FWD:
      return (d0 > 0 && d1 > 0 && d2 > 0) ? luq::gemm_fwd_workspace_bytes(d0, d1, d2) : 0;
    case LUQ_OP_GEMM_DGRAD_FP6:
      return (d0 > 0 && d1 > 0 && d2 > 0) ? luq::gemm_fp6_workspace_bytes(d0, d1, d2) : 0;
    case LUQ_OP_GEMM_WGRAD_FP6:
      return (d0 > 0 && d1 > 0 && d2 > 0) ? luq::gemm_fp6_workspace_bytes(d1, d2, d0) : 0;
    case LUQ_OP_CONV_WGRAD:
      return (d0 > 0 && d1 > 0 && d2 > 0 && d0 < ((int64_t)1 << 31) && d1 < ((int64_t)1 << 28) &&
              d2 < ((int64_t)1 << 28))
                 ? luq::conv3x3_wgrad_workspace_bytes(d0, d1, d2)
                 : 0;
    default:
      return 0;
  }
}

// Checks of luq_quantize_grad's arguments other than the workspace; R loses
// the LUQ_ALPHA_PW2 flag, which goes to *pw2.
static luq_status quantize_grad_checks(const char* fn, const void* g, luq_dtype dt, int64_t rows, int64_t cols,
                                       int* R, int* pw2, int n_samples, const uint8_t* codes,
                                       const uint8_t* codes_t, const float* alpha, const float* maxabs) {
  if (dt != LUQ_F32 && dt != LUQ_BF16) return fail(LUQ_ERR_DTYPE, "%s: dtype", fn);
  luq_status st = check_matrix(rows, cols, codes_t != nullptr, fn);
  if (st != LUQ_OK) return st;
  *pw2 = (*R & LUQ_ALPHA_PW2) ? 1 : 0;
  *R &= ~LUQ_ALPHA_PW2;
  if (*R < 4 || *R > 6) return fail(LUQ_ERR_PARAM, "%s: R must be 4, 5 or 6", fn);
  st = check_samples(n_samples, *R, fn);
  if (st != LUQ_OK) return st;
  if (!alpha) return fail(LUQ_ERR_NULL, "%s: alpha is NULL", fn);
  if (rows * cols > 0) {
    if (!g) return fail(LUQ_ERR_NULL, "%s: g is NULL", fn);
    if (!codes && !codes_t) return fail(LUQ_ERR_NULL, "%s: no code output", fn);
    if (!aligned16(g) || !aligned16(codes) || !aligned16(codes_t))
      return fail(LUQ_ERR_ALIGN, "%s: g, codes and codes_t must be 16-byte aligned", fn);
  }
  if (!aligned4(alpha) || !aligned4(maxabs)) return fail(LUQ_ERR_ALIGN, "%s: alpha / maxabs misaligned", fn);
  return LUQ_OK;
}

luq_status luq_quantize_grad(const void* g, luq_dtype dt, int64_t rows, int64_t cols, int R,
                             uint64_t seed, uint32_t counter, int n_samples, uint8_t* codes,
                             uint8_t* codes_t, float* alpha, float* maxabs, void* ws,
                             size_t ws_bytes, void* stream) {
  const char* fn = "luq_quantize_grad";
  g_last_error[0] = 0;
  int pw2 = 0;
  const luq_status st = quantize_grad_checks(fn, g, dt, rows, cols, &R, &pw2, n_samples, codes, codes_t, alpha,
                                             maxabs);
  if (st != LUQ_OK) return st;
  if (rows * cols > 0) {
    if (!ws || ws_bytes < luq_workspace_size(LUQ_OP_QUANTIZE_GRAD, rows * cols, 0, 0))
      return fail(LUQ_ERR_WORKSPACE, "%s: workspace too small", fn);
    if (!aligned16(ws)) return fail(LUQ_ERR_ALIGN, "%s: ws must be 16-byte aligned", fn);
  }
  return hip_status(luq::launch_luq_quantize(g, dt == LUQ_BF16, rows, cols, R, pw2, seed, counter,
                                             n_samples, codes, codes_t, alpha, maxabs, ws,
                                             static_cast<hipStream_t>(stream)));
}

luq_status luq_quantize_grad_noalloc(const void* g, luq_dtype dt, int64_t rows, int64_t cols, int R,
                                     uint64_t seed, uint32_t counter, int n_samples, uint8_t* codes,
                                     uint8_t* codes_t, float* alpha, float* maxabs, void* stream) {
  const char* fn = "luq_quantize_grad_noalloc";
  g_last_error[0] = 0;
  int pw2 = 0;
  const luq_status st = quantize_grad_checks(fn, g, dt, rows, cols, &R, &pw2, n_samples, codes, codes_t, alpha,
                                             maxabs);
  if (st != LUQ_OK) return st;
  if (luq_workspace_size(LUQ_OP_QUANTIZE_GRAD, rows * cols, 0, 0) > luq::noalloc_scratch_bytes())
    return fail(LUQ_ERR_SHAPE, "%s: the tensor needs more scratch than the library's static array holds", fn);
  return hip_status(luq::launch_luq_quantize_noalloc(g, dt == LUQ_BF16, rows, cols, R, pw2, seed, counter,
                                                     n_samples, codes, codes_t, alpha, maxabs,
                                                     static_cast<hipStream_t>(stream)));
}

luq_status luq_quantize_grad_hindsight(const void* g, luq_dtype dt, int64_t rows, int64_t cols, int R,
                                       uint64_t seed, uint32_t counter, int n_samples, float eta,
                                       uint8_t* codes, uint8_t* codes_t, float* state, float* alpha,
                                       float* maxabs, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "luq_quantize_grad_hindsight";
  g_last_error[0] = 0;
  if (dt != LUQ_F32 && dt != LUQ_BF16) return fail(LUQ_ERR_DTYPE, "%s: dtype", fn);
  luq_status st = check_matrix(rows, cols, codes_t != nullptr, fn);
  if (st != LUQ_OK) return st;
  const int pw2 = (R & LUQ_ALPHA_PW2) ? 1 : 0;
  R &= ~LUQ_ALPHA_PW2;
  if (R < 4 || R > 6) return fail(LUQ_ERR_PARAM, "%s: R must be 4, 5 or 6", fn);
  st = check_samples(n_samples, R, fn);
  if (st != LUQ_OK) return st;
  if (!(eta >= 0.0f && eta <= 1.0f)) return fail(LUQ_ERR_PARAM, "%s: eta must be in [0, 1]", fn);
  if (!alpha) return fail(LUQ_ERR_NULL, "%s: alpha is NULL", fn);
  if (!state) return fail(LUQ_ERR_NULL, "%s: state is NULL", fn);
  const int64_t n = rows * cols;
  if (n > 0) {
    if (!g) return fail(LUQ_ERR_NULL, "%s: g is NULL", fn);
    if (!codes && !codes_t) return fail(LUQ_ERR_NULL, "%s: no code output", fn);
    if (!ws || ws_bytes < luq_workspace_size(LUQ_OP_QUANTIZE_GRAD, n, 0, 0))
      return fail(LUQ_ERR_WORKSPACE, "%s: workspace too small", fn);
    if (!aligned16(g) || !aligned16(codes) || !aligned16(codes_t) || !aligned16(ws))
      return fail(LUQ_ERR_ALIGN, "%s: g, codes, codes_t and ws must be 16-byte aligned", fn);
  }
  if (!aligned4(alpha) || !aligned4(maxabs) || !aligned4(state))
    return fail(LUQ_ERR_ALIGN, "%s: alpha / maxabs / state misaligned", fn);
  return hip_status(luq::launch_luq_quantize_hindsight(g, dt == LUQ_BF16, rows, cols, R, pw2, seed, counter, n_samples,
                                                       eta, codes, codes_t, state, alpha, maxabs, ws,
                                                       static_cast<hipStream_t>(stream)));
}

luq_status int4_quantize(const void* x, luq_dtype dt, int64_t rows, int64_t cols, int is_signed,
                         float clip, uint8_t* codes, uint8_t* codes_t, float* scale, void* ws,
                         size_t ws_bytes, void* stream) {
  g_last_error[0] = 0;
  if (dt != LUQ_F32 && dt != LUQ_BF16) return fail(LUQ_ERR_DTYPE, "%s: dtype", "int4_quantize");
  luq_status st = check_matrix(rows, cols, codes_t != nullptr, "int4_quantize");
  if (st != LUQ_OK) return st;
  if (!(clip == clip) || clip == __builtin_inff())
    return fail(LUQ_ERR_PARAM, "%s: clip must be finite", "int4_quantize");
  if (!scale) return fail(LUQ_ERR_NULL, "%s: scale is NULL", "int4_quantize");
  const int64_t n = rows * cols;
  if (n > 0) {
    if (!x) return fail(LUQ_ERR_NULL, "%s: x is NULL", "int4_quantize");
    if (!codes && !codes_t) return fail(LUQ_ERR_NULL, "%s: no code output", "int4_quantize");
    if (clip <= 0.0f && (!ws || ws_bytes < luq_workspace_size(LUQ_OP_INT4_QUANTIZE, n, 0, 0)))
      return fail(LUQ_ERR_WORKSPACE, "%s: workspace too small", "int4_quantize");
    if (!aligned16(x) || !aligned16(codes) || !aligned16(codes_t) || !aligned16(ws))
      return fail(LUQ_ERR_ALIGN, "%s: x, codes, codes_t and ws must be 16-byte aligned",
                  "int4_quantize");
  }
  if (!aligned4(scale)) return fail(LUQ_ERR_ALIGN, "%s: scale misaligned", "int4_quantize");
  return hip_status(luq::launch_int4_quantize(x, dt == LUQ_BF16, rows, cols, is_signed ? 1 : 0,
                                              clip, codes, codes_t, scale, ws,
                                              static_cast<hipStream_t>(stream)));
}

// Checks shared by the three GEMMs; need = the workspace the call requires.
static luq_status gemm_checks(const char* name, const uint8_t* A, const float* alpha, const uint8_t* B,
                              const float* bscale, int64_t M, int64_t N, int64_t K, const float* C, size_t need,
                              const void* ws, size_t ws_bytes) {
  if (!A || !alpha || !B || !bscale || !C) return fail(LUQ_ERR_NULL, "%s: NULL operand", name);
  if (need && (!ws || ws_bytes < need)) return fail(LUQ_ERR_WORKSPACE, "%s: workspace too small", name);
  if (!aligned16(A) || !aligned16(B) || !aligned16(ws) || !aligned4(C) || !aligned4(alpha) ||
      !aligned4(bscale))
    return fail(LUQ_ERR_ALIGN, "%s: code operands and ws must be 16-byte aligned", name);
  return LUQ_OK;
}

// a_bytes_per_k: 1 for an int8 A operand (summed SMP samples), else codes
// (half a byte).  Code operands are addressed with 32-bit offsets, so each
// must stay below 2 GiB with a tile's worth of rows to spare.
static luq_status gemm_shape(const char* name, int64_t M, int64_t N, int64_t K, int a_bytes_per_k = 0) {
  if (M < 1 || N < 1 || K < 32 || (K & 31))
    return fail(LUQ_ERR_SHAPE, "%s: need M, N >= 1 and K a positive multiple of 32", name);
  if (mul_overflows(M, N) || mul_overflows(M, K) || mul_overflows(N, K))
    return fail(LUQ_ERR_SHAPE, "%s: size overflows", name);
  if (M > INT32_MAX / 2 || N > INT32_MAX / 2)
    return fail(LUQ_ERR_SHAPE, "%s: M and N must be below 2^30", name);
  const int64_t lim = ((int64_t)1 << 31) - ((int64_t)1 << 20);
  const int64_t a_bytes = a_bytes_per_k ? (M + 256) * K : (M + 256) * (K / 2);
  if (a_bytes >= lim || (N + 256) * (K / 2) >= lim)
    return fail(LUQ_ERR_SHAPE, "%s: a code operand reaches 2 GiB", name);
  return LUQ_OK;
}

static luq_status gemm_common(const char* name, const uint8_t* A, const float* alpha, int ns,
                              const uint8_t* B, const float* bscale, int b_signed, int64_t M,
                              int64_t N, int64_t K, float* C, void* ws, size_t ws_bytes,
                              void* stream) {
  if (!A || !alpha || !B || !bscale || !C) return fail(LUQ_ERR_NULL, "%s: NULL operand", name);
  if (ns & LUQ_CARRIER_FP6) {
    if (ns != (LUQ_CARRIER_FP6 | 1))
      return fail(LUQ_ERR_PARAM, "%s: the FP6 carrier takes one sample (n_samples = LUQ_CARRIER_FP6 | 1)", name);
    luq_status st = gemm_shape(name, M, N, K);
    if (st != LUQ_OK) return st;
    if (!luq::gemm_fp6_fits(M, N, K)) return fail(LUQ_ERR_SHAPE, "%s: an FP6 operand reaches 2 GiB", name);
    st = gemm_checks(name, A, alpha, B, bscale, M, N, K, C, luq::gemm_fp6_workspace_bytes(M, N, K), ws, ws_bytes);
    if (st != LUQ_OK) return st;
    return hip_status(luq::launch_gemm_luq_int4_fp6(A, alpha, B, bscale, b_signed ? 1 : 0, M, N, K, C, ws,
                                                    static_cast<hipStream_t>(stream)));
  }
  if (ns != 1 && ns != 2 && ns != (LUQ_SMP_SUM | 2))
    return fail(LUQ_ERR_PARAM, "%s: n_samples must be 1, 2 or LUQ_SMP_SUM | 2", name);
  luq_status st = gemm_shape(name, M, N, K, ns == (LUQ_SMP_SUM | 2) ? 1 : 0);
  if (st != LUQ_OK) return st;
  st = gemm_checks(name, A, alpha, B, bscale, M, N, K, C, luq::gemm_workspace_bytes(M, N, K, ns), ws, ws_bytes);
  if (st != LUQ_OK) return st;
  return hip_status(luq::launch_gemm_luq_int4(A, (int64_t)luq::plane_bytes(M * K), ns, alpha, B,
                                              bscale, b_signed ? 1 : 0, M, N, K, C, ws, ws_bytes,
                                              static_cast<hipStream_t>(stream)));
}

luq_status luq_gemm_dgrad(const uint8_t* g_codes, const float* alpha, int n_samples,
                          const uint8_t* w_codes_t, const float* w_scale, int w_signed,
                          int64_t M, int64_t N, int64_t K, float* dx, void* ws, size_t ws_bytes,
                          void* stream) {
  g_last_error[0] = 0;
  return gemm_common("luq_gemm_dgrad", g_codes, alpha, n_samples, w_codes_t, w_scale, w_signed, M,
                     N, K, dx, ws, ws_bytes, stream);
}

luq_status luq_gemm_wgrad(const uint8_t* g_codes_t, const float* alpha, int n_samples,
                          const uint8_t* a_codes_t, const float* a_scale, int a_signed, int64_t T,
                          int64_t Nout, int64_t Kin, float* dw, void* ws, size_t ws_bytes,
                          void* stream) {
  g_last_error[0] = 0;
  return gemm_common("luq_gemm_wgrad", g_codes_t, alpha, n_samples, a_codes_t, a_scale, a_signed,
                     Nout, Kin, T, dw, ws, ws_bytes, stream);
}

luq_status int4_gemm_fwd(const uint8_t* x_codes, const float* x_scale, int x_signed, const uint8_t* w_codes,
                         const float* w_scale, int w_signed, int64_t M, int64_t N, int64_t K, float* y, void* ws,
                         size_t ws_bytes, void* stream) {
  const char* fn = "int4_gemm_fwd";
  g_last_error[0] = 0;
  if (!x_codes || !x_scale || !w_codes || !w_scale || !y) return fail(LUQ_ERR_NULL, "%s: NULL operand", fn);
  luq_status st = gemm_shape(fn, M, N, K);
  if (st != LUQ_OK) return st;
  st = gemm_checks(fn, x_codes, x_scale, w_codes, w_scale, M, N, K, y, luq::gemm_fwd_workspace_bytes(M, N, K), ws,
                   ws_bytes);
  if (st != LUQ_OK) return st;
  return hip_status(luq::launch_gemm_int4_fwd(x_codes, x_scale, x_signed ? 1 : 0, w_codes, w_scale,
                                              w_signed ? 1 : 0, M, N, K, y, ws, static_cast<hipStream_t>(stream)));
}

luq_status int4_im2col3x3_t(const uint8_t* act_codes, int64_t B, int64_t H, int64_t W, int64_t C,
                            uint8_t* col_t, void* stream) {
  g_last_error[0] = 0;
  if (B < 0 || H < 0 || W < 0 || C < 0) return fail(LUQ_ERR_SHAPE, "%s: negative size", "int4_im2col3x3_t");
  if (mul_overflows(B, H) || mul_overflows(B * H, W) || mul_overflows(B * H * W, 9 * C))
    return fail(LUQ_ERR_SHAPE, "%s: size overflows", "int4_im2col3x3_t");
  const int64_t T = B * H * W;
  if ((C & 1) || (T & 7)) return fail(LUQ_ERR_SHAPE, "%s: C must be even and B*H*W a multiple of 8", "int4_im2col3x3_t");
  if (B > INT32_MAX || H > INT32_MAX || W > INT32_MAX || C > INT32_MAX / 9)
    return fail(LUQ_ERR_SHAPE, "%s: dimension too large", "int4_im2col3x3_t");
  if (T == 0 || C == 0) return LUQ_OK;
  if (!act_codes || !col_t) return fail(LUQ_ERR_NULL, "%s: NULL pointer", "int4_im2col3x3_t");
  if (!aligned16(act_codes) || !aligned16(col_t))
    return fail(LUQ_ERR_ALIGN, "%s: pointers must be 16-byte aligned", "int4_im2col3x3_t");
  return hip_status(luq::launch_im2col3x3_t(act_codes, B, H, W, C, col_t,
                                            static_cast<hipStream_t>(stream)));
}

luq_status luq_conv3x3_dgrad(const uint8_t* g_codes, const float* alpha, int n_samples,
                             const uint8_t* w_codes_t, const float* w_scale, int w_signed, int64_t B,
                             int64_t H, int64_t W, int64_t C, int64_t Cout, float* dact, void* stream) {
  const char* fn = "luq_conv3x3_dgrad";
  g_last_error[0] = 0;
  if (B < 0 || H < 0 || W < 0 || C < 0 || Cout < 0) return fail(LUQ_ERR_SHAPE, "%s: negative size", fn);
  if (n_samples != 1 && n_samples != 2)
    return fail(LUQ_ERR_PARAM, "%s: n_samples must be 1 or 2 (sample planes)", fn);
  if (B > INT32_MAX || H > INT32_MAX || W > INT32_MAX || C > INT32_MAX || Cout > INT32_MAX ||
      mul_overflows(B, H) || mul_overflows(B * H, W) || mul_overflows(B * H * W, Cout) ||
      mul_overflows(9 * C, Cout))
    return fail(LUQ_ERR_SHAPE, "%s: size overflows", fn);
  const int64_t T = B * H * W;
  if (T == 0 || C == 0) return LUQ_OK;
  if (Cout < 32 || (Cout & 31) || Cout > 16384)
    return fail(LUQ_ERR_SHAPE, "%s: Cout must be a multiple of 32 in [32, 16384]", fn);
  if (W > luq::conv3x3_max_width()) return fail(LUQ_ERR_SHAPE, "%s: image width above 256", fn);
  if (C > ((int64_t)1 << 20)) return fail(LUQ_ERR_SHAPE, "%s: more than 2^20 input channels", fn);
  if (T * (Cout / 2) >= ((int64_t)1 << 30) || 9 * C * (Cout / 2) >= ((int64_t)1 << 30))
    return fail(LUQ_ERR_SHAPE, "%s: operand above 1 GiB of codes", fn);
  if (!g_codes || !alpha || !w_codes_t || !w_scale || !dact) return fail(LUQ_ERR_NULL, "%s: NULL operand", fn);
  if (!aligned16(g_codes) || !aligned16(w_codes_t) || !aligned4(dact) || !aligned4(alpha) || !aligned4(w_scale))
    return fail(LUQ_ERR_ALIGN, "%s: code operands must be 16-byte aligned, dact and scales 4-byte", fn);
  return hip_status(luq::launch_conv3x3_dgrad(g_codes, (int64_t)luq::plane_bytes(T * Cout), n_samples, alpha,
                                              w_codes_t, w_scale, w_signed ? 1 : 0, B, H, W, C, Cout, dact,
                                              static_cast<hipStream_t>(stream)));
}

luq_status luq_conv3x3_wgrad(const uint8_t* g_codes_t, const float* alpha, int n_samples,
                             const uint8_t* a_codes_t, const float* a_scale, int a_signed, int64_t B,
                             int64_t H, int64_t W, int64_t C, int64_t Cout, float* dw, void* ws,
                             size_t ws_bytes, void* stream) {
  const char* fn = "luq_conv3x3_wgrad";
  g_last_error[0] = 0;
  if (B < 0 || H < 0 || W < 0 || C < 1 || Cout < 1)
    return fail(LUQ_ERR_SHAPE, "%s: need B, H, W >= 0 and C, Cout >= 1", fn);
  if (n_samples != 1 && n_samples != 2)
    return fail(LUQ_ERR_PARAM, "%s: n_samples must be 1 or 2 (sample planes)", fn);
  if (B > INT32_MAX || H > INT32_MAX || W > INT32_MAX || C > INT32_MAX / 9 || Cout > INT32_MAX ||
      mul_overflows(B, H) || mul_overflows(B * H, W) || mul_overflows(B * H * W, Cout) ||
      mul_overflows(B * H * W, C) || mul_overflows(9 * C, Cout))
    return fail(LUQ_ERR_SHAPE, "%s: size overflows", fn);
  const int64_t T = B * H * W;
  if (T < 32 || (T & 31)) return fail(LUQ_ERR_SHAPE, "%s: B*H*W must be a positive multiple of 32", fn);
  if (T > ((int64_t)1 << 29) || W > ((int64_t)1 << 29)) return fail(LUQ_ERR_SHAPE, "%s: B*H*W above 2^29", fn);
  if (Cout * (T / 2) >= ((int64_t)1 << 30) || C * (T / 2) >= ((int64_t)1 << 30))
    return fail(LUQ_ERR_SHAPE, "%s: operand above 1 GiB of codes", fn);
  if (luq::conv3x3_wgrad_blocks(T, C, Cout) > ((int64_t)1 << 22))
    return fail(LUQ_ERR_SHAPE, "%s: too many channel tiles", fn);
  if (!g_codes_t || !alpha || !a_codes_t || !a_scale || !dw) return fail(LUQ_ERR_NULL, "%s: NULL operand", fn);
  const size_t need = luq::conv3x3_wgrad_workspace_bytes(T, C, Cout);
  if (need && (!ws || ws_bytes < need)) return fail(LUQ_ERR_WORKSPACE, "%s: workspace too small", fn);
  if (!aligned16(g_codes_t) || !aligned16(a_codes_t) || !aligned16(ws) || !aligned4(dw) || !aligned4(alpha) ||
      !aligned4(a_scale))
    return fail(LUQ_ERR_ALIGN, "%s: code operands and ws must be 16-byte aligned, dw and scales 4-byte", fn);
  return hip_status(luq::launch_conv3x3_wgrad(g_codes_t, (int64_t)luq::plane_bytes(T * Cout), n_samples, alpha,
                                              a_codes_t, a_scale, a_signed ? 1 : 0, B, H, W, C, Cout, dw, ws,
                                              static_cast<hipStream_t>(stream)));
}

}  // extern "C"

/*
 * luq.h -- C ABI of libluq: 4-bit LUQ training GEMM hot path on AMD MI355X.
 *
 * Method: "Accurate Neural Training with 4-bit Matrix Multiplications at
 * Standard Formats" (Chmiel, Banner, Hoffer, Ben Yaacov, Soudry; arXiv
 * 2112.10769).  Neural gradients are quantized with logarithmic unbiased
 * quantization (LUQ, Section 4) to a radix-2 FP4 [sign, 3-bit exponent, no
 * mantissa] code; weights and activations with a uniform INT4
 * round-to-nearest quantizer (Section 3.3, Appendix A.1); the backward and
 * update GEMMs of Eqs. backward / update then run on the 4-bit codes with
 * the per-tensor scales applied once to each sum (Appendix A.1).
 *
 * General conventions
 *  - Every pointer argument is DEVICE memory owned by the caller, except
 *    where noted.  The library never allocates or frees memory; it keeps no
 *    state between calls.
 *  - All work is enqueued asynchronously on `stream` (a hipStream_t; NULL is
 *    the null stream).  No call synchronizes with the host, except
 *    luq_query_status.
 *  - Scales (alpha, s) live in device memory: no host round trip.
 *  - Argument errors are detected on the host, before anything is enqueued,
 *    and returned as a luq_status; nothing is launched in that case.
 *    luq_last_error() then holds a message (thread-local).
 *  - Data errors (a non-finite input element) are reported through the
 *    outputs (the scale becomes NaN and every code 0) and, asynchronously,
 *    through a status word in the quantizer's workspace, which
 *    luq_query_status reads (LUQ_ERR_NONFINITE).
 *  - Base pointers must be 16-byte aligned (LUQ_ERR_ALIGN otherwise).
 *
 * Code formats (two 4-bit codes per byte, element 2b in the low nibble)
 *  - LUQ nibble: bit 3 = sign, bits 2..0 = exponent field e.  e = 0 is zero
 *    (sign bit always 0); e >= 1 decodes to (-1)^sign * alpha * 2^(e-1).
 *    Field 011 is the paper's FP4 value 4 (Appendix A.8.1 worked example).
 *  - INT4 nibble: signed codes -7..7 in two's complement, or unsigned codes
 *    0..15; the value is s * q.
 *  - A matrix of codes is stored row-major, each row packed along its
 *    columns.  "codes" is the [rows][cols] layout, "codes_t" the transposed
 *    [cols][rows] layout of the same codes.
 *  - LUQ SMP planes (Section 5.1: n independent samples with one alpha) are
 *    stored one after another, each plane luq_plane_bytes(rows*cols) bytes
 *    apart.
 */
#ifndef LUQ_H
#define LUQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LUQ_ABI_VERSION 9

typedef int luq_status;
enum {
  LUQ_OK = 0,
  LUQ_ERR_NULL = 1,      /* a required pointer is NULL                       */
  LUQ_ERR_SHAPE = 2,     /* a size is negative or breaks a layout rule      */
  LUQ_ERR_DTYPE = 3,     /* unknown luq_dtype                                */
  LUQ_ERR_PARAM = 4,     /* R, n_samples or another parameter out of range   */
  LUQ_ERR_WORKSPACE = 5, /* workspace missing or smaller than required       */
  LUQ_ERR_ALIGN = 6,     /* a pointer is not 16-byte aligned                 */
  LUQ_ERR_HIP = 7,       /* the HIP runtime rejected a launch or a copy      */
  LUQ_ERR_NONFINITE = 8  /* (luq_query_status) the quantized tensor, or the
                            in-hindsight estimate, was NaN or infinite       */
};

typedef enum { LUQ_F32 = 0, LUQ_BF16 = 1 } luq_dtype;

/* Or-ed into the R argument of the LUQ quantizers: power-of-two LUQ (the
 * appendix on power-of-two LUQ), alpha = 2^ceil(log2 m) / 2^R instead of
 * m / 2^R.  Every level is then a power of two and the top level is the
 * least power of two at or above m, so the maximum is not clipped. */
#define LUQ_ALPHA_PW2 0x100

/* Or-ed into n_samples = 2 of the LUQ quantizers and the backward GEMMs
 * (Section 5.1, SMP): the two samples are stored as one signed byte per
 * element, the sum of their decoded values in units of alpha (the averaged
 * gradient is alpha/2 times it), instead of two planes of codes.  It takes
 * the bytes of the two planes and spares the GEMM the decoding; |sum| <= 64
 * for R <= 5. */
#define LUQ_SMP_SUM 0x10

/* Or-ed into n_samples = 1 of luq_gemm_dgrad and luq_gemm_wgrad: the MACs
 * run on the FP6 carrier (the scaled f8f6f4 MFMA of CDNA4, e3m2 x e2m3)
 * instead of INT8.  Every code is exact in FP6 -- the LUQ level alpha 2^(e-1)
 * as the e3m2 value 2^(e-3) (R <= 6), an INT4 code q as the e2m3 value q/8 --
 * and the fp32 sums are exact for reductions of up to 16384 (longer ones are
 * split and combined exactly), so the result equals the INT8 carrier's bit
 * for bit.  The codes are first converted into FP6 blocks in the workspace,
 * which is luq_workspace_size(LUQ_OP_GEMM_DGRAD_FP6 / _WGRAD_FP6, ...). */
#define LUQ_CARRIER_FP6 0x40

/* Operation ids for luq_workspace_size. */
enum {
  LUQ_OP_QUANTIZE_GRAD = 0, /* d0 = number of elements                     */
  LUQ_OP_INT4_QUANTIZE = 1, /* d0 = number of elements                     */
  LUQ_OP_GEMM_DGRAD = 2,    /* d0 = M, d1 = N, d2 = K                        */
  LUQ_OP_GEMM_WGRAD = 3,    /* d0 = T, d1 = Nout, d2 = Kin                   */
  LUQ_OP_GEMM_FWD = 4,      /* d0 = M, d1 = N, d2 = K                        */
  LUQ_OP_CONV_WGRAD = 5,    /* d0 = B*H*W, d1 = C, d2 = Cout                 */
  LUQ_OP_GEMM_DGRAD_FP6 = 6, /* luq_gemm_dgrad with LUQ_CARRIER_FP6: M, N, K  */
  LUQ_OP_GEMM_WGRAD_FP6 = 7  /* luq_gemm_wgrad with LUQ_CARRIER_FP6: T, Nout, Kin */
};

/* ABI version of the loaded library (LUQ_ABI_VERSION of its build). */
int luq_abi_version(void);

/* Static description of a status code. */
const char* luq_status_string(luq_status status);

/* Detail of the last error returned on the calling thread ("" if none). */
const char* luq_last_error(void);

/* Bytes between consecutive SMP planes of a code tensor of n elements:
 * ceil(n/2) rounded up to a multiple of 256. */
size_t luq_plane_bytes(int64_t n);

/* Device workspace (bytes) an operation needs; 0 if none.  The workspace
 * holds per-block partial maxima and a status word (quantizers) or split-K
 * partial sums (GEMMs); its contents on entry do not matter. */
size_t luq_workspace_size(int op, int64_t d0, int64_t d1, int64_t d2);

/*
 * luq_query_status -- the data status of the last quantizer call
 * (luq_quantize_grad, luq_quantize_grad_hindsight or int4_quantize) that
 * used the workspace ws.  Alpha (Eq. alpha) and the INT4 scale (Appendix
 * A.1) are defined only for a finite maximum; every such call writes, on
 * the device and in stream order, whether its maximum was finite.
 *
 *  ws      the workspace passed to that call (device memory, 16-byte
 *          aligned).
 *  stream  the stream the call was enqueued on: the word is copied to the
 *          host after it and the stream is synchronized (so this call may
 *          not be captured into a HIP graph).
 *
 * Returns LUQ_OK (finite input), LUQ_ERR_NONFINITE (a NaN or infinite
 * element; for luq_quantize_grad_hindsight also a NaN or infinite
 * estimate), LUQ_ERR_NULL / LUQ_ERR_ALIGN for a bad ws, LUQ_ERR_HIP if the
 * copy fails, or LUQ_ERR_WORKSPACE if ws holds no quantizer status (no
 * quantizer has written it, or another operation reused it since).  An
 * int4_quantize call with clip > 0 takes no maximum and writes LUQ_OK when
 * it is given a workspace (none otherwise).
 */
luq_status luq_query_status(const void* ws, void* stream);

/*
 * luq_quantize_grad -- LUQ of a neural-gradient tensor (Section 4).
 *
 * Computes m = max|g|, alpha = fl32(m / 2^R) (Eq. alpha; R = 2^(b-1) = 4 for
 * FP4 with b = 3 exponent bits), and for every element and SMP sample s the
 * code of X_q = Q_alpha(T_alpha(g)): stochastic underflow below alpha
 * (Eq. StochasticPruning) and logarithmic stochastic rounding between
 * adjacent levels alpha*2^n (Eq. unbiasedFpQ).  One 16-bit uniform j per
 * element and sample comes from Philox4x32-10 with key = (seed lo, seed hi)
 * and counter = (blk lo, blk hi, s, counter), blk = i >> 3 for the row-major
 * flat index i; word (i >> 1) & 3, half i & 1.  With w the bin width and d
 * the distance of |g| above the bin's lower level, the value rounds up iff
 * j * w < d * 2^16 (exactly), so 0 <= E[Q(g)] - g < w * 2^-16.
 *
 *  g        [rows][cols] row-major, dtype dt (LUQ_F32 or LUQ_BF16).
 *  rows, cols  >= 0.  For rows > 1, cols must be even.  When codes_t is
 *           requested, rows and cols must be multiples of 8.
 *  R        4, 5 or 6: levels alpha * 2^n for n = 0..R; or-ed with
 *           LUQ_ALPHA_PW2 for the power-of-two alpha (alpha is then an
 *           exact power of two, or 0 below the float32 subnormal range).
 *  seed, counter  Philox key and step counter; the codes are a pure
 *           function of (g, R, seed, counter, sample).
 *  n_samples  1 or 2 (SMP planes, Section 5.1), or LUQ_SMP_SUM | 2 (two
 *           samples as int8 sums).  Two samples require R <= 5 so that the
 *           sum of two decoded planes fits an int8 (|sum| <= 2^(R+1)).
 *  codes    out: n_samples planes of [rows][cols] codes (row stride
 *           ceil(cols/2) bytes), or NULL.  With LUQ_SMP_SUM: one [rows][cols]
 *           int8 matrix (row stride cols bytes), byte i the sum over the two
 *           samples of the decoded code (0 or +-2^(e-1)).
 *  codes_t  out: n_samples planes of the transposed [cols][rows] codes (row
 *           stride rows/2 bytes), or NULL; with LUQ_SMP_SUM the transposed
 *           [cols][rows] int8 sums (row stride rows bytes).  At least one of
 *           codes, codes_t.
 *  alpha    out: 1 float.  0 when max|g| = 0 (all codes 0); NaN when g has
 *           a non-finite element (all codes 0; luq_query_status then
 *           returns LUQ_ERR_NONFINITE).
 *  maxabs   out: 1 float, max|g| (non-finite when g is), or NULL.
 *  ws       workspace of luq_workspace_size(LUQ_OP_QUANTIZE_GRAD, rows*cols)
 *           (may be NULL when rows*cols = 0); receives the status word.
 */
luq_status luq_quantize_grad(const void* g, luq_dtype dt, int64_t rows, int64_t cols, int R,
                             uint64_t seed, uint32_t counter, int n_samples, uint8_t* codes,
                             uint8_t* codes_t, float* alpha, float* maxabs, void* ws,
                             size_t ws_bytes, void* stream);

/*
 * luq_quantize_grad_noalloc -- luq_quantize_grad for callers that cannot
 * allocate device memory (code being captured into a HIP graph, tight
 * serving loops, hosts that forbid allocation): the same codes, alpha and
 * maxabs, bit for bit, with the workspace taken from a static device array
 * inside the library instead of a caller's buffer.  The caller still passes
 * the input and the outputs; the call allocates and frees nothing.
 *
 *  Arguments as for luq_quantize_grad, without ws and ws_bytes.
 *  Scratch: one array of luq_workspace_size(LUQ_OP_QUANTIZE_GRAD, n) bytes
 *           (65544: 16384 partial maxima, their fold and a status word; the
 *           same for every n) per GPU the library runs on, held until the
 *           process ends.  A size whose workspace exceeded it would be
 *           refused with LUQ_ERR_SHAPE.
 *  Every call on one GPU uses that GPU's array, which keeps the last call's
 *  contents (nothing in it needs to start at zero): calls that overlap in
 *  time on one GPU (other streams, other host threads) race and must be
 *  ordered by the caller.  The status word it writes is not reachable
 *  through luq_query_status; a non-finite input shows as alpha = NaN.
 *  Errors as for luq_quantize_grad, plus LUQ_ERR_HIP when the array's
 *  device address cannot be found on the current device.
 */
luq_status luq_quantize_grad_noalloc(const void* g, luq_dtype dt, int64_t rows, int64_t cols, int R,
                                     uint64_t seed, uint32_t counter, int n_samples, uint8_t* codes,
                                     uint8_t* codes_t, float* alpha, float* maxabs, void* stream);

/*
 * luq_quantize_grad_hindsight -- LUQ in one pass over g with the
 * in-hindsight maximum (Section 4, "Reducing the data movement"; the
 * hindsight appendix).
 *
 * Instead of measuring max|g| first, alpha = fl32(m / 2^R) comes from the
 * estimate m in *state, carried over from the previous step; the same pass
 * measures max|g| of this tensor, and *state becomes the next estimate
 * (Eq. hindsight):
 *     m' = fl32( fl32(fl32(1 - eta) * max|g|) + fl32(eta * m) ).
 * Codes are those of luq_quantize_grad for that alpha, except that
 * magnitudes at or above alpha * 2^R (the estimate may be below this
 * tensor's maximum), and NaN elements, take the top code R + 1 with their
 * sign.  An estimate that is NaN or infinite gives alpha = NaN and all codes
 * 0; one that is 0 or negative gives alpha = 0 and all codes 0.  With
 * *state = max|g| the codes equal luq_quantize_grad's.  When max|g| is not
 * finite (an overflowed step) *state is left unchanged, so the estimate
 * survives the step; luq_query_status reports LUQ_ERR_NONFINITE for such a
 * step and for a non-finite estimate.  R may carry
 * LUQ_ALPHA_PW2: alpha is then the power-of-two alpha of the estimate (the
 * appendix combines power-of-two LUQ with hindsight).
 *
 *  g, dt, rows, cols, R, seed, counter, n_samples, codes, codes_t
 *           as for luq_quantize_grad.
 *  eta      momentum in [0, 1] (0.1 in the paper's experiments).
 *  state    in/out: 1 float on the device, the estimate m (initialise it,
 *           e.g., with the maxabs of luq_quantize_grad on an earlier step).
 *  alpha    out: 1 float, the alpha used.
 *  maxabs   out: 1 float, max|g| of this tensor (NaN if g has a NaN), or NULL.
 *  ws       workspace of luq_workspace_size(LUQ_OP_QUANTIZE_GRAD, rows*cols).
 *
 * Errors as for luq_quantize_grad; LUQ_ERR_PARAM for eta outside [0, 1],
 * LUQ_ERR_NULL for a NULL state.
 */
luq_status luq_quantize_grad_hindsight(const void* g, luq_dtype dt, int64_t rows, int64_t cols, int R,
                                       uint64_t seed, uint32_t counter, int n_samples, float eta,
                                       uint8_t* codes, uint8_t* codes_t, float* state, float* alpha,
                                       float* maxabs, void* ws, size_t ws_bytes, void* stream);

/*
 * int4_quantize -- uniform INT4 round-to-nearest quantizer (Section 3.3;
 * scale alpha = Delta / (2^b - 1) of Appendix A.1; Delta = max-abs or clip,
 * since the SAWB coefficients the paper used are not given).
 *
 *  m = clip if clip > 0, else max|x| (signed) or max(max x, 0) (unsigned).
 *  Q = 7 (signed, codes -7..7) or 15 (unsigned, codes 0..15).
 *  inv = fl32(Q / m), s = fl32(m / Q), q = clamp(rne(fl32(x * inv))), with a
 *  NaN product (0 * inf for tiny m) giving q = 0.  m = 0: s = 0, codes 0.
 *  Non-finite x (when clip <= 0): s = NaN, codes 0 (luq_query_status:
 *  LUQ_ERR_NONFINITE).
 *
 *  x        [rows][cols] row-major, dtype dt.  Shape rules as for
 *           luq_quantize_grad.
 *  codes, codes_t  out: [rows][cols] and/or [cols][rows] codes (one may be
 *           NULL, not both).
 *  scale    out: 1 float s.
 *  ws       workspace of luq_workspace_size(LUQ_OP_INT4_QUANTIZE, rows*cols)
 *           (may be NULL when clip > 0); receives the status word.
 */
luq_status int4_quantize(const void* x, luq_dtype dt, int64_t rows, int64_t cols, int is_signed,
                         float clip, uint8_t* codes, uint8_t* codes_t, float* scale, void* ws,
                         size_t ws_bytes, void* stream);

/*
 * luq_gemm_dgrad -- the backward GEMM of Eq. backward on codes:
 *   dx[m][n] = (alpha / n_samples) * w_scale * sum_k (sum_s cg_s[m][k]) * cw[n][k]
 * i.e. dX = Q(g) Q(W) with g [M tokens][K out-features] and the weight
 * W [K out][N in] given TRANSPOSED as w_codes_t [N][K] (the codes_t output of
 * int4_quantize on W).  SMP planes are summed exactly before the MACs
 * (Section 5.1 average).  Integer MACs accumulate exactly in int32; the
 * scales are applied once in fp32 (Appendix A.1).
 *
 *  g_codes    n_samples planes of [M][K] LUQ codes (plane stride
 *             luq_plane_bytes(M*K)); with n_samples = LUQ_SMP_SUM | 2 the
 *             [M][K] int8 sums of two samples (luq_quantize_grad's output in
 *             that format), scale alpha / 2.  n_samples = LUQ_CARRIER_FP6 | 1
 *             selects the FP6 carrier for one plane (same result; workspace
 *             luq_workspace_size(LUQ_OP_GEMM_DGRAD_FP6, M, N, K)).
 *  alpha      1 float (device), the LUQ alpha of g.
 *  w_codes_t  [N][K] INT4 codes; w_scale 1 float (device); w_signed 0/1.
 *  M, N >= 1; K >= 32 and a multiple of 32; each code operand below 2 GiB.
 *             Reductions longer than the int32-exact length are split
 *             internally and the partial sums combined exactly, so any K is
 *             exact.  The codes must come from this library: with two samples
 *             every field must be <= 6 (R <= 5), which luq_quantize_grad
 *             enforces.
 *  dx         out: [M][N] fp32, row-major.
 *  ws         workspace of luq_workspace_size(LUQ_OP_GEMM_DGRAD, M, N, K).
 */
luq_status luq_gemm_dgrad(const uint8_t* g_codes, const float* alpha, int n_samples,
                          const uint8_t* w_codes_t, const float* w_scale, int w_signed,
                          int64_t M, int64_t N, int64_t K, float* dx, void* ws, size_t ws_bytes,
                          void* stream);

/*
 * luq_gemm_wgrad -- the update GEMM of Eq. update on codes:
 *   dw[o][i] = (alpha / n_samples) * a_scale * sum_t (sum_s cg_s[t][o]) * ca[t][i]
 * i.e. dW = Q(g)^T Q(a) in the torch weight-gradient layout [Nout][Kin], with
 * both operands given TRANSPOSED (tokens innermost): g_codes_t [Nout][T]
 * (codes_t of luq_quantize_grad on g [T][Nout]) and a_codes_t [Kin][T].
 * Long reductions are split over T with exact int32 partial sums combined
 * in a fixed order, so the result does not depend on the split.
 *
 *  g_codes_t is n_samples planes of codes, or with n_samples =
 *  LUQ_SMP_SUM | 2 the [Nout][T] int8 sums of two samples;
 *  LUQ_CARRIER_FP6 | 1 selects the FP6 carrier for one plane (same result;
 *  workspace luq_workspace_size(LUQ_OP_GEMM_WGRAD_FP6, T, Nout, Kin)).
 *  T >= 32 and a multiple of 32; Nout, Kin >= 1; each code operand below
 *  2 GiB.
 *  ws  workspace of luq_workspace_size(LUQ_OP_GEMM_WGRAD, T, Nout, Kin).
 */
luq_status luq_gemm_wgrad(const uint8_t* g_codes_t, const float* alpha, int n_samples,
                          const uint8_t* a_codes_t, const float* a_scale, int a_signed, int64_t T,
                          int64_t Nout, int64_t Kin, float* dw, void* ws, size_t ws_bytes,
                          void* stream);

/*
 * int4_gemm_fwd -- the forward GEMM of Eq. forward on INT4 codes
 * (Appendix A.1: every MAC on codes, the two scales applied once):
 *   y[m][n] = x_scale * w_scale * sum_k cx[m][k] * cw[n][k]
 * i.e. y = Q(x) Q(W)^T for activations x [M tokens][K in-features] and the
 * weight W [N out][K in] in its natural layout; both are the row-major
 * codes output of int4_quantize, so neither is transposed.  Integer MACs
 * accumulate exactly in int32; reductions longer than the int32-exact
 * length are split and the partial sums combined exactly in a fixed order.
 *
 *  x_codes    [M][K] INT4 codes; x_scale 1 float (device); x_signed 0/1
 *             (unsigned for non-negative activations such as ReLU outputs).
 *  w_codes    [N][K] INT4 codes; w_scale 1 float (device); w_signed 0/1.
 *  M, N >= 1 and below 2^30; K >= 32 and a multiple of 32.
 *  y          out: [M][N] fp32, row-major.
 *  ws         workspace of luq_workspace_size(LUQ_OP_GEMM_FWD, M, N, K)
 *             (0 bytes, NULL allowed, unless the reduction is split).
 *  Errors: LUQ_ERR_NULL, LUQ_ERR_SHAPE, LUQ_ERR_WORKSPACE, LUQ_ERR_ALIGN
 *  (code operands and ws 16-byte aligned; y and scales 4-byte aligned),
 *  LUQ_ERR_HIP; nothing is enqueued on error.
 */
luq_status int4_gemm_fwd(const uint8_t* x_codes, const float* x_scale, int x_signed,
                         const uint8_t* w_codes, const float* w_scale, int w_signed, int64_t M,
                         int64_t N, int64_t K, float* y, void* ws, size_t ws_bytes, void* stream);

/*
 * int4_im2col3x3_t -- lowering of a 3x3 / stride 1 / zero-pad 1 convolution
 * on INT4 codes, written transposed for luq_gemm_wgrad: for activation codes
 * act [B][H][W][C] (NHWC, packed along C), writes
 *   col_t[(kh*3 + kw)*C + c][t] = act[b][y+kh-1][x+kw-1][c]   (0 off-image)
 * for t = (b*H + y)*W + x, packed along t (row stride T/2 bytes, T = B*H*W).
 * C must be even and T a multiple of 8.
 */
luq_status int4_im2col3x3_t(const uint8_t* act_codes, int64_t B, int64_t H, int64_t W, int64_t C,
                            uint8_t* col_t, void* stream);

/*
 * luq_conv3x3_dgrad -- activation gradient of a 3x3 / stride 1 / zero-pad 1
 * convolution on codes: Eq. backward applied to the lowered convolution and
 * folded back onto the input pixels (the adjoint of the lowering), without
 * forming the lowered [T][9*C] gradient:
 *   dact[t][c] = (alpha / n_samples) * w_scale *
 *                sum_{kh,kw} sum_o (sum_s cg_s[t'][o]) * cw[(kh*3 + kw)*C + c][o]
 * for t = (b*H + y)*W + x and t' = (b*H + y + 1 - kh)*W + x + 1 - kw, terms
 * whose t' lies off the image left out.  Every MAC is on codes and
 * accumulates exactly in int32; the scales are applied once in fp32
 * (Appendix A.1), as in luq_gemm_dgrad.
 *
 *  g_codes    n_samples planes of [T][Cout] LUQ codes of the output gradient
 *             (NHWC pixels t, T = B*H*W; plane stride luq_plane_bytes(T*Cout)).
 *  alpha      1 float (device), the LUQ alpha of g.
 *  w_codes_t  [9*C][Cout] INT4 codes: the weight [Cout][3][3][C] (columns in
 *             (kh, kw, c) order) in the transposed layout, i.e. the codes_t
 *             output of int4_quantize on W [Cout][9*C]; w_scale 1 float
 *             (device); w_signed 0/1.
 *  B, H, W, C >= 0 (nothing is done when B*H*W or C is 0); W <= 256;
 *             C <= 2^20; Cout a multiple of 32 in [32, 16384]; each code operand below
 *             1 GiB.  n_samples 1 or 2 (codes from this library, R <= 5 for 2).
 *  dact       out: [T][C] fp32, row-major (NHWC).
 *  No workspace.  Errors: LUQ_ERR_SHAPE, LUQ_ERR_PARAM, LUQ_ERR_NULL,
 *  LUQ_ERR_ALIGN (code operands 16-byte aligned, dact and scales 4-byte),
 *  LUQ_ERR_HIP; nothing is enqueued on error.
 */
luq_status luq_conv3x3_dgrad(const uint8_t* g_codes, const float* alpha, int n_samples,
                             const uint8_t* w_codes_t, const float* w_scale, int w_signed, int64_t B,
                             int64_t H, int64_t W, int64_t C, int64_t Cout, float* dact, void* stream);

/*
 * luq_conv3x3_wgrad -- weight gradient of a 3x3 / stride 1 / zero-pad 1
 * convolution on codes: Eq. update applied to the lowered convolution,
 * without forming the lowered [T][9*C] activations:
 *   dw[o][(kh*3 + kw)*C + c] = (alpha / n_samples) * a_scale *
 *                              sum_t (sum_s cg_s[t][o]) * ca[t'][c]
 * for t = (b*H + y)*W + x and t' = (b*H + y + kh - 1)*W + x + kw - 1, terms
 * whose t' lies off the image left out.  Equal to luq_gemm_wgrad on the
 * int4_im2col3x3_t lowering of the activation codes.  Every MAC is on codes
 * with exact int32 partial sums over pixel ranges, combined exactly in a
 * fixed order; the scales are applied once in fp32 (Appendix A.1).
 *
 *  g_codes_t  n_samples planes of [Cout][T] LUQ codes of the output gradient
 *             (the codes_t output of luq_quantize_grad on g [T][Cout]; plane
 *             stride luq_plane_bytes(T*Cout)).
 *  alpha      1 float (device), the LUQ alpha of g.
 *  a_codes_t  [C][T] INT4 codes of the activations (NHWC pixels t; the
 *             codes_t output of int4_quantize on act [T][C]); a_scale 1 float
 *             (device); a_signed 0/1.
 *  B, H, W >= 0 with T = B*H*W a positive multiple of 32, at most 2^29;
 *             C, Cout >= 1; each code operand below 1 GiB.  n_samples 1 or 2
 *             (sample planes).
 *  dw         out: [Cout][9*C] fp32, columns in (kh, kw, c) order.
 *  ws         workspace of luq_workspace_size(LUQ_OP_CONV_WGRAD, T, C, Cout).
 *  Errors: LUQ_ERR_SHAPE, LUQ_ERR_PARAM, LUQ_ERR_NULL, LUQ_ERR_WORKSPACE,
 *  LUQ_ERR_ALIGN (code operands and ws 16-byte aligned, dw and scales 4-byte),
 *  LUQ_ERR_HIP; nothing is enqueued on error.
 */
luq_status luq_conv3x3_wgrad(const uint8_t* g_codes_t, const float* alpha, int n_samples,
                             const uint8_t* a_codes_t, const float* a_scale, int a_signed, int64_t B,
                             int64_t H, int64_t W, int64_t C, int64_t Cout, float* dw, void* ws,
                             size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LUQ_H */

// Forward 4-bit GEMM (Section 3.3; Appendix A.1): y = Q(x) Q(W)^T with
// INT4 codes of the activations (A, signed or unsigned) and of the weights
// (B), both K-major, exact int32 accumulation and the two per-tensor scales
// applied once; the tile kernel is in gemm_kernel.hpp.
#include "gemm_kernel.hpp"

namespace luq {

size_t gemm_fwd_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  const GemmPlan p = plan_gemm(M, N, K, kMaxExactKInt4);
  if (p.splits <= 1) return 0;
  return (size_t)p.splits * (size_t)M * (size_t)N * sizeof(int32_t);
}

hipError_t launch_gemm_int4_fwd(const uint8_t* X, const float* x_scale, int x_signed, const uint8_t* W,
                                const float* w_scale, int w_signed, int64_t M, int64_t N, int64_t K, float* Y,
                                void* ws, hipStream_t st) {
  const GemmPlan p = plan_gemm(M, N, K, kMaxExactKInt4);
  GemmArgs a;
  a.A = X;
  a.a_plane = 0;
  a.B = W;
  a.M = M;
  a.N = N;
  a.K = K;
  a.alpha = x_scale;
  a.bscale = w_scale;
  a.C = Y;
  a.partial = p.splits > 1 ? static_cast<int32_t*>(ws) : nullptr;
  if (x_signed)
    return w_signed ? gemm_launch_t<kAcInt4S, 1, true>(a, p, st) : gemm_launch_t<kAcInt4S, 1, false>(a, p, st);
  return w_signed ? gemm_launch_t<kAcInt4U, 1, true>(a, p, st) : gemm_launch_t<kAcInt4U, 1, false>(a, p, st);
}

}  // namespace luq

// 4-bit backward and update GEMMs (Eq. backward, Eq. update): A = LUQ codes
// of the neural gradient (n SMP planes, or the int8 sums of two samples),
// B = INT4 codes; the tile kernel is in gemm_kernel.hpp.
#include "gemm_kernel.hpp"

namespace luq {

size_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K, int /*ns*/) {
  const GemmPlan p = plan_gemm(M, N, K, kMaxExactK);
  if (p.splits <= 1) return 0;
  return (size_t)p.splits * (size_t)M * (size_t)N * sizeof(int32_t);
}

hipError_t launch_gemm_luq_int4(const uint8_t* A, int64_t a_plane, int ns, const float* alpha,
                                const uint8_t* B, const float* bscale, int b_signed, int64_t M,
                                int64_t N, int64_t K, float* C, void* ws, size_t /*ws_bytes*/,
                                hipStream_t st) {
  const GemmPlan p = plan_gemm(M, N, K, kMaxExactK);
  GemmArgs a;
  a.A = A;
  a.a_plane = a_plane;
  a.B = B;
  a.M = M;
  a.N = N;
  a.K = K;
  a.alpha = alpha;
  a.bscale = bscale;
  a.C = C;
  a.partial = p.splits > 1 ? static_cast<int32_t*>(ws) : nullptr;
  if (ns == 1)
    return b_signed ? gemm_launch_t<kAcLuq, 1, true>(a, p, st) : gemm_launch_t<kAcLuq, 1, false>(a, p, st);
  if (ns == kSmpSum)
    return b_signed ? gemm_launch_t<kAcSum2, 1, true>(a, p, st) : gemm_launch_t<kAcSum2, 1, false>(a, p, st);
  return b_signed ? gemm_launch_t<kAcLuq, 2, true>(a, p, st) : gemm_launch_t<kAcLuq, 2, false>(a, p, st);
}

}  // namespace luq

// 4-bit backward / update GEMMs on INT8 MFMA (gfx950).
//
//   C[m][n] = (alpha / ns) * s_B * sum_k A[m][k] * B[n][k]
//
// A holds LUQ codes (Section 4 of the paper; ns SMP planes, Section 5.1), B
// INT4 codes (Section 3.3).  Both operands are K-major nibble matrices; the
// quantizers write whichever layout (row-major or transposed) a GEMM needs,
// so the GEMM never transposes.
//
// Carrier: v_mfma_i32_16x16x64_i8 with exact int32 accumulation.  Codes are
// expanded from nibbles to int8 once per workgroup tile, on the way from
// global memory into LDS:
//   LUQ  : a byte LUT (v_perm_b32) maps the exponent field e to 2^(e-1) (or
//          0), then bytes whose sign bit is set are negated with a SWAR
//          xor/add.  SMP planes are added bytewise (|sum| <= 64).
//   INT4 : the nibble is moved to the top of its byte, giving 16*q (signed,
//          two's complement) or 8*q (unsigned) with no further work; the
//          extra power of two is removed exactly in the epilogue.
// The even-k nibbles of a word land in one int8 word and the odd-k nibbles
// in the next.  Both operands use the same order, so the contraction over
// k is unchanged.
//
// The per-tensor scales are applied once to the int32 sums (Appendix A.1):
//   C = fl32( fl32(acc) * fl32( fl32(alpha / ns) * s_B ) * 2^-4|2^-3 ).
// Long reductions are split along K into chunks whose int32 sums cannot
// overflow; chunk sums are added in int64 in a fixed order.
#include "luq_device.hpp"
#include "luq_launch.hpp"

namespace luq {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int kGemmThreads = 256;
constexpr int kBK = 128;                 // k per LDS stage (two MFMA k-steps)
constexpr int kPitch = kBK + 16;         // LDS row pitch in bytes
constexpr int64_t kMaxExactK = 1 << 18;  // |A| <= 64, |B| <= 120: 2^18 * 7680 < 2^31

// ---- nibble -> int8 expansion ------------------------------------------------

__device__ __forceinline__ void expand_luq(uint32_t x, uint32_t& lo, uint32_t& hi) {
  // bytes 0..7 of the table: 0, 1, 2, 4, 8, 16, 32, 64 (indexed by field e)
  const uint32_t t_lo = 0x04020100u, t_hi = 0x40201008u;
  const uint32_t m_lo = __builtin_amdgcn_perm(t_hi, t_lo, x & 0x07070707u);
  const uint32_t m_hi = __builtin_amdgcn_perm(t_hi, t_lo, (x >> 4) & 0x07070707u);
  const uint32_t s_lo = (x >> 3) & 0x01010101u, s_hi = (x >> 7) & 0x01010101u;
  // 0xFF in every byte whose sign bit is set; negation = (m ^ 0xFF) + 1, which
  // never carries out of a byte because m >= 1 wherever the sign is set
  lo = (m_lo ^ ((s_lo << 8) - s_lo)) + s_lo;
  hi = (m_hi ^ ((s_hi << 8) - s_hi)) + s_hi;
}

template <bool SIGNED>
__device__ __forceinline__ void expand_int4(uint32_t x, uint32_t& lo, uint32_t& hi) {
  if constexpr (SIGNED) {
    lo = (x << 4) & 0xF0F0F0F0u;  // 16 * q
    hi = x & 0xF0F0F0F0u;
  } else {
    lo = (x << 3) & 0x78787878u;  // 8 * q
    hi = (x >> 1) & 0x78787878u;
  }
}

// Bytewise int8 addition without carries between bytes.
__device__ __forceinline__ uint32_t add_i8x4(uint32_t a, uint32_t b) {
  const uint32_t s = (a & 0x7F7F7F7Fu) + (b & 0x7F7F7F7Fu);
  return s ^ ((a ^ b) & 0x80808080u);
}

struct GemmArgs {
  const uint8_t* A;
  int64_t a_plane;
  const uint8_t* B;
  int64_t M, N, K;
  const float* alpha;
  const float* bscale;
  float* C;
  int32_t* partial;   // split-K chunk sums [splits][M][N], or null
  int64_t k_chunk;    // k per split (multiple of kBK)
  int tiles_n;        // number of tiles along N
};

// ---- the tile kernel ----------------------------------------------------------

template <int BM, int BN, int NS, bool BSIGNED>
__global__ __launch_bounds__(kGemmThreads) void gemm_luq_int4_kernel(GemmArgs a) {
  static_assert(BM % 32 == 0 && BN % 32 == 0, "wave tiles are multiples of 16");
  constexpr int TM = BM / 32, TN = BN / 32;            // MFMA tiles per wave
  constexpr int ACH = BM * (kBK / 32) / kGemmThreads;  // 16-byte A chunks per thread
  constexpr int BCH = BN * (kBK / 32) / kGemmThreads;
  static_assert(ACH >= 1 && BCH >= 1, "tile too small for the block");
  __shared__ __attribute__((aligned(16))) uint8_t As[2][BM * kPitch];
  __shared__ __attribute__((aligned(16))) uint8_t Bs[2][BN * kPitch];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int64_t m0 = (int64_t)(blockIdx.x / a.tiles_n) * BM;
  const int64_t n0 = (int64_t)(blockIdx.x % a.tiles_n) * BN;
  const int64_t kbeg = (int64_t)blockIdx.y * a.k_chunk;
  int64_t kend = kbeg + a.k_chunk;
  if (kend > a.K) kend = a.K;
  const int nkt = (int)((kend - kbeg + kBK - 1) / kBK);
  const int64_t ld = a.K >> 1;  // bytes per operand row

  uint4 ra[NS][ACH], rb[BCH];
  auto load_tiles = [&](int64_t k0) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int c = tid + i * kGemmThreads, row = c >> 2, kc = c & 3;
      const int64_t m = m0 + row, k = k0 + kc * 32;
      const bool ok = (m < a.M) && (k < kend);
#pragma unroll
      for (int s = 0; s < NS; ++s)
        ra[s][i] = ok ? *reinterpret_cast<const uint4*>(a.A + s * a.a_plane + m * ld + (k >> 1))
                      : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int c = tid + i * kGemmThreads, row = c >> 2, kc = c & 3;
      const int64_t n = n0 + row, k = k0 + kc * 32;
      const bool ok = (n < a.N) && (k < kend);
      rb[i] = ok ? *reinterpret_cast<const uint4*>(a.B + n * ld + (k >> 1)) : make_uint4(0, 0, 0, 0);
    }
  };
  auto store_tiles = [&](int buf) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int c = tid + i * kGemmThreads, row = c >> 2, kc = c & 3;
      uint32_t w[8];
      const uint32_t x0[4] = {ra[0][i].x, ra[0][i].y, ra[0][i].z, ra[0][i].w};
#pragma unroll
      for (int d = 0; d < 4; ++d) expand_luq(x0[d], w[2 * d], w[2 * d + 1]);
      if constexpr (NS == 2) {
        const uint32_t x1[4] = {ra[1][i].x, ra[1][i].y, ra[1][i].z, ra[1][i].w};
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          uint32_t l, h;
          expand_luq(x1[d], l, h);
          w[2 * d] = add_i8x4(w[2 * d], l);
          w[2 * d + 1] = add_i8x4(w[2 * d + 1], h);
        }
      }
      uint4* dst = reinterpret_cast<uint4*>(&As[buf][row * kPitch + kc * 32]);
      dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
      dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int c = tid + i * kGemmThreads, row = c >> 2, kc = c & 3;
      uint32_t w[8];
      const uint32_t x0[4] = {rb[i].x, rb[i].y, rb[i].z, rb[i].w};
#pragma unroll
      for (int d = 0; d < 4; ++d) expand_int4<BSIGNED>(x0[d], w[2 * d], w[2 * d + 1]);
      uint4* dst = reinterpret_cast<uint4*>(&Bs[buf][row * kPitch + kc * 32]);
      dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
      dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
    }
  };

  v4i acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = v4i{0, 0, 0, 0};

  if (nkt > 0) load_tiles(kbeg);
  for (int t = 0; t < nkt; ++t) {
    const int buf = t & 1;
    store_tiles(buf);
    __syncthreads();
    if (t + 1 < nkt) load_tiles(kbeg + (int64_t)(t + 1) * kBK);
    const uint8_t* as = &As[buf][(wm * (BM / 2) + (lane & 15)) * kPitch + (lane >> 4) * 16];
    const uint8_t* bs = &Bs[buf][(wn * (BN / 2) + (lane & 15)) * kPitch + (lane >> 4) * 16];
#pragma unroll
    for (int kk = 0; kk < kBK; kk += 64) {
      v4i fa[TM], fb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) fa[i] = *reinterpret_cast<const v4i*>(as + i * 16 * kPitch + kk);
#pragma unroll
      for (int j = 0; j < TN; ++j) fb[j] = *reinterpret_cast<const v4i*>(bs + j * 16 * kPitch + kk);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
  }

  // D layout of the 16x16 MFMA: lane l, register r -> row 4*(l/16)+r, column l%16
  const int64_t rbase = m0 + wm * (BM / 2) + 4 * (lane >> 4);
  const int64_t cbase = n0 + wn * (BN / 2) + (lane & 15);
  if (a.partial) {
    int32_t* P = a.partial + (int64_t)blockIdx.y * a.M * a.N;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t row = rbase + i * 16 + r, col = cbase + j * 16;
          if (row < a.M && col < a.N) P[row * a.N + col] = acc[i][j][r];
        }
  } else {
    const float sc = __fmul_rn(__fmul_rn(*a.alpha, 1.0f / NS), *a.bscale) * (BSIGNED ? 0x1p-4f : 0x1p-3f);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t row = rbase + i * 16 + r, col = cbase + j * 16;
          if (row < a.M && col < a.N) a.C[row * a.N + col] = __fmul_rn((float)acc[i][j][r], sc);
        }
  }
}

// Sums the split-K chunk sums in int64 (fixed order) and applies the scales.
template <int NS, bool BSIGNED>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const int32_t* __restrict__ partial,
                                                            int splits, int64_t MN,
                                                            const float* alpha, const float* bscale,
                                                            float* __restrict__ C) {
  const float sc = __fmul_rn(__fmul_rn(*alpha, 1.0f / NS), *bscale) * (BSIGNED ? 0x1p-4f : 0x1p-3f);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < MN;
       i += (int64_t)gridDim.x * blockDim.x) {
    int64_t s = 0;
    for (int p = 0; p < splits; ++p) s += partial[p * MN + i];
    C[i] = __fmul_rn((float)s, sc);
  }
}

// ---- planning and launch ----------------------------------------------------------

struct GemmPlan {
  int bm, bn;
  int64_t tiles_m, tiles_n;
  int splits;
  int64_t k_chunk;
};

static GemmPlan plan_gemm(int64_t M, int64_t N, int64_t K) {
  GemmPlan p;
  p.bm = 128;
  p.bn = 128;
  p.tiles_m = (M + p.bm - 1) / p.bm;
  p.tiles_n = (N + p.bn - 1) / p.bn;
  const int64_t tiles = p.tiles_m * p.tiles_n;
  const int64_t ktiles = (K + kBK - 1) / kBK;
  int64_t splits = 1;
  // too few tiles to fill 256 CUs: split the reduction (>= 8 k-tiles each)
  if (tiles < 512) {
    splits = (512 + tiles - 1) / tiles;
    const int64_t max_by_len = ktiles / 8 > 0 ? ktiles / 8 : 1;
    if (splits > max_by_len) splits = max_by_len;
  }
  // int32-exact chunk length
  const int64_t min_splits = (K + kMaxExactK - 1) / kMaxExactK;
  if (splits < min_splits) splits = min_splits;
  if (splits < 1) splits = 1;
  int64_t chunk_tiles = (ktiles + splits - 1) / splits;
  p.k_chunk = chunk_tiles * kBK;
  p.splits = (int)((ktiles + chunk_tiles - 1) / chunk_tiles);
  return p;
}

size_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K, int /*ns*/) {
  const GemmPlan p = plan_gemm(M, N, K);
  if (p.splits <= 1) return 0;
  return (size_t)p.splits * (size_t)M * (size_t)N * sizeof(int32_t);
}

template <int NS, bool BSIGNED>
static hipError_t gemm_launch_t(const GemmArgs& a0, const GemmPlan& p, hipStream_t st) {
  GemmArgs a = a0;
  a.tiles_n = (int)p.tiles_n;
  a.k_chunk = p.k_chunk;
  const dim3 grid((unsigned)(p.tiles_m * p.tiles_n), (unsigned)p.splits);
  hipLaunchKernelGGL((gemm_luq_int4_kernel<128, 128, NS, BSIGNED>), grid, dim3(kGemmThreads), 0, st, a);
  if (p.splits > 1) {
    const int64_t MN = a.M * a.N;
    int64_t nb = (MN + 255) / 256;
    if (nb > 8192) nb = 8192;
    hipLaunchKernelGGL((splitk_reduce_kernel<NS, BSIGNED>), dim3((unsigned)nb), dim3(256), 0, st,
                       a.partial, p.splits, MN, a.alpha, a.bscale, a.C);
  }
  return hipGetLastError();
}

hipError_t launch_gemm_luq_int4(const uint8_t* A, int64_t a_plane, int ns, const float* alpha,
                                const uint8_t* B, const float* bscale, int b_signed, int64_t M,
                                int64_t N, int64_t K, float* C, void* ws, size_t /*ws_bytes*/,
                                hipStream_t st) {
  const GemmPlan p = plan_gemm(M, N, K);
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
    return b_signed ? gemm_launch_t<1, true>(a, p, st) : gemm_launch_t<1, false>(a, p, st);
  return b_signed ? gemm_launch_t<2, true>(a, p, st) : gemm_launch_t<2, false>(a, p, st);
}

}  // namespace luq

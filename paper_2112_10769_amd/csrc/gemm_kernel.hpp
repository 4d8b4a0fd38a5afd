// 4-bit GEMMs on INT8 MFMA (gfx950): the tile kernel, shared by the backward /
// update GEMMs (gemm.hip) and the forward GEMM (gemm_fwd.hip).
//
//   C[m][n] = (alpha / ns) * s_B * sum_k A[m][k] * B[n][k]
//
// A holds LUQ codes (Section 4 of the paper; ns SMP planes, Section 5.1), B
// INT4 codes (Section 3.3).  Both operands are K-major nibble matrices; the
// quantizers write whichever layout (row-major or transposed) a GEMM needs,
// so the GEMM never transposes.
//
// Carrier: v_mfma_i32_32x32x32_i8 with exact int32 accumulation.  Codes are
// expanded from nibbles to int8 once per workgroup tile, on the way from
// global memory into LDS:
//   LUQ  : a byte LUT (v_perm_b32) maps the exponent field e to 2^(e-1) (or
//          0), then bytes whose sign bit is set are negated with a SWAR
//          xor/add.  Two SMP planes are expanded to excess-64 bytes and
//          summed with one word add (|sum| <= 64, no carries).
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
#pragma once

#include "luq_device.hpp"
#include "luq_launch.hpp"

namespace luq {

// Code type of the A operand.
constexpr int kAcLuq = 0;     // LUQ codes, NS planes (Section 4, 5.1)
constexpr int kAcInt4S = 1;   // signed INT4 codes (-7..7)
constexpr int kAcInt4U = 2;   // unsigned INT4 codes (0..15)
constexpr int kAcSum2 = 3;    // int8 sums of two LUQ samples (Section 5.1), one byte per k

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));

// Word 3 of a raw buffer descriptor on gfx9 (32-bit data, no swizzle).
constexpr int kBufferFlags = 0x00020000;
// A buffer offset beyond any operand's range: such loads return zeros.
constexpr int kOutOfRange = 0x7FFFFFF0;

constexpr int kGemmThreads = 256;
constexpr int kKAlign = 128;            // k-chunk granularity of a split
// int32-exact reduction lengths: |A| <= 64 (LUQ) or 120 (INT4 as 16q / 8q),
// |B| <= 120: 2^18 * 7680 < 2^31 and 2^17 * 14400 < 2^31
constexpr int64_t kMaxExactK = 1 << 18;
constexpr int64_t kMaxExactKInt4 = 1 << 17;

// ---- nibble -> int8 expansion ------------------------------------------------

__device__ __forceinline__ void expand_luq(uint32_t x, uint32_t& lo, uint32_t& hi) {
  // bytes 0..7 of the table: 0, 1, 2, 4, 8, 16, 32, 64 (indexed by field e)
  const uint32_t t_lo = 0x04020100u, t_hi = 0x40201008u;
  const uint32_t m_lo = __builtin_amdgcn_perm(t_hi, t_lo, x & 0x07070707u);
  const uint32_t m_hi = __builtin_amdgcn_perm(t_hi, t_lo, (x >> 4) & 0x07070707u);
  // byte masks of the negative elements: v_perm_b32 selectors 8..11 copy
  // bit 7 of bytes 1 and 3 of either source into a whole byte, so with the
  // sources (y << 8, y) selector bytes (10, 8, 11, 9) give byte i = bit 7 of
  // byte i of y; y = x for the odd-k nibbles, x << 4 for the even-k ones
  constexpr uint32_t kSignSel = 0x090B080Au;
  const uint32_t y = x << 4;
  const uint32_t k_lo = __builtin_amdgcn_perm(y << 8, y, kSignSel);
  const uint32_t k_hi = __builtin_amdgcn_perm(x << 8, x, kSignSel);
  // negation = (m ^ 0xFF) + 1, which never carries out of a byte because
  // m >= 1 wherever the sign is set
  lo = (m_lo ^ k_lo) + (k_lo & 0x01010101u);
  hi = (m_hi ^ k_hi) + (k_hi & 0x01010101u);
}

// SMP operand (two LUQ planes, R <= 5 so every value is in [-32, 32]): each
// plane is expanded to excess-64 bytes u = 64 + v (a LUT of 64 + 2^(e-1),
// and 128 - that for negative codes, as (P ^ 0x7F) + 1), so that the byte
// sum u0 + u1 = 128 + v0 + v1 lies in [64, 192] and one word add carries
// nothing across bytes; flipping bit 7 then gives v0 + v1 in two's
// complement.
__device__ __forceinline__ void expand_luq_excess64(uint32_t x, uint32_t& lo, uint32_t& hi) {
  // bytes 0..7: 64 + {0, 1, 2, 4, 8, 16, 32, 64}
  const uint32_t t_lo = 0x44424140u, t_hi = 0x80605048u;
  const uint32_t p_lo = __builtin_amdgcn_perm(t_hi, t_lo, x & 0x07070707u);
  const uint32_t p_hi = __builtin_amdgcn_perm(t_hi, t_lo, (x >> 4) & 0x07070707u);
  const uint32_t s_lo = (x >> 3) & 0x01010101u, s_hi = (x >> 7) & 0x01010101u;
  lo = (p_lo ^ ((s_lo << 7) - s_lo)) + s_lo;
  hi = (p_hi ^ ((s_hi << 7) - s_hi)) + s_hi;
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

struct GemmArgs {
  const uint8_t* A;
  int64_t a_plane;
  const uint8_t* B;
  int64_t M, N, K;
  const float* alpha;
  const float* bscale;
  float* C;
  int32_t* partial;   // split-K chunk sums [splits][M][N], or null
  int64_t k_chunk;    // k per split (multiple of kKAlign)
  int tiles_m, tiles_n;
  int vec;            // rows of C (or partial) are 16-byte aligned: vector stores
};

// Block -> output tile.  Blocks are dispatched round-robin over the 8 XCDs
// (each with its own L2), so when the tile count allows, consecutive runs of
// tiles are given to one XCD; within that run tiles are visited in groups of
// 8 tile-rows so that the A rows and B rows in flight are shared.
__device__ __forceinline__ void tile_coords(int bid, int ntm, int ntn, int& tm, int& tn) {
  const int total = ntm * ntn;
  int L = bid;
  if ((total & 7) == 0) L = (bid & 7) * (total >> 3) + (bid >> 3);
  constexpr int G = 8;
  const int per_group = G * ntn;
  const int first_m = (L / per_group) * G;
  const int gsize = min(ntm - first_m, G);
  const int in_group = L - (L / per_group) * per_group;
  tm = first_m + in_group % gsize;
  tn = in_group / gsize;
}

// fl32(fl32(alpha / NS) * s_B) times the exact powers of two of the
// expansions (B: 2^-4 signed, 2^-3 unsigned; an INT4 A the same).
template <int AC, int NS, bool BSIGNED>
__device__ __forceinline__ float epilogue_scale(float alpha, float bscale) {
  constexpr float kInvSamples = AC == kAcSum2 ? 0.5f : 1.0f / NS;
  float sc = __fmul_rn(__fmul_rn(alpha, kInvSamples), bscale) * (BSIGNED ? 0x1p-4f : 0x1p-3f);
  if constexpr (AC == kAcInt4S) sc *= 0x1p-4f;
  if constexpr (AC == kAcInt4U) sc *= 0x1p-3f;
  return sc;
}

// ---- the tile kernel ----------------------------------------------------------
//
// 256 threads = 2 x 2 waves; a wave owns a (BM/2) x (BN/2) block of C as
// (BM/64) x (BN/64) tiles of the 32x32 MFMA.  Per k-stage of BK (64 or 128):
//   - the packed tile for stage t+2 is loaded into registers,
//   - stage t is multiplied out of LDS buffer t%2,
//   - stage t+1 (loaded one iteration earlier) is expanded into LDS buffer
//     (t+1)%2,
// all in one block of straight-line code, with the expansion and loads cut
// into one piece per 32-deep k-step and placed after that k-step's MFMAs, so
// the VALU work issues between MFMAs.  The MFMA takes the B fragment as its
// first operand, so each lane ends up with 4 consecutive columns of one C row.
//
// FULLK: K is a multiple of kKAlign, so every stage of a split lies inside
// the operands' rows and no chunk needs a per-lane range check; stages past
// the end of the split are then never multiplied.  Otherwise chunks past
// the split's end read as zeros and the loop may multiply one zero stage.
// The 64-deep variant keeps three waves per SIMD.
//
// AC is the A operand's code type: LUQ (NS planes), INT4 (the forward
// product, NS = 1), expanded like B, or the int8 sums of two LUQ samples
// (NS = 1): 32 bytes per 32-deep chunk, whose bytes only need the even / odd
// k split of the nibble expansions (two byte permutes per 8 values).
template <int BM, int BN, int BK, int AC, int NS, bool BSIGNED, bool FULLK>
__global__ __launch_bounds__(kGemmThreads, BK == 64 ? 3 : 1) void gemm_luq_int4_kernel(GemmArgs a) {
  static_assert(BM % 64 == 0 && BN % 64 == 0, "wave tiles are multiples of 32");
  static_assert(BK == 64 || BK == 128, "k per stage");
  constexpr int kBK = BK;
  constexpr int kPitch = BK + 16;                      // LDS row pitch in bytes
  constexpr int KC = BK / 32;                          // 16-byte chunks per row and stage
  constexpr int TM = BM / 64, TN = BN / 64;            // 32x32 MFMA tiles per wave
  constexpr int ACH = BM * KC / kGemmThreads;          // 16-byte A chunks per thread and stage
  constexpr int BCH = BN * KC / kGemmThreads;
  static_assert(ACH >= 1 && BCH >= 1, "tile too small for the block");
  constexpr int STAGE = (BM + BN) * kPitch;            // bytes of one LDS stage
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  int tm, tn;
  tile_coords(blockIdx.x, a.tiles_m, a.tiles_n, tm, tn);
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  const int64_t kbeg = (int64_t)blockIdx.y * a.k_chunk;
  const int64_t kend = min(kbeg + a.k_chunk, a.K);
  const int nkt = (int)((kend - kbeg + kBK - 1) / kBK);
  constexpr bool kI8 = AC == kAcSum2;
  constexpr int NA = kI8 ? 2 : NS;          // 16-byte A registers per chunk
  const int64_t ld = a.K >> 1;              // bytes per B row (and per nibble A row)
  const int64_t lda = kI8 ? a.K : ld;       // bytes per A row

  // Operands are read through buffer descriptors whose range is the operand
  // itself: rows past M (or N) fall outside the range, and a chunk past the
  // end of this split's k range is given an offset outside it, so both read
  // as zeros without a branch.
  __amdgpu_buffer_rsrc_t rsa[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s)
    rsa[s] = __builtin_amdgcn_make_buffer_rsrc((void*)(a.A + s * a.a_plane), (short)0,
                                               (int)(a.M * lda), kBufferFlags);
  const __amdgpu_buffer_rsrc_t rsb =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.B, (short)0, (int)(a.N * ld), kBufferFlags);
  int offa[ACH], kca[ACH], offb[BCH], kcb[BCH];
#pragma unroll
  for (int i = 0; i < ACH; ++i) {
    const int c = tid + i * kGemmThreads, row = c / KC, kc = c % KC;
    kca[i] = kc * 32;
    offa[i] = kI8 ? (int)((m0 + row) * lda + kbeg + kc * 32) : (int)((m0 + row) * ld + (kbeg >> 1) + kc * 16);
  }
#pragma unroll
  for (int i = 0; i < BCH; ++i) {
    const int c = tid + i * kGemmThreads, row = c / KC, kc = c % KC;
    kcb[i] = kc * 32;
    offb[i] = (int)((n0 + row) * ld + (kbeg >> 1) + kc * 16);
  }

  struct Regs {
    v4u a[NA][ACH];
    v4u b[BCH];
  };
  // Work of one stage is split into KS pieces, one per 32-deep k-step: piece
  // kk covers the A and B chunks i with i % KS == kk.
  constexpr int KS = kBK / 32;
  auto load_piece = [&](Regs& r, int t, int kk) {
    const int64_t k0 = kbeg + (int64_t)t * kBK;
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      if (i % KS != kk) continue;
      const bool in = FULLK || (k0 + kca[i]) < kend;
      if constexpr (kI8) {
        const int off = in ? offa[i] + t * kBK : kOutOfRange;
        r.a[0][i] = __builtin_amdgcn_raw_buffer_load_b128(rsa[0], off, 0, 0);
        r.a[1][i] = __builtin_amdgcn_raw_buffer_load_b128(rsa[0], in ? off + 16 : kOutOfRange, 0, 0);
      } else {
        const int off = in ? offa[i] + t * (kBK / 2) : kOutOfRange;
#pragma unroll
        for (int s = 0; s < NS; ++s) r.a[s][i] = __builtin_amdgcn_raw_buffer_load_b128(rsa[s], off, 0, 0);
      }
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      if (i % KS != kk) continue;
      const int off = FULLK || (k0 + kcb[i]) < kend ? offb[i] + t * (kBK / 2) : kOutOfRange;
      r.b[i] = __builtin_amdgcn_raw_buffer_load_b128(rsb, off, 0, 0);
    }
  };
  auto expand_piece = [&](const Regs& r, int buf, int kk) {
    uint8_t* As = lds + buf * STAGE;
    uint8_t* Bs = As + BM * kPitch;
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      if (i % KS != kk) continue;
      const int c = tid + i * kGemmThreads, row = c / KC, kc = c % KC;
      uint32_t w[8];
      const uint32_t x0[4] = {r.a[0][i][0], r.a[0][i][1], r.a[0][i][2], r.a[0][i][3]};
      if constexpr (kI8) {
        // bytes of k = 8d .. 8d+7 are words 2d, 2d+1 of the 32-byte chunk
        const uint32_t x[8] = {x0[0], x0[1], x0[2], x0[3], r.a[1][i][0], r.a[1][i][1], r.a[1][i][2], r.a[1][i][3]};
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          w[2 * d] = __builtin_amdgcn_perm(x[2 * d + 1], x[2 * d], 0x06040200u);      // k even
          w[2 * d + 1] = __builtin_amdgcn_perm(x[2 * d + 1], x[2 * d], 0x07050301u);  // k odd
        }
      } else if constexpr (AC != kAcLuq) {
#pragma unroll
        for (int d = 0; d < 4; ++d) expand_int4<AC == kAcInt4S>(x0[d], w[2 * d], w[2 * d + 1]);
      } else if constexpr (NS == 1) {
#pragma unroll
        for (int d = 0; d < 4; ++d) expand_luq(x0[d], w[2 * d], w[2 * d + 1]);
      } else {
        const uint32_t x1[4] = {r.a[1][i][0], r.a[1][i][1], r.a[1][i][2], r.a[1][i][3]};
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          uint32_t l0, h0, l1, h1;
          expand_luq_excess64(x0[d], l0, h0);
          expand_luq_excess64(x1[d], l1, h1);
          w[2 * d] = (l0 + l1) ^ 0x80808080u;
          w[2 * d + 1] = (h0 + h1) ^ 0x80808080u;
        }
      }
      uint4* dst = reinterpret_cast<uint4*>(As + row * kPitch + kc * 32);
      dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
      dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      if (i % KS != kk) continue;
      const int c = tid + i * kGemmThreads, row = c / KC, kc = c % KC;
      uint32_t w[8];
      const uint32_t x0[4] = {r.b[i][0], r.b[i][1], r.b[i][2], r.b[i][3]};
#pragma unroll
      for (int d = 0; d < 4; ++d) expand_int4<BSIGNED>(x0[d], w[2 * d], w[2 * d + 1]);
      uint4* dst = reinterpret_cast<uint4*>(Bs + row * kPitch + kc * 32);
      dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
      dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
    }
  };

  v16i acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = v16i{};

  // 32x32x32 MFMA operands: lane l supplies row l%32 and 16 consecutive k
  // (positions 16*(l/32) .. +15 of the 32-k step) of its fragment.
  struct Frags {
    v4i a[TM], b[TN];
  };
  auto read_frags = [&](int buf, int kk, Frags& f) {
    const uint8_t* As = lds + buf * STAGE;
    const uint8_t* as = As + (wm * (BM / 2) + (lane & 31)) * kPitch + (lane >> 5) * 16 + kk * 32;
    const uint8_t* bs = As + BM * kPitch + (wn * (BN / 2) + (lane & 31)) * kPitch + (lane >> 5) * 16 + kk * 32;
#pragma unroll
    for (int i = 0; i < TM; ++i) f.a[i] = *reinterpret_cast<const v4i*>(as + i * 32 * kPitch);
#pragma unroll
    for (int j = 0; j < TN; ++j) f.b[j] = *reinterpret_cast<const v4i*>(bs + j * 32 * kPitch);
  };
  auto mfmas = [&](const Frags& f) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(f.b[j], f.a[i], acc[i][j], 0, 0, 0);
  };

  // One pipeline step, straight-line code between barriers: for each k-step
  // of stage `cb` (in LDS), the fragments of the next k-step are read ahead,
  // the MFMAs of this k-step issue, and one piece of the next stage (the
  // registers `r`) is expanded into the other buffer, after which that
  // piece's registers are reloaded from stage `tload` into `rl`.  Source
  // order interleaves the expansion work with the MFMAs.
  auto step = [&](int cb, const Regs& r, Regs& rl, int tload) {
    Frags f[2];
    read_frags(cb, 0, f[0]);
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      if (kk + 1 < KS) read_frags(cb, kk + 1, f[(kk + 1) & 1]);
      mfmas(f[kk & 1]);
      expand_piece(r, cb ^ 1, kk);
      load_piece(rl, tload, kk);
    }
    __syncthreads();
  };

  Regs r0, r1;
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) load_piece(r0, 0, kk);
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) load_piece(r1, 1, kk);
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) expand_piece(r0, 0, kk);
  __syncthreads();
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) load_piece(r0, 2, kk);
  int t = 0;
  for (; t + 2 <= nkt; t += 2) {
    step(0, r1, r1, t + 3);   // multiply t, expand t+1 (r1), then reuse r1 for t+3
    step(1, r0, r0, t + 4);   // multiply t+1, expand t+2 (r0), then reuse r0 for t+4
  }
  // an odd stage count leaves stage t in buffer 0 (with FULLK the stage
  // expanded beside it may hold another split's codes; it is not multiplied)
  if (t < nkt) step(0, r1, r1, t + 3);

  // Epilogue through LDS.  In MFMA tile (i, j), lane l holds row l%32 and, in
  // registers 4q..4q+3, the 4 consecutive columns 8q + 4*(l/32) + 0..3 (the
  // swapped operands).  Each wave stages 32 rows of its block at a time as a
  // row-major slab in its own part of the (now idle) stage buffers, then
  // stores whole row segments: WN/4 consecutive lanes cover one row of the
  // wave's block, so a store instruction writes 64*16/WN-row runs of
  // contiguous 16-byte chunks.  C gets the scaled fp32 values, the split-K
  // workspace the raw int32 sums.
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int EP = WN + 4;      // slab row pitch in 32-bit words
  constexpr int LPR = WN / 4;     // lanes per row in the store phase
  constexpr int RPI = 64 / LPR;   // rows per store instruction (lanes past RPI * LPR idle)
  static_assert(4 * 32 * EP * 4 <= 2 * STAGE, "epilogue slabs fit in the stage buffers");
  static_assert(WM % 32 == 0 && LPR <= 64 && 32 % RPI == 0, "slab shape");
  uint32_t* E = reinterpret_cast<uint32_t*>(lds) + wave * 32 * EP;
  const bool part = a.partial != nullptr;
  const float sc = part ? 0.0f : epilogue_scale<AC, NS, BSIGNED>(*a.alpha, *a.bscale);
  uint32_t* out = part ? reinterpret_cast<uint32_t*>(a.partial + (int64_t)blockIdx.y * a.M * a.N)
                       : reinterpret_cast<uint32_t*>(a.C);
  const int64_t rbase = m0 + wm * WM, cbase = n0 + wn * WN;
  const int srow = lane / LPR, scol = (lane % LPR) * 4;
  const bool sact = lane < RPI * LPR;
  __syncthreads();  // every wave is done with the stage buffers
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v4u v;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int32_t x = acc[i][j][4 * q + r];
          v[r] = part ? (uint32_t)x : __float_as_uint(__fmul_rn((float)x, sc));
        }
        *reinterpret_cast<v4u*>(E + (lane & 31) * EP + j * 32 + 8 * q + 4 * (lane >> 5)) = v;
      }
    __syncthreads();
#pragma unroll
    for (int rr = 0; rr < 32; rr += RPI) {
      const int64_t row = rbase + i * 32 + rr + srow;
      const int64_t col = cbase + scol;
      if (sact && row < a.M) {
        const v4u v = *reinterpret_cast<const v4u*>(E + (rr + srow) * EP + scol);
        uint32_t* dst = out + row * a.N + col;
        if (a.vec && col + 3 < a.N) {
          *reinterpret_cast<v4u*>(dst) = v;
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (col + r < a.N) dst[r] = v[r];
        }
      }
    }
    __syncthreads();  // the slab is rewritten by the next i
  }
}

// ---- the 256 x 256 tile: eight waves, the B operand in registers ---------------
//
// 512 threads = 2 x 4 waves; a wave owns a 128 x 64 block of C (4 x 2 tiles of
// the 32x32 MFMA), so two waves share each SIMD and the expansion, address and
// LDS work of one overlaps the MFMAs of the other.  Only A passes through LDS,
// expanded to int8 once per workgroup (the LUQ expansion is the costly one,
// and LDS stores run at a quarter of the LDS read rate).  Each wave loads the
// nibbles of its own 64 B rows straight into registers (the wave of the other
// row half loads the same rows) and expands every fragment just before its
// MFMAs, which is a shift and a mask per word.
//
// k order: a 128-deep stage is 64 nibble bytes of every row.  At k-step kk,
// lane half h = lane/32 supplies the k of nibble bytes 32h + 8kk .. +7 of the
// stage, for both operands, so a lane's B nibbles of a whole stage are one
// contiguous 32-byte segment.  The products summed are the same, in another
// order.  A sits in LDS as 8 slots of 16 expanded bytes per row, slot 2kk + h
// holding those k.
//
// Pipeline (one barrier per stage): stage t is multiplied from LDS buffer t%2
// with B registers set t%2, while the A codes of stage t+1 are expanded into
// the other buffer; each A chunk and each B half-segment is reloaded (A with
// stage t+3, B with stage t+2) as soon as its registers are consumed.
//
// PF sets how far ahead the MFMA operands are fetched, so that the LDS read
// latency is covered by the previous k-step's MFMAs:
//   0: each k-step's fragments are read and expanded just before its MFMAs;
//   1: the A fragments of k-step kk+1 are read while kk is multiplied;
//   2: as 1, and the B fragments of kk+1 are expanded during kk too;
//   3: as 2 across the stage boundary as well (the next stage's first B
//      fragments at the last k-step), with the B reload one k-step earlier.
// Every mode sums the same products; the launcher picks the deepest mode that
// fits the 256 registers of two waves per SIMD for the operand kinds.
constexpr int kW8Threads = 512;

template <int AC, int NS, bool BSIGNED, bool FULLK, int PF>
__global__ __launch_bounds__(kW8Threads, 1) void gemm_w8_kernel(GemmArgs a) {
  constexpr int BM = 256, kBK = 128, kThr = kW8Threads;
  constexpr int kPitch = kBK + 16;        // A row: 8 slots of 16 bytes, 16 bytes of pad
  constexpr int STAGE = BM * kPitch;
  constexpr int TM = 4, TN = 2;           // 32x32 tiles per wave
  constexpr int ACH = BM * 4 / kThr;      // 16-byte A chunks per thread and stage
  constexpr bool kI8 = AC == kAcSum2;
  constexpr int NA = kI8 ? 2 : NS;
  static_assert(ACH == 2, "one A half-chunk per k-step");
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3, h = lane >> 5;
  int tm, tn;
  tile_coords(blockIdx.x, a.tiles_m, a.tiles_n, tm, tn);
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * 256;
  const int64_t kbeg = (int64_t)blockIdx.y * a.k_chunk;
  const int64_t kend = min(kbeg + a.k_chunk, a.K);
  const int nkt = (int)((kend - kbeg + kBK - 1) / kBK);
  const int64_t ld = a.K >> 1;              // bytes per B row (and per nibble A row)
  const int64_t lda = kI8 ? a.K : ld;       // bytes per A row

  __amdgpu_buffer_rsrc_t rsa[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s)
    rsa[s] = __builtin_amdgcn_make_buffer_rsrc((void*)(a.A + s * a.a_plane), (short)0,
                                               (int)(a.M * lda), kBufferFlags);
  const __amdgpu_buffer_rsrc_t rsb =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.B, (short)0, (int)(a.N * ld), kBufferFlags);
  // A loader: chunk i of a thread is row c/4, 16 nibble bytes (32 k) at 16*(c%4)
  int offa[ACH], kca[ACH], slota[ACH], rowa[ACH];
#pragma unroll
  for (int i = 0; i < ACH; ++i) {
    const int c = tid + i * kThr, row = c >> 2, kc = c & 3;
    kca[i] = kc * 32;
    rowa[i] = row;
    slota[i] = 4 * (kc & 1) + (kc >> 1);  // slot of the chunk's first half; the second is 2 further
    offa[i] = kI8 ? (int)((m0 + row) * lda + kbeg + kc * 32) : (int)((m0 + row) * ld + (kbeg >> 1) + kc * 16);
  }
  // B: rows n0 + 64wn + 32j + lane%32, the 32-byte segment 32h of each stage
  int offb[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) offb[j] = (int)((n0 + wn * 64 + j * 32 + (lane & 31)) * ld + (kbeg >> 1) + h * 32);

  struct ARegs {
    v4u a[NA][ACH];
  };
  struct BRegs {
    v4u b[TN][2];
  };
  auto load_a = [&](ARegs& r, int t, int i) {
    const int64_t k0 = kbeg + (int64_t)t * kBK;
    const bool in = FULLK || (k0 + kca[i]) < kend;
    if constexpr (kI8) {
      const int off = in ? offa[i] + t * kBK : kOutOfRange;
      r.a[0][i] = __builtin_amdgcn_raw_buffer_load_b128(rsa[0], off, 0, 0);
      r.a[1][i] = __builtin_amdgcn_raw_buffer_load_b128(rsa[0], in ? off + 16 : kOutOfRange, 0, 0);
    } else {
      const int off = in ? offa[i] + t * (kBK / 2) : kOutOfRange;
#pragma unroll
      for (int s = 0; s < NS; ++s) r.a[s][i] = __builtin_amdgcn_raw_buffer_load_b128(rsa[s], off, 0, 0);
    }
  };
  auto load_b = [&](BRegs& r, int t, int q) {
    const bool in = FULLK || (kbeg + (int64_t)t * kBK + h * 64 + q * 32) < kend;
#pragma unroll
    for (int j = 0; j < TN; ++j)
      r.b[j][q] = __builtin_amdgcn_raw_buffer_load_b128(rsb, in ? offb[j] + t * (kBK / 2) + q * 16 : kOutOfRange, 0, 0);
  };
  // half hf of A chunk i (its k 16hf .. 16hf+15) -> 16 bytes of LDS
  auto expand_a = [&](const ARegs& r, int buf, int i, int hf) {
    uint32_t w[4];
    if constexpr (kI8) {
      const v4u x = r.a[hf][i];
      w[0] = __builtin_amdgcn_perm(x[1], x[0], 0x06040200u);  // k even
      w[1] = __builtin_amdgcn_perm(x[1], x[0], 0x07050301u);  // k odd
      w[2] = __builtin_amdgcn_perm(x[3], x[2], 0x06040200u);
      w[3] = __builtin_amdgcn_perm(x[3], x[2], 0x07050301u);
    } else if constexpr (AC != kAcLuq) {
      expand_int4<AC == kAcInt4S>(r.a[0][i][2 * hf], w[0], w[1]);
      expand_int4<AC == kAcInt4S>(r.a[0][i][2 * hf + 1], w[2], w[3]);
    } else if constexpr (NS == 1) {
      expand_luq(r.a[0][i][2 * hf], w[0], w[1]);
      expand_luq(r.a[0][i][2 * hf + 1], w[2], w[3]);
    } else {
#pragma unroll
      for (int d = 0; d < 2; ++d) {
        uint32_t l0, h0, l1, h1;
        expand_luq_excess64(r.a[0][i][2 * hf + d], l0, h0);
        expand_luq_excess64(r.a[1][i][2 * hf + d], l1, h1);
        w[2 * d] = (l0 + l1) ^ 0x80808080u;
        w[2 * d + 1] = (h0 + h1) ^ 0x80808080u;
      }
    }
    *reinterpret_cast<uint4*>(lds + buf * STAGE + rowa[i] * kPitch + ((slota[i] + 2 * hf) << 4)) =
        make_uint4(w[0], w[1], w[2], w[3]);
  };

  v16i acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = v16i{};

  // A fragment i of k-step kk: row 128wm + 32i + lane%32, slot 2kk + h
  const int aoff = (wm * 128 + (lane & 31)) * kPitch + (h << 4);
  auto read_a = [&](int buf, int kk, v4i (&fa)[TM]) {
    const uint8_t* as = lds + buf * STAGE + aoff + (kk << 5);
#pragma unroll
    for (int i = 0; i < TM; ++i) fa[i] = *reinterpret_cast<const v4i*>(as + i * 32 * kPitch);
  };
  // B fragment j of k-step kk: nibble dwords 2kk, 2kk+1 of the lane's segment
  auto frag_b = [&](const BRegs& r, int kk, v4i (&fb)[TN]) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      uint32_t l0, h0, l1, h1;
      expand_int4<BSIGNED>(r.b[j][kk >> 1][2 * (kk & 1)], l0, h0);
      expand_int4<BSIGNED>(r.b[j][kk >> 1][2 * (kk & 1) + 1], l1, h1);
      fb[j] = v4i{(int)l0, (int)h0, (int)l1, (int)h1};
    }
  };

  // fragments fetched one k-step ahead (PF >= 1), carried across stages (PF 3)
  v4i fa2[2][TM], fb2[2][TN];
  auto mma = [&](const v4i (&fa)[TM], const v4i (&fb)[TN]) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fb[j], fa[i], acc[i][j], 0, 0, 0);
  };
  // multiply stage t from buffer cb and B set rb while expanding the A codes
  // of stage t+1 (ra) into the other buffer; rbn is the next stage's B set
  auto step = [&](int cb, ARegs& ra, int ta, BRegs& rb, int tb, const BRegs& rbn) {
    if constexpr (PF >= 1) read_a(cb, 0, fa2[0]);
    if constexpr (PF == 2) frag_b(rb, 0, fb2[0]);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      // the first B half-segment and A chunk are consumed: reload them now
      // (the scheduler would otherwise sink the loads to the barrier)
      if (kk == (PF == 3 ? 1 : 2)) {
        load_b(rb, tb, 0);
        if (PF != 3) load_a(ra, ta, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (PF == 3 && kk == 2) {
        load_a(ra, ta, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
      if constexpr (PF == 0) {
        v4i fa[TM], fb[TN];
        read_a(cb, kk, fa);
        frag_b(rb, kk, fb);
        mma(fa, fb);
      } else if constexpr (PF == 1) {
        v4i fb[TN];
        if (kk + 1 < 4) read_a(cb, kk + 1, fa2[(kk + 1) & 1]);
        frag_b(rb, kk, fb);
        mma(fa2[kk & 1], fb);
      } else {
        if (kk + 1 < 4) {
          read_a(cb, kk + 1, fa2[(kk + 1) & 1]);
          frag_b(rb, kk + 1, fb2[(kk + 1) & 1]);
        } else if (PF == 3) {
          frag_b(rbn, 0, fb2[0]);
        }
        mma(fa2[kk & 1], fb2[kk & 1]);
      }
      expand_a(ra, cb ^ 1, kk >> 1, kk & 1);
    }
    load_b(rb, tb, 1);
    load_a(ra, ta, 1);
    __syncthreads();
    // keep the next stage's work below the barrier: hoisted above it, the
    // expansion of registers loaded in this stage would wait for those loads
    __builtin_amdgcn_sched_barrier(0);
  };

  ARegs r0, r1;
  BRegs b0, b1;
#pragma unroll
  for (int i = 0; i < ACH; ++i) load_a(r0, 0, i);
  load_b(b0, 0, 0);
  load_b(b0, 0, 1);
#pragma unroll
  for (int i = 0; i < ACH; ++i) load_a(r1, 1, i);
  load_b(b1, 1, 0);
  load_b(b1, 1, 1);
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) expand_a(r0, 0, kk >> 1, kk & 1);
  if constexpr (PF == 3) frag_b(b0, 0, fb2[0]);
  __syncthreads();
#pragma unroll
  for (int i = 0; i < ACH; ++i) load_a(r0, 2, i);
  int t = 0;
  for (; t + 2 <= nkt; t += 2) {
    step(0, r1, t + 3, b0, t + 2, b1);  // multiply t, expand t+1 (r1); reload r1 with t+3, b0 with t+2
    step(1, r0, t + 4, b1, t + 3, b0);  // multiply t+1, expand t+2 (r0); reload r0 with t+4, b1 with t+3
  }
  if (t < nkt) step(0, r1, t + 3, b0, t + 2, b1);

  // Epilogue through LDS, as in the four-wave kernel: each wave stages 32 rows
  // of its 128 x 64 block at a time and stores whole 256-byte row segments.
  constexpr int WN = 64;
  constexpr int EP = WN + 4;
  constexpr int LPR = WN / 4, RPI = 64 / LPR;
  static_assert(8 * 32 * EP * 4 <= 2 * STAGE, "epilogue slabs fit in the stage buffers");
  uint32_t* E = reinterpret_cast<uint32_t*>(lds) + wave * 32 * EP;
  const bool part = a.partial != nullptr;
  const float sc = part ? 0.0f : epilogue_scale<AC, NS, BSIGNED>(*a.alpha, *a.bscale);
  uint32_t* out = part ? reinterpret_cast<uint32_t*>(a.partial + (int64_t)blockIdx.y * a.M * a.N)
                       : reinterpret_cast<uint32_t*>(a.C);
  const int64_t rbase = m0 + wm * 128, cbase = n0 + wn * WN;
  const int srow = lane / LPR, scol = (lane % LPR) * 4;
  __syncthreads();  // every wave is done with the stage buffers
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v4u v;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int32_t x = acc[i][j][4 * q + r];
          v[r] = part ? (uint32_t)x : __float_as_uint(__fmul_rn((float)x, sc));
        }
        *reinterpret_cast<v4u*>(E + (lane & 31) * EP + j * 32 + 8 * q + 4 * (lane >> 5)) = v;
      }
    __syncthreads();
#pragma unroll
    for (int rr = 0; rr < 32; rr += RPI) {
      const int64_t row = rbase + i * 32 + rr + srow;
      const int64_t col = cbase + scol;
      if (row < a.M) {
        const v4u v = *reinterpret_cast<const v4u*>(E + (rr + srow) * EP + scol);
        uint32_t* dst = out + row * a.N + col;
        if (a.vec && col + 3 < a.N) {
          *reinterpret_cast<v4u*>(dst) = v;
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (col + r < a.N) dst[r] = v[r];
        }
      }
    }
    __syncthreads();  // the slab is rewritten by the next i
  }
}

// Sums the split-K chunk sums in int64 and applies the scales.  A block owns
// 64 consecutive outputs; its four waves add every fourth chunk (coalesced
// 256-byte reads), then combine through LDS in a fixed order.
template <int AC, int NS, bool BSIGNED>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const int32_t* __restrict__ partial,
                                                            int splits, int64_t MN,
                                                            const float* alpha, const float* bscale,
                                                            float* __restrict__ C) {
  __shared__ int64_t part[4][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t i = (int64_t)blockIdx.x * 64 + lane;
  int64_t s = 0;
  if (i < MN) {
    int p = wave;
    for (; p + 12 < splits; p += 16) {
      const int32_t v0 = partial[(int64_t)p * MN + i], v1 = partial[(int64_t)(p + 4) * MN + i];
      const int32_t v2 = partial[(int64_t)(p + 8) * MN + i], v3 = partial[(int64_t)(p + 12) * MN + i];
      s += (int64_t)v0 + v1 + v2 + v3;
    }
    for (; p < splits; p += 4) s += partial[(int64_t)p * MN + i];
  }
  part[wave][lane] = s;
  __syncthreads();
  if (wave == 0 && i < MN) {
    const int64_t tot = part[0][lane] + part[1][lane] + part[2][lane] + part[3][lane];
    const float sc = epilogue_scale<AC, NS, BSIGNED>(*alpha, *bscale);
    C[i] = __fmul_rn((float)tot, sc);
  }
}

// ---- planning and launch ----------------------------------------------------------

struct GemmPlan {
  int bm, bn, bk;
  int64_t tiles_m, tiles_n;
  int splits;
  int64_t k_chunk;
};

static GemmPlan plan_gemm(int64_t M, int64_t N, int64_t K, int64_t max_exact_k) {
  GemmPlan p;
  auto tiles = [&](int bm, int bn) { return ((M + bm - 1) / bm) * ((N + bn - 1) / bn); };
  // 256x256 tiles (the eight-wave kernel, one workgroup per CU) halve the
  // expansion and LDS work per MAC; they pay off for long reductions.  Short
  // reductions (the conv dX with K = 64) are bound by the fp32 output and
  // prefer the 128x128 tile, which keeps two workgroups per CU.
  if (K >= 1024 && tiles(256, 256) >= 256) {
    p.bm = 256;
    p.bn = 256;
  } else if (M <= 64 && N >= 192 && K >= 65536) {
    // few output rows and a long reduction (the conv dW: 64 x 576 x 200704):
    // wide tiles so that the A rows are re-read for fewer column tiles
    p.bm = 64;
    p.bn = 192;
  } else if (tiles(128, 128) >= 128) {
    p.bm = 128;
    p.bn = 128;
  } else {
    p.bm = 64;
    p.bn = 64;
  }
  // a reduction of at most 64 fits one 64-deep stage: half the LDS, so more
  // workgroups per CU overlap their loads with other tiles' output stores
  p.bk = (K <= 64 && p.bm == 128) ? 64 : 128;
  p.tiles_m = (M + p.bm - 1) / p.bm;
  p.tiles_n = (N + p.bn - 1) / p.bn;
  const int64_t nt = p.tiles_m * p.tiles_n;
  const int64_t ktiles = (K + kKAlign - 1) / kKAlign;
  int64_t splits = 1;
  // too few tiles to fill 256 CUs: split the reduction (>= 8 k-stages each);
  // the wide tiles aim at one workgroup per CU, since every split adds
  // M x N partial sums to write and read back
  if (nt < 256) {
    const int64_t target = p.bn == 192 ? 256 : 512;
    splits = (target + nt - 1) / nt;
    const int64_t max_by_len = ktiles / 8 > 0 ? ktiles / 8 : 1;
    if (splits > max_by_len) splits = max_by_len;
  }
  // int32-exact chunk length
  const int64_t min_splits = (K + max_exact_k - 1) / max_exact_k;
  if (splits < min_splits) splits = min_splits;
  if (splits < 1) splits = 1;
  const int64_t chunk_tiles = (ktiles + splits - 1) / splits;
  p.k_chunk = chunk_tiles * kKAlign;
  p.splits = (int)((ktiles + chunk_tiles - 1) / chunk_tiles);
  return p;
}

template <int BM, int BN, int BK, int AC, int NS, bool BSIGNED>
static void launch_tile(const GemmArgs& a, dim3 grid, hipStream_t st) {
  if (a.K % kKAlign == 0)
    hipLaunchKernelGGL((gemm_luq_int4_kernel<BM, BN, BK, AC, NS, BSIGNED, true>), grid, dim3(kGemmThreads), 0, st, a);
  else
    hipLaunchKernelGGL((gemm_luq_int4_kernel<BM, BN, BK, AC, NS, BSIGNED, false>), grid, dim3(kGemmThreads), 0, st,
                       a);
}

template <int AC, int NS, bool BSIGNED>
static hipError_t gemm_launch_t(const GemmArgs& a0, const GemmPlan& p, hipStream_t st) {
  GemmArgs a = a0;
  a.tiles_m = (int)p.tiles_m;
  a.tiles_n = (int)p.tiles_n;
  a.k_chunk = p.k_chunk;
  const dim3 grid((unsigned)(p.tiles_m * p.tiles_n), (unsigned)p.splits);
  // 16-byte stores need 16-byte aligned rows
  a.vec = (a.N % 4) == 0 && (((uintptr_t)(a.partial ? (void*)a.partial : (void*)a.C)) & 15) == 0;
  if (p.bm == 256) {
    // prefetch depth by register budget (deeper modes spill where not taken)
    constexpr bool kLuq1 = AC == kAcLuq && NS == 1;
    constexpr int kPfFull = AC == kAcSum2 ? (BSIGNED ? 3 : 2) : kLuq1 ? 2 : 1;
    constexpr int kPfPart = AC == kAcSum2 || kLuq1 ? 2 : AC == kAcLuq ? 0 : 1;
    if (a.K % kKAlign == 0)
      hipLaunchKernelGGL((gemm_w8_kernel<AC, NS, BSIGNED, true, kPfFull>), grid, dim3(kW8Threads), 0, st, a);
    else
      hipLaunchKernelGGL((gemm_w8_kernel<AC, NS, BSIGNED, false, kPfPart>), grid, dim3(kW8Threads), 0, st, a);
  }
  else if (p.bm == 128 && p.bk == 64)
    launch_tile<128, 128, 64, AC, NS, BSIGNED>(a, grid, st);
  else if (p.bm == 128)
    launch_tile<128, 128, 128, AC, NS, BSIGNED>(a, grid, st);
  else if (p.bn == 192)
    launch_tile<64, 192, 128, AC, NS, BSIGNED>(a, grid, st);
  else
    launch_tile<64, 64, 128, AC, NS, BSIGNED>(a, grid, st);
  if (p.splits > 1) {
    const int64_t MN = a.M * a.N;
    hipLaunchKernelGGL((splitk_reduce_kernel<AC, NS, BSIGNED>), dim3((unsigned)((MN + 63) / 64)), dim3(256), 0, st,
                       a.partial, p.splits, MN, a.alpha, a.bscale, a.C);
  }
  return hipGetLastError();
}

}  // namespace luq

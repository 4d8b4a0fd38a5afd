// 4-bit GEMMs on the FP6 carrier (gfx950 v_mfma_scale_f32_32x32x64_f8f6f4,
// 10.1 PF dense against INT8's 5.0 POPS):
//
//   C[m][n] = (alpha / ns) * s_B * sum_k A[m][k] * B[n][k]
//
// with A the LUQ codes of a neural gradient (Section 4) and B INT4 codes
// (Section 3.3), as in gemm_kernel.hpp, whose results this path reproduces
// bit for bit.
//
// Carrier.  Both 4-bit code sets are exact in FP6, and the conversion is a
// bit spread with no arithmetic:
//   LUQ nibble (sign bit 3, exponent field e in bits 0..2) shifted left by 2
//   is the e3m2 code of (-1)^s 2^(e-3) (e = 0 gives +0): the LUQ level
//   alpha 2^(e-1) over 4 alpha, for every e <= 7 (R <= 6);
//   an unsigned INT4 nibble q is the e2m3 code of q/8 (codes 0..7 are the
//   subnormals 0..7/8, codes 8..15 the binade 1..15/8); a signed code -7..7
//   is the e2m3 code of sign and |q|/8.
// So every product is A_true * B_true * 2^-5 (LUQ x INT4) and, while
// sum_k |A_true B_true| < 2^24, every partial sum is a multiple of 2^-5 below
// 2^19: the fp32 accumulation is exact whatever its order.  With |A_true| <=
// 2^6 and |B_true| <= 15 that holds for reductions of up to 16384; longer ones
// are split and the exact partial sums combined in int64.
//
// Layout.  A pre-pass converts each operand once (not once per tile) into
// fragment-major blocks of 32 rows x 64 k (1536 bytes): lane l of the MFMA
// operand holds row l%32, k = 32 (l/32) + i for i = 0..31, as 32 six-bit codes
// (192 bits, code i at bit 6i); the block stores dwords 0..3 of the 64 lanes
// (1024 bytes) and then dwords 4..5 (512 bytes), so that a wave reads a
// fragment with one 16-byte and one 8-byte LDS read per lane, both
// conflict-free.  Blocks are stored [k block][row block], so the blocks a
// stage of one tile reads are contiguous runs and the tiles in flight read
// neighbouring runs (with [row block][k block] the row blocks of one k block
// sit a multiple of every power-of-two interleave apart, and all of them fell
// on one L2 channel); rows and k past the matrix hold code 0.
//
// GEMM.  A workgroup of 4 waves (2 x 2) owns a BM x BN tile; per stage of
// 128 k its A and B blocks go from global memory straight into a ring of
// three LDS buffers (direct-to-LDS 16-byte loads, no registers, no
// conversion) two stages ahead of the one being multiplied; each wave
// multiplies its (BM/2) x (BN/2) block with the 32x32x64 MFMA.
// The epilogue maps the exact fp32 sums onto the INT8 carrier's integer sums
// (an exact power-of-two scale) and applies the same fp32 scale arithmetic,
// so C equals luq_gemm_dgrad / luq_gemm_wgrad's INT8 result bit for bit.
#include "gemm_kernel.hpp"

namespace luq {

constexpr int kF6Block = 1536;        // bytes of one 32 x 64 fragment block
constexpr int kF6Part1 = 1024;        // offset of lane dwords 4..5 in a block
constexpr int kF6KB = 2;              // k blocks (of 64) per pipeline stage
constexpr int kF6Bufs = 3;            // LDS stage buffers (a ring)
constexpr int64_t kMaxExactKFp6 = 16384;

// e3m2 / e2m3 format codes of the scaled MFMA's operand-format fields
constexpr int kFmtE2M3 = 2;
constexpr int kFmtE3M2 = 3;
constexpr int kScaleOne = 127;        // E8M0 2^0

// Code kinds of the pre-pass.
constexpr int kF6Luq = 0;             // LUQ -> e3m2
constexpr int kF6Int4S = 1;           // signed INT4 -> e2m3 (sign and magnitude)
constexpr int kF6Int4U = 2;           // unsigned INT4 -> e2m3

// Eight codes of a word (nibble i at bits 4i) into eight 6-bit slots (slot i
// at bits 6i of the 48-bit lo:hi), the nibble at the slot's bit 0, or (S = 2)
// at its bit 2.  Even and odd bytes are spread in separate 16-bit halves so
// no shifted nibble lands on another.
template <int S>
__device__ __forceinline__ void spread6(uint32_t x, uint32_t& lo, uint32_t& hi) {
  const uint32_t xe = x & 0x00FF00FFu, xo = (x >> 8) & 0x00FF00FFu;
  // a byte (two nibbles) becomes a 12-bit group: slot 2j at 0..5, 2j+1 at 6..11
  const uint32_t ye = ((xe & 0x000F000Fu) << S) | ((xe & 0x00F000F0u) << (2 + S));
  const uint32_t yo = ((xo & 0x000F000Fu) << S) | ((xo & 0x00F000F0u) << (2 + S));
  // groups: bytes 0 and 2 in ye's halves, bytes 1 and 3 in yo's
  lo = (ye & 0xFFFu) | ((yo & 0xFFFu) << 12) | (ye >> 16 << 24);
  hi = (ye >> 24) | (yo >> 16 << 4);
}

// The 6-bit codes of 8 nibbles of kind KIND, packed as spread6 does.
template <int KIND>
__device__ __forceinline__ void fp6_codes8(uint32_t x, uint32_t& lo, uint32_t& hi) {
  if constexpr (KIND == kF6Luq) {
    spread6<2>(x, lo, hi);
  } else if constexpr (KIND == kF6Int4U) {
    spread6<0>(x, lo, hi);
  } else {
    // two's complement nibbles -7..7 -> magnitude (bits 0..2) and sign (bit 3),
    // spread, then the sign moved from slot bit 3 to slot bit 5
    const uint32_t s = (x >> 3) & 0x11111111u;
    const uint32_t mag = ((x ^ ((s << 4) - s)) + s) | (s << 3);  // no carry: a negative nibble is >= 9
    spread6<0>(mag, lo, hi);
    constexpr uint32_t kLo3 = 0x08208208u, kHi3 = 0x2082u;       // bit 3 of slots 0..4 / 5..7
    lo = (lo & ~kLo3) | ((lo & kLo3) << 2);
    hi = (hi & ~kHi3) | ((hi & kHi3) << 2);
  }
}

// Pre-pass: one thread per (row block, k block, lane).  Reads the lane's 32
// codes (16 bytes of a K-major nibble row) and writes its 24 bytes of the
// fragment block.  Consecutive waves take consecutive k blocks of one row
// block, so a workgroup reads 128 contiguous bytes of each row.
template <int KIND>
__global__ __launch_bounds__(256) void fp6_pack_kernel(const uint8_t* __restrict__ src, int64_t rows, int64_t K,
                                                      int64_t nkb, int64_t nrb, uint8_t* __restrict__ dst) {
  const int64_t nblocks = nrb * nkb;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t blk = t >> 6;
  if (blk >= nblocks) return;
  const int lane = (int)(t & 63);
  const int64_t rb = blk / nkb, kb = blk - rb * nkb;
  const int64_t row = rb * 32 + (lane & 31);
  const int64_t k0 = kb * 64 + 32 * (lane >> 5);
  v4u x = {0u, 0u, 0u, 0u};
  if (row < rows && k0 < K) x = *reinterpret_cast<const v4u*>(src + row * (K >> 1) + (k0 >> 1));
  uint32_t lo[4], hi[4];
#pragma unroll
  for (int d = 0; d < 4; ++d) fp6_codes8<KIND>(x[d], lo[d], hi[d]);
  // 48-bit pieces at bits 0, 48, 96, 144 of the lane's 192 bits
  const v4u p0 = {lo[0], hi[0] | (lo[1] << 16), __builtin_amdgcn_alignbit(hi[1], lo[1], 16), lo[2]};
  const v2u32 p1 = {hi[2] | (lo[3] << 16), __builtin_amdgcn_alignbit(hi[3], lo[3], 16)};
  uint8_t* b = dst + (kb * nrb + rb) * kF6Block;
  *reinterpret_cast<v4u*>(b + 16 * lane) = p0;
  *reinterpret_cast<v2u32*>(b + kF6Part1 + 8 * lane) = p1;
}

struct Fp6GemmArgs {
  const uint8_t* A;     // fragment blocks of A [ceil(M/32)][nkb]
  const uint8_t* B;     // fragment blocks of B [ceil(N/32)][nkb]
  int64_t M, N;
  int nkb;              // k blocks per row (K rounded up to 64, / 64)
  int kb_chunk;         // k blocks per split (a multiple of kF6KB)
  int a_bytes, b_bytes; // operand sizes (buffer ranges)
  const float* alpha;
  const float* bscale;
  float* C;
  int32_t* partial;     // split sums [splits][M][N] on the INT8 carrier's scale, or null
  int tiles_m, tiles_n;
  int vec;
};

typedef int v2i __attribute__((ext_vector_type(2)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

// FA / FB: MFMA formats of A and B; AC, BSIGNED: the INT8 carrier the result
// is mapped onto (its epilogue scale); kToCarrier = the INT8 carrier's sum
// over the fp32 sum (an exact power of two).
template <int BM, int BN, int FA, int FB, int AC, bool BSIGNED>
__global__ __launch_bounds__(256, 1) void gemm_fp6_kernel(Fp6GemmArgs a) {
  constexpr int RA = BM / 32, RB = BN / 32;           // row blocks of the tile
  constexpr int TM = BM / 64, TN = BN / 64;           // 32x32 MFMA tiles per wave
  constexpr int STAGE = (RA + RB) * kF6KB * kF6Block;
  constexpr int NCH = STAGE / 16;                      // 16-byte chunks per stage
  constexpr int CH = NCH / 256;                        // per thread
  static_assert(NCH % 256 == 0, "whole chunks per thread");
  constexpr int kBlkCh = kF6Block / 16;                // 96 chunks per block
  constexpr int CHA = RA * kF6KB * kBlkCh / 256;       // rounds of A chunks (then B)
  static_assert(RA * kF6KB * kBlkCh % 256 == 0, "a load round reads one operand");
  __shared__ __attribute__((aligned(16))) uint8_t lds[kF6Bufs * STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  int tm, tn;
  tile_coords(blockIdx.x, a.tiles_m, a.tiles_n, tm, tn);
  const int rb0 = tm * RA, nb0 = tn * RB;
  const int kb_beg = blockIdx.y * a.kb_chunk;
  const int kb_end = min(kb_beg + a.kb_chunk, a.nkb);
  const int nst = (kb_end - kb_beg + kF6KB - 1) / kF6KB;
  const int rows_a = (int)((a.M + 31) >> 5), rows_b = (int)((a.N + 31) >> 5);

  const __amdgpu_buffer_rsrc_t rsa = __builtin_amdgcn_make_buffer_rsrc((void*)a.A, (short)0, a.a_bytes, kBufferFlags);
  const __amdgpu_buffer_rsrc_t rsb = __builtin_amdgcn_make_buffer_rsrc((void*)a.B, (short)0, a.b_bytes, kBufferFlags);

  // The stage image in LDS: A blocks [kbl][rbl], then B blocks [kbl][rbl].
  // Chunk c = tid + 256 i of the image comes from block (row block, k block)
  // at byte off; rounds i < CHA read A, the others B (so the descriptor of a
  // load is uniform).  A stage further along k is kF6KB k blocks further.
  const int sa = kF6KB * rows_a * kF6Block, sb = kF6KB * rows_b * kF6Block;
  int src[CH], kbl_of[CH];
  bool rowok[CH];
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    const bool isb = i >= CHA;
    const int c = tid + i * 256 - (isb ? CHA * 256 : 0);
    const int blk = c / kBlkCh;
    const int off = (c - blk * kBlkCh) * 16;
    const int R = isb ? RB : RA;
    const int kbl = blk / R, rbl = blk - kbl * R;
    const int rb = (isb ? nb0 : rb0) + rbl;
    rowok[i] = rb < (isb ? rows_b : rows_a);
    kbl_of[i] = kbl;
    src[i] = ((kb_beg + kbl) * (isb ? rows_b : rows_a) + rb) * kF6Block + off;
  }
  // Stage t goes straight from global memory into buffer t % 3 (16 bytes per
  // lane; a wave's 64 chunks of a round are 1 KB of consecutive LDS).  Every
  // thread issues exactly CH such loads per stage -- a stage past the end or
  // a block off the matrix reads zeros -- so "my loads of stage t+1 are in
  // LDS" is the static wait vmcnt(CH) once stage t+2 is issued.
  auto dma = [&](int t) {
    uint8_t* dst = lds + (t % kF6Bufs) * STAGE + wave * 64 * 16;
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const bool in = t < nst && rowok[i] && kb_beg + t * kF6KB + kbl_of[i] < kb_end;
      const int off = in ? src[i] + t * (i < CHA ? sa : sb) : kOutOfRange;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(i < CHA ? rsa : rsb,
                                               (__attribute__((address_space(3))) void*)(dst + i * 256 * 16), 16,
                                               off, 0, 0, 0);
    }
  };
  // s_waitcnt immediates (gfx9 encoding): vmcnt(CH) alone, lgkmcnt(0) alone
  constexpr int kWaitVmCH = (CH & 15) | (7 << 4) | (15 << 8) | ((CH >> 4) << 14);
  constexpr int kWaitLgkm0 = 15 | (7 << 4) | (0 << 8) | (3 << 14);
  // A workgroup barrier that orders memory operations in the compiler but,
  // unlike __syncthreads(), does not wait for the loads still in flight into
  // the next buffers; the waits it needs are explicit before it.
  auto barrier = [&]() { asm volatile("s_barrier" ::: "memory"); };

  v16f acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = v16f{};

  struct Frags {
    v8i a[TM], b[TN];
  };
  auto frag = [&](const uint8_t* blk) {
    const v4i p0 = *reinterpret_cast<const v4i*>(blk + 16 * lane);
    const v2i p1 = *reinterpret_cast<const v2i*>(blk + kF6Part1 + 8 * lane);
    return v8i{p0[0], p0[1], p0[2], p0[3], p1[0], p1[1], 0, 0};
  };
  auto read_frags = [&](int buf, int kk, Frags& f) {
    const uint8_t* As = lds + buf * STAGE + kk * RA * kF6Block;
    const uint8_t* Bs = lds + buf * STAGE + RA * kF6KB * kF6Block + kk * RB * kF6Block;
#pragma unroll
    for (int i = 0; i < TM; ++i) f.a[i] = frag(As + (wm * TM + i) * kF6Block);
#pragma unroll
    for (int j = 0; j < TN; ++j) f.b[j] = frag(Bs + (wn * TN + j) * kF6Block);
  };
  auto mfmas = [&](const Frags& f) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(f.b[j], f.a[i], acc[i][j], FB, FA, 0, kScaleOne,
                                                                    0, kScaleOne);
  };

  // Pipeline over a ring of three stage buffers, one barrier per stage.  In
  // step t: stage t+2 is issued into buffer (t+2)%3 (last read in step t-1,
  // which the previous barrier closed); stage t is multiplied from buffer
  // t%3; then each thread waits for its own loads of stage t+1 and the
  // barrier makes everyone's visible, after which stage t+1's first
  // fragments are read while stage t's last MFMAs still run.
  static_assert(kF6KB == 2, "the step below is written for two k-steps per stage");
  dma(0);
  dma(1);
  __builtin_amdgcn_s_waitcnt(kWaitVmCH);
  barrier();
  Frags f0, f1;
  read_frags(0, 0, f0);
  for (int t = 0; t < nst; ++t) {
    const int cb = t % kF6Bufs;
    dma(t + 2);
    read_frags(cb, 1, f1);
    mfmas(f0);
    mfmas(f1);
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    __builtin_amdgcn_s_waitcnt(kWaitVmCH);
    barrier();
    if (t + 1 < nst) read_frags((t + 1) % kF6Bufs, 0, f0);
  }
  // loads of stages past the end may still be writing zeros into the buffers
  // the epilogue reuses
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  // Epilogue through LDS, as gemm_luq_int4_kernel's: lane l of MFMA tile
  // (i, j) holds row l%32 and, in registers 4q..4q+3, columns
  // 8q + 4 (l/32) + 0..3.  The fp32 sums times kToCarrier are the INT8
  // carrier's integer sums (exact), scaled by the same fp32 factor.
  constexpr float kToCarrier = (AC == kAcLuq ? 32.0f : 64.0f) * (BSIGNED ? 16.0f : 8.0f) *
                               (AC == kAcInt4S ? 16.0f : (AC == kAcInt4U ? 8.0f : 1.0f));
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int EP = WN + 4;
  constexpr int LPR = WN / 4;
  constexpr int RPI = 64 / LPR;
  static_assert(4 * 32 * EP * 4 <= kF6Bufs * STAGE, "epilogue slabs fit in the stage buffers");
  uint32_t* E = reinterpret_cast<uint32_t*>(lds) + wave * 32 * EP;
  const bool part = a.partial != nullptr;
  const float sc = part ? 0.0f : epilogue_scale<AC, 1, BSIGNED>(*a.alpha, *a.bscale);
  uint32_t* out = part ? reinterpret_cast<uint32_t*>(a.partial + (int64_t)blockIdx.y * a.M * a.N)
                       : reinterpret_cast<uint32_t*>(a.C);
  const int64_t rbase = (int64_t)tm * BM + wm * WM, cbase = (int64_t)tn * BN + wn * WN;
  const int srow = lane / LPR, scol = (lane % LPR) * 4;
  const bool sact = lane < RPI * LPR;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v4u v;
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          const float x = acc[i][j][4 * q + rr] * kToCarrier;
          v[rr] = part ? (uint32_t)(int32_t)x : __float_as_uint(__fmul_rn(x, sc));
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
          for (int k = 0; k < 4; ++k)
            if (col + k < a.N) dst[k] = v[k];
        }
      }
    }
    __syncthreads();
  }
}

// ---- planning and launch ------------------------------------------------------

struct Fp6Plan {
  int bm;
  int64_t tiles_m, tiles_n;
  int nkb, kb_chunk, splits;
  size_t a_bytes, b_bytes, part_bytes;
};

static size_t round256(size_t b) { return (b + 255) & ~(size_t)255; }

static Fp6Plan plan_fp6(int64_t M, int64_t N, int64_t K) {
  Fp6Plan p;
  auto tiles = [&](int b) { return ((M + b - 1) / b) * ((N + b - 1) / b); };
  p.bm = (K >= 1024 && tiles(256) >= 256) ? 256 : 128;
  p.tiles_m = (M + p.bm - 1) / p.bm;
  p.tiles_n = (N + p.bm - 1) / p.bm;
  p.nkb = (int)((K + 63) / 64);
  const int64_t nt = p.tiles_m * p.tiles_n;
  const int64_t stages = (p.nkb + kF6KB - 1) / kF6KB;
  int64_t splits = 1;
  if (nt < 256) {  // too few tiles for 256 CUs: split the reduction (>= 8 stages each)
    splits = (512 + nt - 1) / nt;
    const int64_t by_len = stages / 8 > 0 ? stages / 8 : 1;
    if (splits > by_len) splits = by_len;
  }
  const int64_t exact = (K + kMaxExactKFp6 - 1) / kMaxExactKFp6;
  if (splits < exact) splits = exact;
  if (splits < 1) splits = 1;
  const int64_t chunk_stages = (stages + splits - 1) / splits;
  p.kb_chunk = (int)(chunk_stages * kF6KB);
  p.splits = (int)((p.nkb + p.kb_chunk - 1) / p.kb_chunk);
  p.a_bytes = (size_t)((M + 31) / 32) * p.nkb * kF6Block;
  p.b_bytes = (size_t)((N + 31) / 32) * p.nkb * kF6Block;
  p.part_bytes = p.splits > 1 ? (size_t)p.splits * M * N * sizeof(int32_t) : 0;
  return p;
}

size_t gemm_fp6_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  const Fp6Plan p = plan_fp6(M, N, K);
  return round256(p.a_bytes) + round256(p.b_bytes) + p.part_bytes;
}

bool gemm_fp6_fits(int64_t M, int64_t N, int64_t K) {
  const Fp6Plan p = plan_fp6(M, N, K);
  const size_t lim = ((size_t)1 << 31) - ((size_t)1 << 20);
  return p.a_bytes < lim && p.b_bytes < lim;
}

template <int KIND>
static void launch_pack(const uint8_t* src, int64_t rows, int64_t K, int nkb, uint8_t* dst, hipStream_t st) {
  const int64_t nrb = (rows + 31) / 32;
  const int64_t threads = nrb * nkb * 64;
  hipLaunchKernelGGL((fp6_pack_kernel<KIND>), dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st, src, rows,
                     K, (int64_t)nkb, nrb, dst);
}

template <int BM, int AC, bool BSIGNED>
static void launch_fp6_tile(const Fp6GemmArgs& a, dim3 grid, hipStream_t st) {
  constexpr int FA = AC == kAcLuq ? kFmtE3M2 : kFmtE2M3;
  hipLaunchKernelGGL((gemm_fp6_kernel<BM, BM, FA, kFmtE2M3, AC, BSIGNED>), grid, dim3(256), 0, st, a);
}

template <int AC, bool BSIGNED>
static void launch_fp6_t(const Fp6GemmArgs& a, const Fp6Plan& p, hipStream_t st) {
  const dim3 grid((unsigned)(p.tiles_m * p.tiles_n), (unsigned)p.splits);
  if (p.bm == 256)
    launch_fp6_tile<256, AC, BSIGNED>(a, grid, st);
  else
    launch_fp6_tile<128, AC, BSIGNED>(a, grid, st);
  if (p.splits > 1) {
    const int64_t MN = a.M * a.N;
    hipLaunchKernelGGL((splitk_reduce_kernel<AC, 1, BSIGNED>), dim3((unsigned)((MN + 63) / 64)), dim3(256), 0, st,
                       a.partial, p.splits, MN, a.alpha, a.bscale, a.C);
  }
}

hipError_t launch_gemm_luq_int4_fp6(const uint8_t* A, const float* alpha, const uint8_t* B, const float* bscale,
                                    int b_signed, int64_t M, int64_t N, int64_t K, float* C, void* ws,
                                    hipStream_t st) {
  const Fp6Plan p = plan_fp6(M, N, K);
  uint8_t* wa = static_cast<uint8_t*>(ws);
  uint8_t* wb = wa + round256(p.a_bytes);
  int32_t* wp = p.splits > 1 ? reinterpret_cast<int32_t*>(wb + round256(p.b_bytes)) : nullptr;
  launch_pack<kF6Luq>(A, M, K, p.nkb, wa, st);
  if (b_signed)
    launch_pack<kF6Int4S>(B, N, K, p.nkb, wb, st);
  else
    launch_pack<kF6Int4U>(B, N, K, p.nkb, wb, st);
  Fp6GemmArgs a;
  a.A = wa;
  a.B = wb;
  a.M = M;
  a.N = N;
  a.nkb = p.nkb;
  a.kb_chunk = p.kb_chunk;
  a.a_bytes = (int)p.a_bytes;
  a.b_bytes = (int)p.b_bytes;
  a.alpha = alpha;
  a.bscale = bscale;
  a.C = C;
  a.partial = wp;
  a.tiles_m = (int)p.tiles_m;
  a.tiles_n = (int)p.tiles_n;
  a.vec = (N % 4) == 0 && (((uintptr_t)(wp ? (void*)wp : (void*)C)) & 15) == 0;
  if (b_signed)
    launch_fp6_t<kAcLuq, true>(a, p, st);
  else
    launch_fp6_t<kAcLuq, false>(a, p, st);
  return hipGetLastError();
}

}  // namespace luq

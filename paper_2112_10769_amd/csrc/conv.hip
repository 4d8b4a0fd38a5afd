// Activation gradient of a 3x3 / stride 1 / zero-pad 1 convolution on 4-bit
// codes, as an implicit GEMM (Eq. backward applied to the lowered
// convolution, the lowering folded back onto pixels):
//
//   dact[t][c] = (alpha / ns) * s_W * sum_{kh, kw} sum_o
//                  (sum_s cg_s[t'][o]) * cW[(kh*3 + kw)*C + c][o]
//
// with t = (b*H + y)*W + x and t' the pixel (b, y + 1 - kh, x + 1 - kw),
// terms off the image left out.  cg are the LUQ codes of the output
// gradient g [T][Cout] (NHWC, row-major), cW the INT4 codes of the weight
// [Cout][3][3][C] in the transposed layout [9*C][Cout].  No lowered matrix
// is formed: the output is T x C floats, not T x 9C.
//
// Tile form (any shape; images of at most 64 pixels with Cout 32 or 64 and C a
// multiple of 32 take the row form further down): a tile is kBM consecutive
// pixels times 64 channels.  For each 64-deep chunk of Cout a workgroup
// expands into LDS:
//   - the gradient codes of the tile's pixels and of the W + 1 pixels on
//     either side (every tap of every pixel reads inside that halo, because a
//     tap shifts the flat pixel index by (1 - kh) * W + (1 - kw)),
//   - the 9 x 64 x 64 weight codes of the chunk (once per workgroup when
//     Cout <= 64: they then stay in LDS for all its tiles);
// then multiplies nine taps of two 32-deep k-steps.  A tap's A fragment is
// the halo shifted by the tap's pixel offset; a lane whose pixel's tap falls
// off the image reads a zero row instead.  Workgroups are persistent (about
// two per CU) and walk their tiles in order; the codes of the next (tile,
// chunk) are loaded into registers while the current one is multiplied, so
// the loads of one tile overlap the MFMAs and output stores of the previous.
// Expansion and MFMA carrier are those of the GEMMs (gemm_kernel.hpp): exact
// int32 sums, scales applied once.
#include "gemm_kernel.hpp"

namespace luq {

constexpr int kConvThreads = 256;
constexpr int kConvBM = 256;       // pixels per workgroup (4 waves x 64)
constexpr int kConvBN = 64;        // channels per workgroup
constexpr int kConvPitch = 80;     // LDS row pitch (64 int8 + 16 pad)

constexpr int kConvEP = 64 + 4;                               // epilogue slab pitch (words)
constexpr int kConvSlabs = 4 * 32 * kConvEP * 4;               // epilogue slabs (bytes)

template <int MAXW>
struct ConvLds {
  static constexpr int kHalo = kConvBM + 2 * (MAXW + 1);        // halo rows
  // A region: the halo, then (past the epilogue slabs, which reuse the
  // region) an all-zero row that stays zero
  static constexpr int kZeroRow =
      ((kHalo * kConvPitch > kConvSlabs ? kHalo * kConvPitch : kConvSlabs) + kConvPitch - 1) / kConvPitch;
  static constexpr int kABytes = (kZeroRow + 1) * kConvPitch;
  static constexpr int kBBytes = 9 * kConvBN * kConvPitch;
  static constexpr int kBytes = kABytes + kBBytes;
  static constexpr int kAPieces = (2 * kHalo + kConvThreads - 1) / kConvThreads;   // per thread
  static constexpr int kBPieces = (2 * 9 * kConvBN + kConvThreads - 1) / kConvThreads;
};

struct ConvArgs {
  const uint8_t* g;      // LUQ codes [T][Cout], ns planes
  int64_t g_plane;
  const uint8_t* w;      // INT4 codes [9*C][Cout]
  const float* alpha;
  const float* wscale;
  float* dact;           // [T][C]
  int T, H, W, C, Cout;
  int tiles_m;           // pixel tiles; each workgroup walks blockIdx.x + k * gridDim.x
  int vec;               // dact rows 16-byte aligned with C % 4 == 0
};

template <int MAXW, int NS, bool WSIGNED>
__global__ __launch_bounds__(kConvThreads, MAXW <= 64 ? 2 : 1) void conv3x3_dgrad_kernel(ConvArgs a) {
  using Lds = ConvLds<MAXW>;
  __shared__ __attribute__((aligned(16))) uint8_t lds[Lds::kBytes];
  static_assert(kConvSlabs <= Lds::kZeroRow * kConvPitch, "epilogue slabs stay below the zero row");
  uint8_t* As = lds;
  uint8_t* Bs = lds + Lds::kABytes;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c0 = blockIdx.y * kConvBN;
  const int hoff = a.W + 1;                       // halo rows before a tile
  const int hrows = kConvBM + 2 * hoff;
  const int rowb = a.Cout >> 1;                   // bytes per code row (both operands)
  const int nchunks = (a.Cout + 63) >> 6;
  const bool resident = nchunks == 1;             // weights expanded once

  __amdgpu_buffer_rsrc_t rsg[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s)
    rsg[s] = __builtin_amdgcn_make_buffer_rsrc((void*)(a.g + s * a.g_plane), (short)0, a.T * rowb, kBufferFlags);
  const __amdgpu_buffer_rsrc_t rsw =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.w, (short)0, 9 * a.C * rowb, kBufferFlags);

  // the zero row (read by taps off the image)
  if (tid < 4) reinterpret_cast<uint4*>(As + Lds::kZeroRow * kConvPitch)[tid] = make_uint4(0, 0, 0, 0);

  // Tile of the k-th item of this workgroup: tiles of consecutive pixels go
  // to one XCD (blocks are dealt round-robin over the 8 XCDs and the grid is
  // a multiple of 8 wide), so the halos two neighbours share hit one L2.
  auto tile_of = [&](int k) {
    int L = blockIdx.x + k * gridDim.x;
    if ((a.tiles_m & 7) == 0 && (gridDim.x & 7) == 0) L = (L & 7) * (a.tiles_m >> 3) + (L >> 3);
    return L;
  };
  const int nitems = ((a.tiles_m - (int)blockIdx.x + (int)gridDim.x - 1) / (int)gridDim.x) * nchunks;

  // ---- loads of item it (tile it / nchunks, Cout chunk it % nchunks) into
  // registers: halo pieces (row h, half hf: 32 codes of o) and weight pieces
  struct Regs {
    v4u ga[Lds::kAPieces][NS];
    v4u wb[Lds::kBPieces];
  };
  auto load = [&](Regs& r, int it) {
    const bool live = it < nitems;
    const int t0 = tile_of(live ? it / nchunks : 0) * kConvBM;
    const int cc = live ? it % nchunks : 0;
#pragma unroll
    for (int q = 0; q < Lds::kAPieces; ++q) {
      const int p = tid + q * kConvThreads;
      const int h = p >> 1, hf = p & 1;
      const int pix = t0 - hoff + h;
      const bool in = live && p < 2 * hrows && pix >= 0 && pix < a.T && cc * 64 + hf * 32 < a.Cout;
      const int off = in ? pix * rowb + cc * 32 + hf * 16 : kOutOfRange;
#pragma unroll
      for (int s = 0; s < NS; ++s) r.ga[q][s] = __builtin_amdgcn_raw_buffer_load_b128(rsg[s], off, 0, 0);
    }
    const bool wlive = live && (!resident || it == 0);
#pragma unroll
    for (int q = 0; q < Lds::kBPieces; ++q) {
      const int p = tid + q * kConvThreads;
      const int row = p >> 1, hf = p & 1;              // row = tap * 64 + c
      const int tap = row >> 6, c = row & 63;
      const bool in = wlive && p < 2 * 9 * kConvBN && c0 + c < a.C && cc * 64 + hf * 32 < a.Cout;
      const int off = in ? (tap * a.C + c0 + c) * rowb + cc * 32 + hf * 16 : kOutOfRange;
      r.wb[q] = __builtin_amdgcn_raw_buffer_load_b128(rsw, off, 0, 0);
    }
  };
  // ---- expand to int8 in LDS (even-k nibbles of a word in one word, odd-k
  // in the next; both operands alike)
  auto expand = [&](const Regs& r, bool weights) {
#pragma unroll
    for (int q = 0; q < Lds::kAPieces; ++q) {
      const int p = tid + q * kConvThreads;
      if (p >= 2 * hrows) continue;
      const int h = p >> 1, hf = p & 1;
      uint32_t w[8];
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        if constexpr (NS == 1) {
          expand_luq(r.ga[q][0][d], w[2 * d], w[2 * d + 1]);
        } else {
          uint32_t l0, h0, l1, h1;
          expand_luq_excess64(r.ga[q][0][d], l0, h0);
          expand_luq_excess64(r.ga[q][1][d], l1, h1);
          w[2 * d] = (l0 + l1) ^ 0x80808080u;
          w[2 * d + 1] = (h0 + h1) ^ 0x80808080u;
        }
      }
      uint4* dst = reinterpret_cast<uint4*>(As + h * kConvPitch + hf * 32);
      dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
      dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
    }
    if (!weights) return;
#pragma unroll
    for (int q = 0; q < Lds::kBPieces; ++q) {
      const int p = tid + q * kConvThreads;
      if (p >= 2 * 9 * kConvBN) continue;
      const int row = p >> 1, hf = p & 1;
      uint32_t w[8];
#pragma unroll
      for (int d = 0; d < 4; ++d) expand_int4<WSIGNED>(r.wb[q][d], w[2 * d], w[2 * d + 1]);
      uint4* dst = reinterpret_cast<uint4*>(Bs + row * kConvPitch + hf * 32);
      dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
      dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
    }
  };

  const float sc = epilogue_scale<kAcLuq, NS, WSIGNED>(*a.alpha, *a.wscale);
  const int zbase = Lds::kZeroRow * kConvPitch + (lane >> 5) * 16;
  v16i acc[2][2];
  int abase[2];
  uint32_t tapok[2];
  Regs r;
  load(r, 0);
  for (int it = 0; it < nitems; ++it) {
    const int cc = it % nchunks;
    const int t0 = tile_of(it / nchunks) * kConvBM;
    if (cc == 0) {
      // per lane: the LDS byte offsets of its two A-fragment rows (pixel rows
      // wave*64 + i*32 + lane%32 of the tile) and which of the nine taps of
      // each stay on the image
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int rr = wave * 64 + i * 32 + (lane & 31);
        const int t = t0 + rr;
        abase[i] = (rr + hoff) * kConvPitch + (lane >> 5) * 16;
        uint32_t ok = 0;
        if (t < a.T) {
          const int hw = a.H * a.W;
          const int rem = t % hw;
          const int y = rem / a.W, x = rem - (rem / a.W) * a.W;
#pragma unroll
          for (int kh = 0; kh < 3; ++kh)
#pragma unroll
            for (int kw = 0; kw < 3; ++kw) {
              const int ys = y + 1 - kh, xs = x + 1 - kw;
              if (ys >= 0 && ys < a.H && xs >= 0 && xs < a.W) ok |= 1u << (kh * 3 + kw);
            }
        }
        tapok[i] = ok;
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = v16i{};
    }
    expand(r, !resident || it == 0);
    load(r, it + 1);  // the next item's codes load while this one is multiplied
    __syncthreads();

    // ---- nine taps x two 32-deep k-steps
#pragma unroll
    for (int tap = 0; tap < 9; ++tap) {
      const int kh = tap / 3, kw = tap % 3;
      const int shift = ((1 - kh) * a.W + (1 - kw)) * kConvPitch;
      int aoff[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) aoff[i] = (tapok[i] >> tap) & 1 ? abase[i] + shift : zbase;
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        v4i fa[2], fb[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) fa[i] = *reinterpret_cast<const v4i*>(As + aoff[i] + kk * 32);
#pragma unroll
        for (int j = 0; j < 2; ++j)
          fb[j] = *reinterpret_cast<const v4i*>(Bs + (tap * 64 + j * 32 + (lane & 31)) * kConvPitch +
                                                (lane >> 5) * 16 + kk * 32);
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fb[j], fa[i], acc[i][j], 0, 0, 0);
      }
    }
    __syncthreads();  // every wave is done with the operands in LDS
    if (cc != nchunks - 1) continue;

    // ---- epilogue through LDS slabs in the A region (below the zero row):
    // lane l of MFMA tile (i, j) holds pixel row l%32 and, in registers
    // 4q..4q+3, channels 8q + 4*(l/32) + 0..3 of the 32.  Each wave stages
    // 32 rows x 64 channels, then stores 16-byte row segments (16 lanes per
    // row, 4 rows per instruction).
    uint32_t* E = reinterpret_cast<uint32_t*>(As) + wave * 32 * kConvEP;
    const int srow = lane >> 4, scol = (lane & 15) * 4;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          v4u v;
#pragma unroll
          for (int k = 0; k < 4; ++k) v[k] = __float_as_uint(__fmul_rn((float)acc[i][j][4 * q + k], sc));
          *reinterpret_cast<v4u*>(E + (lane & 31) * kConvEP + j * 32 + 8 * q + 4 * (lane >> 5)) = v;
        }
      // the slab is private to the wave: a wave barrier orders its writes
      // before its reads
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
#pragma unroll
      for (int rr = 0; rr < 32; rr += 4) {
        const int t = t0 + wave * 64 + i * 32 + rr + srow;
        const int c = c0 + scol;
        if (t < a.T && c < a.C) {
          const v4u v = *reinterpret_cast<const v4u*>(E + (rr + srow) * kConvEP + scol);
          float* dst = a.dact + (int64_t)t * a.C + c;
          if (a.vec) {
            // non-temporal: the output (T x C floats) is written once and
            // would only push the operands out of the caches (18.2 -> 17.3 us
            // on a 64x56x56x64 layer)
            __builtin_nontemporal_store(v, reinterpret_cast<v4u*>(dst));
          } else {
#pragma unroll
            for (int k = 0; k < 4; ++k)
              if (c + k < a.C) dst[k] = __uint_as_float(v[k]);
          }
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    }
    __syncthreads();  // the slabs are free before the next expansion
  }
}

template <int MAXW, int NS>
static void conv_launch_w(const ConvArgs& a, int wsigned, dim3 grid, hipStream_t st) {
  if (wsigned)
    hipLaunchKernelGGL((conv3x3_dgrad_kernel<MAXW, NS, true>), grid, dim3(kConvThreads), 0, st, a);
  else
    hipLaunchKernelGGL((conv3x3_dgrad_kernel<MAXW, NS, false>), grid, dim3(kConvThreads), 0, st, a);
}

// ---------------------------------------------------------------------------
// Activation gradient, row form (W <= 64, Cout 32 or 64, C a multiple of 32):
// output image row (b, y) reads the gradient rows y - 1, y, y + 1 of its own
// image and nothing else, so a workgroup walks a run of consecutive image
// rows and keeps the expanded gradient codes of four rows in an LDS ring: the
// three the current output row reads and the one being filled for the next.
// Every code is expanded once per workgroup (the tile form expands the W + 1
// pixels on either side of each tile again).  The weights of the workgroup's
// channels (9 taps x Cout) are expanded once into registers, so LDS holds only
// the ring (26 KB with its zero row) and up to four workgroups fit a CU.
//
// A wave owns 32 pixels of the row (one of its 32-pixel tiles) times 32
// channels.  Per output row it reads one A fragment from the ring per (tap,
// k-step) -- pixel x + 1 - kw of gradient row y + 1 - kh; a ring row carries a
// zero pixel on either side of the image, and a kernel row off the image
// reads an all-zero ring row -- and multiplies it with its weights.  The
// output row goes from the accumulators straight to memory with ordinary
// stores: each lane holds four consecutive channels of one pixel per register
// quad, and a wave's four stores fill the 128 bytes of its channels of each
// pixel.
// ---------------------------------------------------------------------------
constexpr int kDrThreads = 256;
constexpr int kDrPitch = 80;                   // ring bytes per pixel (64 codes + 16 pad)
constexpr int kDrSlot = 66 * kDrPitch;         // one ring row: pixels -1 .. 64
constexpr int kDrSlots = 4;                    // ring rows, then one all-zero row
constexpr int kDrAhead = 2;                    // gradient rows loaded ahead of their expansion

struct ConvDrArgs {
  const uint8_t* g;      // LUQ codes [T][Cout], ns planes
  int64_t g_plane;
  const uint8_t* w;      // INT4 codes [9*C][Cout]
  const float* alpha;
  const float* wscale;
  float* dact;           // [T][C], 16-byte aligned
  int rows, H, W, C;     // rows = B * H image rows
  int npt;               // 32-pixel tiles per row: 1 or 2
  int cblk;              // channels per workgroup, 32 * 4 / npt
  int rq, rrem;          // rows per range: rq, and rq + 1 for the first rrem ranges
};

template <int NS, bool WSIGNED, int NK, int LA>
__global__ __launch_bounds__(kDrThreads, 4) void conv3x3_dgrad_rows_kernel(ConvDrArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t ring[(kDrSlots + 1) * kDrSlot];
  constexpr int rowb = NK * 16;       // code bytes per pixel or weight row (Cout / 2)
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int pt = a.npt == 2 ? wave & 1 : 0;                 // pixel tile of the wave
  const int cw = blockIdx.y * a.cblk + 32 * (a.npt == 2 ? wave >> 1 : wave);   // its first channel
  const bool cact = cw < a.C;
  // consecutive row ranges share gradient rows: give each XCD (blocks are
  // dealt round-robin over the 8) a run of consecutive ranges
  int L = blockIdx.x;
  if ((gridDim.x & 7) == 0) L = (L & 7) * (gridDim.x >> 3) + (L >> 3);
  // range L: rq rows, one more for the first rrem ranges
  const int r0 = L * a.rq + min(L, a.rrem);
  const int r1 = r0 + a.rq + (L < a.rrem ? 1 : 0);

  __amdgpu_buffer_rsrc_t rsg[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s)
    rsg[s] = __builtin_amdgcn_make_buffer_rsrc((void*)(a.g + s * a.g_plane), (short)0, a.rows * a.W * rowb,
                                               kBufferFlags);
  const __amdgpu_buffer_rsrc_t rsw =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.w, (short)0, 9 * a.C * rowb, kBufferFlags);

  // ---- the wave's weights as B fragments: lane l holds channel cw + l % 32
  // and, for k-step kk, codes o = 32 kk + 16 (l / 32) .. + 15, expanded in the
  // k order of the ring's rows (even-k nibbles of a raw word, then odd-k).
  // Loaded here, expanded while the ring is cleared.
  v4i fb[9][NK];
  v2u32 wraw[9][NK];
  {
    const int c = cw + (lane & 31);
#pragma unroll
    for (int tap = 0; tap < 9; ++tap)
#pragma unroll
      for (int kk = 0; kk < NK; ++kk) {
        const int off = cact ? (tap * a.C + c) * rowb + kk * 16 + (lane >> 5) * 8 : kOutOfRange;
        wraw[tap][kk] = __builtin_amdgcn_raw_buffer_load_b64(rsw, off, 0, 0);
      }
  }

  // ---- ring: row R sits in slot (R + 1) % 4 (R >= -1), pixel x at x + 1;
  // pixel -1 and pixels W .. 64 of every slot, and all of slot 4, stay zero.
  // A gradient row is W * NK pieces of 16 bytes (32 codes): thread tid loads
  // and expands piece tid.  Every load and store of the row loop is issued
  // unconditionally (out-of-range offsets where there is nothing to move), so
  // that the compiler's waits for a row's codes count the stores issued after
  // them exactly and never wait for those stores.
  const int px = NK == 2 ? tid >> 1 : tid, hf = NK == 2 ? tid & 1 : 0;
  const bool pact = tid < a.W * NK;
  auto load_row = [&](int R, v4u (&v)[NS]) __attribute__((always_inline)) {
    const bool in = pact && R >= 0 && R < a.rows && R <= r1;
    const int off = in ? (R * a.W + px) * rowb + hf * 16 : kOutOfRange;
#pragma unroll
    for (int s = 0; s < NS; ++s) v[s] = __builtin_amdgcn_raw_buffer_load_b128(rsg[s], off, 0, 0);
  };
  auto put_row = [&](int R, const v4u (&v)[NS]) __attribute__((always_inline)) {
    if (!pact) return;
    uint32_t w[8];
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      if constexpr (NS == 1) {
        expand_luq(v[0][d], w[2 * d], w[2 * d + 1]);
      } else {
        uint32_t l0, h0, l1, h1;
        expand_luq_excess64(v[0][d], l0, h0);
        expand_luq_excess64(v[1][d], l1, h1);
        w[2 * d] = (l0 + l1) ^ 0x80808080u;
        w[2 * d + 1] = (h0 + h1) ^ 0x80808080u;
      }
    }
    uint4* dst = reinterpret_cast<uint4*>(ring + ((R + 1) & 3) * kDrSlot + (px + 1) * kDrPitch + hf * 32);
    dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
    dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
  };

  // rows R + 2 .. R + LA are loaded ahead, in register sets (row - r0) % LA
  v4u ahead[LA][NS];
  {
    v4u v0[NS], v1[NS], v2[NS];
    load_row(r0 - 1, v0);
    load_row(r0, v1);
    load_row(r0 + 1, v2);
#pragma unroll
    for (int k = 2; k <= LA; ++k) load_row(r0 + k, ahead[k % LA]);
    // clear the ring while the loads are in flight
    for (int i = tid; i < (kDrSlots + 1) * kDrSlot / 16; i += kDrThreads)
      reinterpret_cast<uint4*>(ring)[i] = make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int tap = 0; tap < 9; ++tap)
#pragma unroll
      for (int kk = 0; kk < NK; ++kk) {
        uint32_t w0, w1, w2, w3;
        expand_int4<WSIGNED>(wraw[tap][kk][0], w0, w1);
        expand_int4<WSIGNED>(wraw[tap][kk][1], w2, w3);
        fb[tap][kk] = v4i{(int)w0, (int)w1, (int)w2, (int)w3};
      }
    __syncthreads();
    put_row(r0 - 1, v0);
    put_row(r0, v1);
    put_row(r0 + 1, v2);
  }
  __syncthreads();

  const float sc = epilogue_scale<kAcLuq, NS, WSIGNED>(*a.alpha, *a.wscale);
  const int x = 32 * pt + (lane & 31);
  // the lane's A-fragment bytes at pixel x + 1 (kw = 0) of a ring row
  const int abase = (x + 2) * kDrPitch + (lane >> 5) * 16;
  // the lane's output bytes within an output row (four quads of channels)
  const int obase = (cact && x < a.W) ? (x * a.C + cw + 4 * (lane >> 5)) * 4 : kOutOfRange;
  const int orow = a.W * a.C;
  int y = r0 % a.H;
  // one output row; k = (R - r0) % LA selects the register sets
  auto row = [&](int R, v4u (&put)[NS], v4u (&issue)[NS]) __attribute__((always_inline)) {
    const bool live = R < r1;
    load_row(R + LA + 1, issue);       // read by output row R + LA
    v16i acc = v16i{};
    if (live && cact) {
#pragma unroll
      for (int kh = 0; kh < 3; ++kh) {
        // gradient row R + 1 - kh, or the zero row where it leaves the image
        const bool off = (kh == 0 && y == a.H - 1) || (kh == 2 && y == 0);
        const uint8_t* src = ring + (off ? kDrSlots : (R + 2 - kh) & 3) * kDrSlot + abase;
        v4i fa[3][NK];
#pragma unroll
        for (int kw = 0; kw < 3; ++kw)
#pragma unroll
          for (int kk = 0; kk < NK; ++kk)
            fa[kw][kk] = *reinterpret_cast<const v4i*>(src - kw * kDrPitch + kk * 32);
#pragma unroll
        for (int kw = 0; kw < 3; ++kw)
#pragma unroll
          for (int kk = 0; kk < NK; ++kk)
            acc = __builtin_amdgcn_mfma_i32_32x32x32_i8(fb[kh * 3 + kw][kk], fa[kw][kk], acc, 0, 0, 0);
      }
    }
    if (live && R + 2 <= r1) put_row(R + 2, put);   // read by output row R + 1
    // the output row: each lane four quads of four consecutive channels
    const __amdgpu_buffer_rsrc_t rso = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(a.dact + (int64_t)(live ? R : r0) * orow), (short)0, orow * 4, kBufferFlags);
    const int o = live ? obase : kOutOfRange;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      v4u v;
#pragma unroll
      for (int k = 0; k < 4; ++k) v[k] = __float_as_uint(__fmul_rn((float)acc[4 * q + k], sc));
      __builtin_amdgcn_raw_buffer_store_b128(v, rso, o + (o == kOutOfRange ? 0 : 32 * q), 0, 0);
    }
    y = y + 1 == a.H ? 0 : y + 1;
    __syncthreads();
  };
  auto trip = [&](int R) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < LA; ++k) row(R + k, ahead[(k + 2) % LA], ahead[(k + 1) % LA]);
  };
  // the first trip is peeled: the loop is then entered only from code that
  // ends with a row's stores, as its back edge does, so the waits inside it
  // are computed for the steady state
  trip(r0);
  for (int R = r0 + LA; R < r1; R += LA) trip(R);
}

static bool conv_dr_eligible(int64_t W, int64_t C, int64_t Cout, bool vec) {
  return W <= 64 && (Cout == 32 || Cout == 64) && C % 32 == 0 && vec;
}

template <int NS, int NK>
static void conv_dr_launch(const ConvDrArgs& d, int wsigned, dim3 grid, hipStream_t st) {
  if (wsigned) hipLaunchKernelGGL((conv3x3_dgrad_rows_kernel<NS, true, NK, kDrAhead>), grid, dim3(kDrThreads), 0, st, d);
  else hipLaunchKernelGGL((conv3x3_dgrad_rows_kernel<NS, false, NK, kDrAhead>), grid, dim3(kDrThreads), 0, st, d);
}

int conv3x3_max_width() { return 256; }

hipError_t launch_conv3x3_dgrad(const uint8_t* g, int64_t g_plane, int ns, const float* alpha, const uint8_t* w,
                                const float* wscale, int w_signed, int64_t B, int64_t H, int64_t W, int64_t C,
                                int64_t Cout, float* dact, hipStream_t st) {
  ConvArgs a;
  a.g = g;
  a.g_plane = g_plane;
  a.w = w;
  a.alpha = alpha;
  a.wscale = wscale;
  a.dact = dact;
  a.T = (int)(B * H * W);
  a.H = (int)H;
  a.W = (int)W;
  a.C = (int)C;
  a.Cout = (int)Cout;
  a.tiles_m = (a.T + kConvBM - 1) / kConvBM;
  a.vec = (C % 4) == 0 && (((uintptr_t)dact) & 15) == 0;
  if (conv_dr_eligible(W, C, Cout, a.vec != 0)) {
    ConvDrArgs d;
    d.g = g;
    d.g_plane = g_plane;
    d.w = w;
    d.alpha = alpha;
    d.wscale = wscale;
    d.dact = dact;
    d.rows = (int)(B * H);
    d.H = (int)H;
    d.W = (int)W;
    d.C = (int)C;
    d.npt = W > 32 ? 2 : 1;
    d.cblk = 32 * 4 / d.npt;
    // row ranges: k = 1..4 workgroups per CU (four fit), the k that puts the
    // fewest rows on the busiest CU (k workgroups of ceil(rows / ranges)
    // rows), the larger k on a tie; a multiple of 8 ranges.  The ResNet layer
    // (3584 rows) gets 512 ranges of 7 rows: 14.8 us against 16.3 with 1024
    // ranges of 3 or 4 rows
    const int cb = (int)((C + d.cblk - 1) / d.cblk);
    int nr = 1;
    int64_t best = -1;
    for (int k = 1; k <= 4; ++k) {
      int n = k * 256 / cb;
      n = n < 8 ? 8 : n & ~7;
      if (n > d.rows) n = d.rows;
      const int64_t per_cu = ((int64_t)n * cb + 255) / 256;
      const int64_t cost = per_cu * ((d.rows + n - 1) / n);
      if (best < 0 || cost <= best) {
        best = cost;
        nr = n;
      }
    }
    d.rq = d.rows / nr;
    d.rrem = d.rows - d.rq * nr;
    const dim3 grid((unsigned)nr, (unsigned)cb);
    if (ns == 1) {
      if (Cout == 64) conv_dr_launch<1, 2>(d, w_signed, grid, st);
      else conv_dr_launch<1, 1>(d, w_signed, grid, st);
    } else {
      if (Cout == 64) conv_dr_launch<2, 2>(d, w_signed, grid, st);
      else conv_dr_launch<2, 1>(d, w_signed, grid, st);
    }
    return hipGetLastError();
  }
  // persistent workgroups: about two per CU (one for wide images), a multiple
  // of 8 wide, each taking tiles blockIdx.x, blockIdx.x + gridDim.x, ...
  const int ctiles = (int)((C + kConvBN - 1) / kConvBN);
  int per = (W <= 64 ? 512 : 256) / ctiles;
  per = per < 8 ? 8 : per & ~7;
  const int gx = a.tiles_m < per ? a.tiles_m : per;
  const dim3 grid((unsigned)gx, (unsigned)ctiles);
  if (W <= 64) {
    if (ns == 1) conv_launch_w<64, 1>(a, w_signed, grid, st);
    else conv_launch_w<64, 2>(a, w_signed, grid, st);
  } else {
    if (ns == 1) conv_launch_w<256, 1>(a, w_signed, grid, st);
    else conv_launch_w<256, 2>(a, w_signed, grid, st);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Weight gradient of the same convolution, as an implicit GEMM (Eq. update
// applied to the lowered convolution, without forming the lowered matrix):
//
//   dW[o][(kh*3 + kw)*C + c] = (alpha / ns) * s_a * sum_t (sum_s cg_s[t][o]) * ca[t'][c]
//
// with t' = t + (kh - 1)*W + kw - 1 in the flat pixel index for t = (b, y, x),
// terms whose t' lies off the image left out.  Operands are the transposed
// code layouts (pixels innermost): g^T [Cout][T] and a^T [C][T].
//
// With u = t + kw - 1 a term reads cg[u - kw + 1] and ca[u + (kh - 1)*W]: the
// three taps of a kernel row share one activation operand.  The term is valid
// iff y(u) + kh - 1 lies on the image and, for kw = 0, x(u) != W - 1, for
// kw = 2, x(u) != 0 (the shift by one pixel then stays inside the row).  So a
// workgroup owns one kernel row kh and a 64 x 64 block of (o, c), and per
// stage of 128 pixels u expands into LDS:
//   - three copies of the gradient codes of its 64 output channels, copy kw
//     shifted by 1 - kw pixels and and-ed with the byte mask of the u valid
//     for (kh, kw) (mask tables built once per pixel range);
//   - the activation codes of its 64 input channels at the pixels
//     u + (kh - 1)*W: a window of 160 pixels from the 32-pixel boundary below.
// Each of four waves (two halves of o times two halves of c) builds one B
// fragment per 32-deep k-step from the window (dword reads, and v_alignbyte
// when the window's wave-uniform byte offset is not a multiple of 4) and
// multiplies it with the three copies.  Two groups of four waves take the two
// halves of the workgroup's pixel range, each with its own double-buffered
// stages; their sums are added through LDS at the end.  The reduction over
// pixel ranges is split over workgroups, and their int32 sums are combined
// exactly, in a fixed order, by conv_wgrad_reduce_kernel.
//
// Bytes in LDS are in natural pixel order (the shifts need it).  Carriers are
// those of the GEMMs: LUQ codes as their values (two samples as their int8
// sum), unsigned INT4 as 8q, signed INT4 as 16q.
// ---------------------------------------------------------------------------

constexpr int kWgKG = 2;                                   // wave groups (pixel halves)
constexpr int kWgGroup = 256;                              // threads per wave group
constexpr int kWgThreads = kWgKG * kWgGroup;
constexpr int kWgBK = 128;                                 // pixels per stage
constexpr int kWgGPitch = kWgBK + 16;                      // gradient copy row (bytes)
constexpr int kWgGCopy = 64 * kWgGPitch;
constexpr int kWgWin = kWgBK + 32;                         // activation window (pixels)
constexpr int kWgBPitch = kWgWin + 4;                      // an odd number of dwords
constexpr int kWgStage = 3 * kWgGCopy + 64 * kWgBPitch;
constexpr int kWgMaxLg = 1280;                             // pixels per wave group and range
// Pixels one workgroup sums in int32 (both wave groups together).  A term is
// at most 64 * 120 in magnitude: LUQ values up to 2^6 (R = 6, or the sum of
// two R = 5 samples) times INT4 carriers up to 8 * 15 or 16 * 7, and
// 2^18 * 7680 < 2^31.
constexpr int64_t kWgMaxWgPixels = (int64_t)1 << 18;
constexpr int kWgFar = 1 << 30;                            // a stage start past every image (T <= 2^29)
static_assert(kWgKG * 2 * kWgStage + 3 * kWgKG * kWgMaxLg <= 160 * 1024, "LDS");

struct ConvWgArgs {
  const uint8_t* g;      // LUQ codes [Cout][T], ns planes
  int64_t g_plane;
  const uint8_t* a;      // INT4 codes [C][T]
  const float* alpha;
  const float* ascale;
  float* dw;             // [Cout][9C]
  int32_t* partial;      // [nsplit][Cout][9C] sums of the splits, or null
  int T, H, W, C, Cout;
  int lg;                // pixels per wave group and range, a multiple of 2 * kWgBK
  int nranges;           // ranges of kWgKG * lg pixels covering [0, T)
  int nsplit;            // workgroups per (kh, tile); split s sums ranges s, s + nsplit, ...
  int nblk;              // blocks per tile: 24 * ceil(nsplit / 8)
  int ctiles;
  int vec;               // 16-byte stores of dW rows
};

// LUQ value bytes of four spread codes: 0 for field 0, else +-2^(field-1)
__device__ __forceinline__ uint32_t luq_value_bytes(uint32_t s) {
  const uint32_t m = __builtin_amdgcn_perm(0x40201008u, 0x04020100u, s & 0x07070707u);
  const uint32_t q = ((s >> 3) & 0x01010101u) | 0x0C0C0C0Cu;  // perm selector 12 / 13: 0x00 / 0xFF
  return (m ^ __builtin_amdgcn_perm(0u, 0u, q)) + (q & 0x01010101u);
}

// excess-64 LUQ value bytes (64 + v) of four spread codes; the sum of two
// samples' bytes, xor 0x80, is v0 + v1 in two's complement (R <= 5)
__device__ __forceinline__ uint32_t luq_ex64_bytes(uint32_t s) {
  const uint32_t p = __builtin_amdgcn_perm(0x80605048u, 0x44424140u, s & 0x07070707u);
  const uint32_t sg = (s >> 3) & 0x01010101u;
  return (p ^ ((sg << 7) - sg)) + sg;
}

template <int NS, bool ASIGNED>
__global__ __launch_bounds__(kWgThreads, 1) void conv3x3_wgrad_kernel(ConvWgArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[kWgKG * 2 * kWgStage];
  __shared__ __attribute__((aligned(16))) uint8_t vmask[3][kWgKG * kWgMaxLg];

  // blocks are dealt round-robin over the 8 XCDs: block 24q + 8kh + x takes
  // split 8q + x of row kh, so the three rows of a split share one XCD's L2
  // (the same gradient codes, overlapping activation windows)
  const int tile = blockIdx.x / a.nblk, bid = blockIdx.x - tile * a.nblk;
  const int kh = (bid >> 3) % 3;
  const int split = (bid / 24) * 8 + (bid & 7);
  if (split >= a.nsplit) return;
  const int ct = tile % a.ctiles, ot = tile / a.ctiles;
  const int o0 = ot * 64, c0 = ct * 64;

  const int tid = threadIdx.x, lane = tid & 63;
  const int kg = tid / kWgGroup, lt = tid % kWgGroup, wv = lt >> 6;
  const int oi = wv & 1, cj = wv >> 1;
  const int rowb = a.T >> 1;                       // bytes per code row of either operand
  const int shift = (kh - 1) * a.W;                // activation pixel of u: u + shift
  const int r = ((shift % 32) + 32) % 32;          // window byte of pixel k0 + shift
  const int nst = a.lg / kWgBK;
  uint8_t* mybuf = lds + kg * 2 * kWgStage;

  __amdgpu_buffer_rsrc_t rsg[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s)
    rsg[s] = __builtin_amdgcn_make_buffer_rsrc((void*)(a.g + s * a.g_plane), (short)0, a.Cout * rowb, kBufferFlags);
  const __amdgpu_buffer_rsrc_t rsa =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.a, (short)0, a.C * rowb, kBufferFlags);

  // load slots: lane lt handles row lt/4 and chunk j = lt%4 of both operands:
  // gradient pixels k0 + 32j .. +31 (and, for j = 0 / 3, the dword of the 8
  // pixels before / after the stage), window pixels 32j .. 32j + 31; the
  // 64 lanes of the group's first wave also take window chunk 4 of row lt.
  // Few, wide loads: the address unit, not HBM, limits this loop.
  const int lrow = lt >> 2, lj = lt & 3;
  const bool gok = o0 + lrow < a.Cout;
  const bool aok = c0 + lrow < a.C;
  struct Regs {
    v4u g[NS];
    uint32_t ge[NS];
    v4u b, b4;  // window chunk lj; chunk 4 (lanes of wave 0 of the group only)
  };
  // every step issues the same loads, without branches (a stage past the
  // range is loaded from k0 = kWgFar, beyond every image, which reads
  // nothing), so the compiler can wait for exactly the older stage's loads
  // and keep the newer ones in flight
  auto load = [&](Regs& R, int k0) {
    const int pg = k0 + 32 * lj;
    const int offg = gok && pg < a.T ? (o0 + lrow) * rowb + (pg >> 1) : kOutOfRange;
    const int pe = lj == 0 ? k0 - 8 : k0 + kWgBK;
    const bool eok = gok && (lj == 0 || lj == 3) && pe >= 0 && pe < a.T;
    const int offe = eok ? (o0 + lrow) * rowb + (pe >> 1) : kOutOfRange;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      R.g[s] = __builtin_amdgcn_raw_buffer_load_b128(rsg[s], offg, 0, 0);
      R.ge[s] = __builtin_amdgcn_raw_buffer_load_b32(rsg[s], offe, 0, 0);
    }
    // window chunks of 32 pixels (all on or all off [0, T)): chunk lj of row
    // lt/4 for every lane, chunk 4 of row lt for the 64 lanes of wave 0
    const int wbase = k0 + shift - r;
    const int pb = wbase + 32 * lj;
    R.b = __builtin_amdgcn_raw_buffer_load_b128(
        rsa, aok && pb >= 0 && pb < a.T ? (c0 + lrow) * rowb + (pb >> 1) : kOutOfRange, 0, 0);
    if (wv == 0) {
      const int p4 = wbase + 4 * 32;
      R.b4 = __builtin_amdgcn_raw_buffer_load_b128(
          rsa, c0 + lt < a.C && p4 >= 0 && p4 < a.T ? (c0 + lt) * rowb + (p4 >> 1) : kOutOfRange, 0, 0);
    }
  };
  // gradient chunk -> natural-order value bytes w, and the neighbouring pixel
  // outside the stage (before: nibble 7 of the dword, after: nibble 0) in e
  auto g_decode = [&](const Regs& R, uint32_t (&w)[8], uint32_t& e) {
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      uint32_t l0, h0;
      spread_nibbles(R.g[0][d], l0, h0);
      if constexpr (NS == 1) {
        w[2 * d] = luq_value_bytes(l0);
        w[2 * d + 1] = luq_value_bytes(h0);
      } else {
        uint32_t l1, h1;
        spread_nibbles(R.g[1][d], l1, h1);
        w[2 * d] = (luq_ex64_bytes(l0) + luq_ex64_bytes(l1)) ^ 0x80808080u;
        w[2 * d + 1] = (luq_ex64_bytes(h0) + luq_ex64_bytes(h1)) ^ 0x80808080u;
      }
    }
    const uint32_t n0 = lj == 0 ? R.ge[0] >> 28 : R.ge[0] & 0xFu;
    if constexpr (NS == 1) {
      e = luq_value_bytes(n0);
    } else {
      const uint32_t n1 = lj == 0 ? R.ge[1] >> 28 : R.ge[1] & 0xFu;
      e = (luq_ex64_bytes(n0) + luq_ex64_bytes(n1)) ^ 0x80808080u;  // zero above byte 0
    }
  };
  // the three shifted, masked copies of a decoded chunk; tpos = the chunk's
  // first pixel relative to the range (mask table index)
  auto g_store = [&](const uint32_t (&w)[8], uint32_t e, uint8_t* stage, int tpos) {
    // lanes 4*row + j hold the chunks j = 0..3 of a row: quad_perm (1,2,3,3)
    // gives each lane its right neighbour's w[0], (0,0,1,2) its left one's w[7]
    const uint32_t nx = (uint32_t)__builtin_amdgcn_mov_dpp((int)w[0], 0xF9, 0xF, 0xF, true);
    const uint32_t pv = (uint32_t)__builtin_amdgcn_mov_dpp((int)w[7], 0x90, 0xF, 0xF, true);
    const uint32_t next = lj == 3 ? e : nx;           // pixel 32j + 32 in byte 0
    const uint32_t prev = lj == 0 ? (e << 24) : pv;   // pixel 32j - 1 in byte 3
    uint32_t c0w[8], c2w[8];
#pragma unroll
    for (int d = 0; d < 8; ++d) {
      c0w[d] = __builtin_amdgcn_alignbyte(d < 7 ? w[d + 1] : next, w[d], 1u);  // u holds pixel u + 1
      c2w[d] = __builtin_amdgcn_alignbyte(w[d], d > 0 ? w[d - 1] : prev, 3u);  // u holds pixel u - 1
    }
    const uint4* m0 = reinterpret_cast<const uint4*>(&vmask[0][tpos]);
    const uint4* m1 = reinterpret_cast<const uint4*>(&vmask[1][tpos]);
    const uint4* m2 = reinterpret_cast<const uint4*>(&vmask[2][tpos]);
    uint8_t* base = stage + lrow * kWgGPitch + 32 * lj;
#pragma unroll
    for (int hlf = 0; hlf < 2; ++hlf) {
      const uint4 k0m = m0[hlf], k2m = m2[hlf];
      const uint4 k1m = kh == 1 ? make_uint4(0u, 0u, 0u, 0u) : m1[hlf];
      const int d = 4 * hlf;
      reinterpret_cast<uint4*>(base)[hlf] =
          make_uint4(c0w[d] & k0m.x, c0w[d + 1] & k0m.y, c0w[d + 2] & k0m.z, c0w[d + 3] & k0m.w);
      // copy 1 needs no mask for the middle row (pixels past T load as zero)
      reinterpret_cast<uint4*>(base + kWgGCopy)[hlf] =
          kh == 1 ? make_uint4(w[d], w[d + 1], w[d + 2], w[d + 3])
                  : make_uint4(w[d] & k1m.x, w[d + 1] & k1m.y, w[d + 2] & k1m.z, w[d + 3] & k1m.w);
      reinterpret_cast<uint4*>(base + 2 * kWgGCopy)[hlf] =
          make_uint4(c2w[d] & k2m.x, c2w[d + 1] & k2m.y, c2w[d + 2] & k2m.z, c2w[d + 3] & k2m.w);
    }
  };
  // the window piece: natural-order bytes 8q (unsigned) or 16q (signed)
  auto b_chunk = [&](const v4u& x4, uint32_t* dst) {
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      const uint32_t x = x4[d];
      if constexpr (ASIGNED) {
        const uint32_t z = x << 4;
        dst[2 * d] = __builtin_amdgcn_perm(x, z, 0x05010400u) & 0xF0F0F0F0u;
        dst[2 * d + 1] = __builtin_amdgcn_perm(x, z, 0x07030602u) & 0xF0F0F0F0u;
      } else {
        const uint32_t y = x >> 4;
        dst[2 * d] = (__builtin_amdgcn_perm(y, x, 0x05010400u) << 3) & 0x78787878u;
        dst[2 * d + 1] = (__builtin_amdgcn_perm(y, x, 0x07030602u) << 3) & 0x78787878u;
      }
    }
  };
  auto b_store = [&](const Regs& R, uint8_t* stage) {
    uint8_t* win = stage + 3 * kWgGCopy;
    b_chunk(R.b, reinterpret_cast<uint32_t*>(win + lrow * kWgBPitch + 32 * lj));
    if (wv == 0) b_chunk(R.b4, reinterpret_cast<uint32_t*>(win + lt * kWgBPitch + 4 * 32));
  };

  // mask tables of the range [rbase, rbase + kWgKG * lg): 0xFF where u is on
  // [0, T), y(u) + kh - 1 on the image and (copy 0) x(u) != W - 1, (copy 2)
  // x(u) != 0
  auto build_masks = [&](int rbase) {
    const int n4 = kWgKG * a.lg / 4;
    for (int i = tid; i < n4; i += kWgThreads) {
      const int u0 = rbase + 4 * i;  // T is a multiple of 4: u0 .. u0 + 3 all on or all off
      uint32_t m0 = 0, m1 = 0, m2 = 0;
      if (u0 < a.T) {
        const int row = u0 / a.W;
        int x = u0 - row * a.W;
        int y = row % a.H;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const bool yv = kh == 0 ? y != 0 : (kh == 2 ? y != a.H - 1 : true);
          if (yv) {
            m1 |= 0xFFu << (8 * k);
            if (x != a.W - 1) m0 |= 0xFFu << (8 * k);
            if (x != 0) m2 |= 0xFFu << (8 * k);
          }
          if (++x == a.W) {
            x = 0;
            if (++y == a.H) y = 0;
          }
        }
      }
      reinterpret_cast<uint32_t*>(vmask[0])[i] = m0;
      reinterpret_cast<uint32_t*>(vmask[1])[i] = m1;
      reinterpret_cast<uint32_t*>(vmask[2])[i] = m2;
    }
  };

  const int r32 = lane & 31, h = lane >> 5;
  const int aoff = (oi * 32 + r32) * kWgGPitch;
  const int boff = 3 * kWgGCopy + (cj * 32 + r32) * kWgBPitch;
  const uint32_t ra = (uint32_t)(r & 3);
  v16i acc[3];
#pragma unroll
  for (int kw = 0; kw < 3; ++kw) acc[kw] = v16i{};
  auto mfma_kstep = [&](const uint8_t* stage, int kk) {
    const int p = kk * 32 + 16 * h;
    const int s = r + p;
    const uint32_t* src = reinterpret_cast<const uint32_t*>(stage + boff + (s & ~3));
    v4i fb;
    if (ra == 0) {
#pragma unroll
      for (int d = 0; d < 4; ++d) fb[d] = (int)src[d];
    } else {
      uint32_t x[5];
#pragma unroll
      for (int d = 0; d < 5; ++d) x[d] = src[d];
#pragma unroll
      for (int d = 0; d < 4; ++d) fb[d] = (int)__builtin_amdgcn_alignbyte(x[d + 1], x[d], ra);
    }
#pragma unroll
    for (int kw = 0; kw < 3; ++kw) {
      const v4i fa = *reinterpret_cast<const v4i*>(stage + kw * kWgGCopy + aoff + p);
      acc[kw] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fb, fa, acc[kw], 0, 0, 0);
    }
  };

  for (int rg = split; rg < a.nranges; rg += a.nsplit) {
    const int rbase = rg * (kWgKG * a.lg);
    const int gbase = rbase + kg * a.lg;
    const int tbase = kg * a.lg;
    // one pipeline step: multiply stage t (buffer cb) while expanding stage
    // t+1 (registers R) into the other buffer; R is refilled with stage t+3
    // as soon as it is decoded.
    // The last step expands an empty stage into the idle buffer: no branch,
    // so the wait counts stay static.
    auto step = [&](int cb, int t, Regs& R) {
      uint8_t* cur = mybuf + cb * kWgStage;
      uint8_t* nxt = mybuf + (cb ^ 1) * kWgStage;
      const int tpos = (t + 1 < nst ? tbase + (t + 1) * kWgBK : 0) + 32 * lj;
      uint32_t w[8], e;
      mfma_kstep(cur, 0);
      g_decode(R, w, e);
      b_store(R, nxt);
      load(R, t + 3 < nst ? gbase + (t + 3) * kWgBK : kWgFar);  // R is free: refill it early
      mfma_kstep(cur, 1);
      g_store(w, e, nxt, tpos);
      mfma_kstep(cur, 2);
      mfma_kstep(cur, 3);
      __syncthreads();
    };
    Regs r0, r1;
    load(r0, gbase);
    load(r1, 1 < nst ? gbase + kWgBK : kWgFar);
    build_masks(rbase);  // while the first stages load
    __syncthreads();     // mask tables written
    {
      uint32_t w[8], e;
      g_decode(r0, w, e);
      g_store(w, e, mybuf, tbase + 32 * lj);
      b_store(r0, mybuf);
    }
    load(r0, 2 < nst ? gbase + 2 * kWgBK : kWgFar);
    __syncthreads();
    for (int t = 0; t < nst; t += 2) {  // nst is even
      step(0, t, r1);      // multiply t, expand t+1 (r1), reload r1 with t+3
      step(1, t + 1, r0);  // multiply t+1, expand t+2 (r0), reload r0 with t+4
    }
  }

  // Epilogue through LDS (the stage buffers are free after the last
  // barrier): each wave group stores its sums as rows [o][kw][c] of a slab of
  // its own; then every thread adds the groups' values of 4 consecutive c and
  // writes them, so each (o, kw) row of 64 channels leaves as 256
  // contiguous bytes.  Lane l holds output channel oi*32 + l%32 and input
  // channels cj*32 + 8q + 4*(l/32) + 0..3 of tap (kh, kw) in registers 4q..4q+3.
  constexpr int EP = 3 * 64 + 4;  // slab row pitch (int32): rows 4 banks apart
  static_assert(kWgKG * 64 * EP * 4 <= kWgKG * 2 * kWgStage, "epilogue slabs fit");
  int32_t* slab = reinterpret_cast<int32_t*>(lds);
  {
    int32_t* my = slab + kg * 64 * EP + (oi * 32 + r32) * EP + cj * 32 + 4 * h;
#pragma unroll
    for (int kw = 0; kw < 3; ++kw)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<v4i*>(my + kw * 64 + 8 * q) =
            v4i{acc[kw][4 * q], acc[kw][4 * q + 1], acc[kw][4 * q + 2], acc[kw][4 * q + 3]};
  }
  __syncthreads();
  const bool part = a.partial != nullptr;
  const float sc = part ? 0.0f : epilogue_scale<kAcLuq, NS, ASIGNED>(*a.alpha, *a.ascale);
  const int64_t ncol = 9LL * a.C;
  uint32_t* out = part ? reinterpret_cast<uint32_t*>(a.partial + (int64_t)split * a.Cout * ncol)
                       : reinterpret_cast<uint32_t*>(a.dw);
  // 192 rows (o, kw) of 16 four-channel pieces
  for (int i = tid; i < 64 * 3 * 16; i += kWgThreads) {
    const int row = i >> 4, j = i & 15;
    const int ol = row / 3, kw = row - 3 * (row / 3);
    const int o = o0 + ol, c = c0 + 4 * j;
    if (o >= a.Cout || c >= a.C) continue;
    v4i x = *reinterpret_cast<const v4i*>(slab + ol * EP + kw * 64 + 4 * j);
#pragma unroll
    for (int g = 1; g < kWgKG; ++g) x += *reinterpret_cast<const v4i*>(slab + g * 64 * EP + ol * EP + kw * 64 + 4 * j);
    v4u v;
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = part ? (uint32_t)x[k] : __float_as_uint(__fmul_rn((float)x[k], sc));
    uint32_t* dst = out + (int64_t)o * ncol + (kh * 3 + kw) * a.C + c;
    if (a.vec) {
      *reinterpret_cast<v4u*>(dst) = v;
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (c + k < a.C) dst[k] = v[k];
    }
  }
}

// dW = scale * (sum over splits of the int32 sums), summed exactly in int64
// in a fixed order.  A block owns 256 consecutive outputs; its 16 waves take
// the splits p = wave, wave + 16, ... with 16-byte loads (4 outputs a lane,
// several splits in flight), then the 16 partial sums are added through LDS.
constexpr int kRedThreads = 1024;

template <int NS, bool ASIGNED>
__global__ __launch_bounds__(kRedThreads) void conv_wgrad_reduce_kernel(const int32_t* __restrict__ partial,
                                                                       int splits, int64_t MN, int vec,
                                                                       const float* alpha, const float* ascale,
                                                                       float* __restrict__ out) {
  __shared__ int64_t red[kRedThreads / 64][256];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t i0 = (int64_t)blockIdx.x * 256 + 4 * lane;
  int64_t s[4] = {0, 0, 0, 0};
  if (vec && i0 + 3 < MN) {
    // up to 8 splits per wave in flight before the first add
    for (int p0 = wave; p0 < splits; p0 += 8 * 16) {
      v4i v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int p = p0 + 16 * u;
        v[u] = p < splits ? *reinterpret_cast<const v4i*>(partial + (int64_t)p * MN + i0) : v4i{0, 0, 0, 0};
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int k = 0; k < 4; ++k) s[k] += v[u][k];
    }
  } else {
    for (int p = wave; p < splits; p += 16)
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (i0 + k < MN) s[k] += partial[(int64_t)p * MN + i0 + k];
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) red[wave][4 * lane + k] = s[k];
  __syncthreads();
  if (threadIdx.x < 256) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    int64_t tot = 0;
#pragma unroll
    for (int w = 0; w < kRedThreads / 64; ++w) tot += red[w][threadIdx.x];
    if (i < MN) out[i] = __fmul_rn((float)tot, epilogue_scale<kAcLuq, NS, ASIGNED>(*alpha, *ascale));
  }
}

// ---------------------------------------------------------------------------
// Weight gradient, row form (W <= 64, C and Cout multiples of 32).  A
// workgroup owns one 32 x 32 (o, c) block of all nine taps over a range of
// image rows; each of its eight waves keeps the nine accumulator tiles of
// that block for its own run of rows, so an operand code is expanded once
// per wave that reads it (the activation rows at the ends of a run by two
// waves) and the expanded operands never pass through LDS.
//
// With r = b*H + y the flat image row and t = r*W + x, the tap (kh, kw) term
// of pixel t reads the activation at flat row r + kh - 1, column x + kw - 1.
// A row is multiplied as ceil(W / 32) k-steps of 32 columns (columns past W
// carry zero gradient codes).  The raw codes of a chunk of rows (the
// gradient rows, and the activation rows with one more on either side) are
// staged in LDS by 16-byte loads that write LDS directly, each channel's
// codes contiguous as in memory.  In one k-step a lane takes 16 gradient
// codes of channel o and, for each kernel row kh, the 16 activation codes of
// channel c at columns x + kw - 1, cut by funnel shifts from one 4-dword window of that
// activation row: an activation row is read and expanded once per wave and
// serves the three kernel rows of three consecutive gradient rows.  Column
// x + kw - 1 off the row (x = 0 with kw = 0, x = W - 1 with kw = 2) is
// cleared; a kernel row off the image (y + kh - 1 outside [0, H)) skips its
// three MFMAs.  Both operands use the GEMMs' expansions, which share one k
// permutation, so the products summed are the same.  The eight waves add
// their tiles through LDS; the workgroup writes the int32 sums of its block
// for its row range, and conv_wgrad_reduce_kernel adds the ranges in int64
// (with one range the scales are applied directly).
// ---------------------------------------------------------------------------
constexpr int kWrThreads = 512;
constexpr int kWrWaves = kWrThreads / 64;
constexpr int kWrLdsBytes = kWrWaves / 2 * 9 * 4 * 64 * 16;   // the tile sums; the staging reuses it
// pixels one workgroup sums in int32: 2^18 - 64 (a row of slack) times at
// most 64 * 120 per term stays below 2^31
constexpr int64_t kWrMaxPixels = ((int64_t)1 << 18) - 64;

// dwords staged per channel for n rows of width W: from the 16-byte block
// holding the first code (up to 31 codes before it), through the last k-step
// window (up to 64 + 16 codes past the rows' start of the last row), a
// multiple of 4; the LDS pitch adds one dword so that channels fall in
// different banks
__host__ __device__ constexpr int wr_seg_dwords(int n, int W) { return ((n * W + 31 + 80) / 8 + 4 + 3) / 4 * 4; }
// LDS pitch of a staged channel: at least seg dwords, 4 * (an odd number)
__host__ __device__ constexpr int wr_pitch(int seg) { return (seg / 4) % 2 ? seg : seg + 4; }
// s_waitcnt immediate (gfx9 encoding) of vmcnt(0) alone
constexpr int kWaitVm0 = (0 & 15) | (7 << 4) | (15 << 8) | (0 << 14);

struct ConvWrArgs {
  const uint8_t* g;      // LUQ codes [Cout][T], ns planes
  int64_t g_plane;
  const uint8_t* a;      // INT4 codes [C][T]
  const float* alpha;
  const float* ascale;
  float* dw;             // [Cout][9C]
  int32_t* partial;      // [nr][Cout][9C] int32 sums of the row ranges, or null (nr == 1)
  int T, H, W, C, Cout;
  int rows;              // B * H
  int nr;                // row ranges
  int ch;                // rows per staged chunk
  int oblk, cblk;        // 32-wide channel blocks
  int vec;               // 16-byte stores of dW rows
};

template <int NS, bool ASIGNED>
__global__ __launch_bounds__(kWrThreads, 1) void conv3x3_wgrad_rows_kernel(ConvWrArgs a) {
  __shared__ __attribute__((aligned(16))) uint32_t lds[kWrLdsBytes / 4];
  const int tid = threadIdx.x, lane = tid & 63;
  // the wave index in a scalar register: the row bounds, offsets and branches
  // derived from it are then wave-uniform scalar work
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r32 = lane & 31, h = lane >> 5;
  // blocks are dispatched round-robin over the XCDs: give each XCD runs of
  // consecutive (range, block) indices, whose blocks share operand rows
  const int total = a.nr * a.oblk * a.cblk;
  int L = blockIdx.x;
  if ((total & 7) == 0) L = (L & 7) * (total >> 3) + (L >> 3);
  const int cbk = L % a.cblk, obk = (L / a.cblk) % a.oblk, range = L / (a.cblk * a.oblk);
  const int rr0 = (int)((int64_t)range * a.rows / a.nr);
  const int rr1 = (int)((int64_t)(range + 1) * a.rows / a.nr);
  const int nk = (a.W + 31) >> 5;            // k-steps per row

  __amdgpu_buffer_rsrc_t rsg[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s)
    rsg[s] = __builtin_amdgcn_make_buffer_rsrc((void*)(a.g + s * a.g_plane), (short)0,
                                               (int)(((int64_t)a.Cout * a.T) >> 1), kBufferFlags);
  const __amdgpu_buffer_rsrc_t rsa =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.a, (short)0, (int)(((int64_t)a.C * a.T) >> 1), kBufferFlags);

  // gradient columns past W: per-lane masks of the 16 codes, per k-step
  uint32_t mg[2][2];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int v = a.W - 32 * k - 16 * h;    // valid codes of the lane's 16
    mg[k][0] = v >= 8 ? ~0u : (v <= 0 ? 0u : (1u << (4 * v)) - 1u);
    mg[k][1] = v >= 16 ? ~0u : (v <= 8 ? 0u : (1u << (4 * (v - 8))) - 1u);
  }
  // activation columns off the row: x = 0 with kw = 0 (k-step 0, lane half 0,
  // code 0) and x = W - 1 with kw = 2
  const uint32_t mleft = h == 0 ? ~0xFu : ~0u;
  const int xe = a.W - 1, ke = xe >> 5, he = (xe >> 4) & 1, je = xe & 15;
  const uint32_t mright0 = (h == he && je < 8) ? ~(0xFu << (4 * je)) : ~0u;
  const uint32_t mright1 = (h == he && je >= 8) ? ~(0xFu << (4 * (je - 8))) : ~0u;

  v16i acc[9];
#pragma unroll
  for (int t = 0; t < 9; ++t) acc[t] = v16i{};

  struct Raw {
    uint32_t g[NS][3];
    uint32_t x[4];
  };

  for (int cr0 = rr0; cr0 < rr1; cr0 += a.ch) {
    const int nrow = min(a.ch, rr1 - cr0);
    // ---- stage the raw codes of the chunk: per channel, dwords from the
    // 16-byte block holding the first code; T is a multiple of 32, so every
    // channel's block starts at the same offset of its row range.  Within an
    // operand (a gradient plane, the activations) channels lie back to back
    // at a pitch of 4 * (odd) dwords, so that the channels a k-step reads fall
    // at most two to a bank; each operand starts on a 1 KB boundary.  Each
    // wave instruction loads 64 consecutive 16-byte pieces of one operand
    // straight into LDS.
    const int pg = wr_pitch(wr_seg_dwords(nrow, a.W)), pa = wr_pitch(wr_seg_dwords(nrow + 2, a.W));
    const int qg = pg / 4, qa = pa / 4;                 // pieces per channel
    const int rg = (32 * qg + 63) / 64 * 64;            // pieces per gradient plane, whole wave loads
    const int ra = (32 * qa + 63) / 64 * 64;
    uint32_t* ldsg = lds;                               // plane p, channel k at 4 * (p * rg + k * qg)
    uint32_t* ldsa = lds + 4 * NS * rg;                 // channel k at k * pa
    const int64_t g0 = ((int64_t)cr0 * a.W) >> 5 << 2;             // dword of row cr0's first code, 16-B block
    const int64_t a0 = ((int64_t)(cr0 - 1) * a.W - 1) >> 5 << 2;   // column -1 of row cr0 - 1 (floor)
    __syncthreads();  // the previous chunk is consumed
    {
      const int ntot = NS * rg + ra;
      for (int c0 = wave * 64; c0 < ntot; c0 += kWrThreads) {
        uint32_t* dst = lds + 4 * c0;
        if (c0 < NS * rg) {
          const int pl = c0 >= rg ? 1 : 0;              // gradient plane (uniform)
          const int u = c0 - pl * rg + lane;
          const int k = u / qg, j = u - k * qg;
          const int off = u < 32 * qg ? (int)((((int64_t)(obk * 32 + k) * (a.T >> 3)) + g0 + 4 * j) << 2)
                                      : kOutOfRange;
          // (a descriptor taken from the array inside the call drops the
          // kernel's host stub: copy it first)
          const __amdgpu_buffer_rsrc_t rsp = rsg[NS == 2 ? pl : 0];
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rsp, (__attribute__((address_space(3))) void*)dst, 16, off, 0, 0, 0);
        } else {
          const int u = c0 - NS * rg + lane;
          const int k = u / qa, j = u - k * qa;
          const int64_t dwi = (int64_t)(cbk * 32 + k) * (a.T >> 3) + a0 + 4 * j;
          const int off = (u < 32 * qa && dwi >= 0) ? (int)(dwi << 2) : kOutOfRange;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rsa, (__attribute__((address_space(3))) void*)dst, 16, off, 0, 0, 0);
        }
      }
      // the loads into LDS are done before the barrier
      __builtin_amdgcn_s_waitcnt(kWaitVm0);
    }
    __syncthreads();

    // ---- this wave's rows of the chunk, one pass per k-step: step i reads
    // activation row r0 - 1 + i and, for i >= 2, multiplies gradient row
    // r0 - 2 + i
    const int r0 = cr0 + (wave * nrow) / kWrWaves, r1 = cr0 + ((wave + 1) * nrow) / kWrWaves;
    const int n = r1 - r0, per = n + 2;
    const uint32_t* lg = ldsg + r32 * pg + 2 * h;
    const uint32_t* la = ldsa + r32 * pa + 2 * h;
    const int gplane = 4 * rg;                          // dwords between gradient planes
    const int ga = (int)a0, gg = (int)g0;
    for (int kst = 0; kst < (n > 0 ? nk : 0); ++kst) {
      // code offsets (within a channel) of the window start and of the
      // gradient chunk at step 0; they advance by W per step
      const int xa0 = (r0 - 1) * a.W + 32 * kst - 1;
      const int xg0 = (r0 - 2) * a.W + 32 * kst;
      int yy = r0 % a.H;  // image row of the next gradient row
      auto load = [&](Raw& R, int i) {
        if (i >= per) return;
        const int wa = ((xa0 + i * a.W) >> 3) - ga;   // window's first dword in its channel
#pragma unroll
        for (int j = 0; j < 4; ++j) R.x[j] = la[wa + j];
        if (i >= 2) {
          const int wg = ((xg0 + i * a.W) >> 3) - gg;
#pragma unroll
          for (int p = 0; p < NS; ++p)
#pragma unroll
            for (int j = 0; j < 3; ++j) R.g[p][j] = lg[p * gplane + wg + j];
        }
      };
      // the three shifted activation fragments of a window
      auto expand_x = [&](const Raw& R, v4i (&w)[3], int i) {
        const int ob = (xa0 + i * a.W) & 7;
#pragma unroll
        for (int kw = 0; kw < 3; ++kw) {
          const int sh = ob + kw;
          uint32_t x0, x1;
          if (sh < 8) {
            x0 = __builtin_amdgcn_alignbit(R.x[1], R.x[0], 4 * sh);
            x1 = __builtin_amdgcn_alignbit(R.x[2], R.x[1], 4 * sh);
          } else {
            x0 = __builtin_amdgcn_alignbit(R.x[2], R.x[1], 4 * (sh - 8));
            x1 = __builtin_amdgcn_alignbit(R.x[3], R.x[2], 4 * (sh - 8));
          }
          if (kw == 0 && kst == 0) x0 &= mleft;
          if (kw == 2 && kst == ke) {
            x0 &= mright0;
            x1 &= mright1;
          }
          uint32_t l0, h0, l1, h1;
          expand_int4<ASIGNED>(x0, l0, h0);
          expand_int4<ASIGNED>(x1, l1, h1);
          w[kw] = v4i{(int)l0, (int)h0, (int)l1, (int)h1};
        }
      };
      auto expand_g = [&](const Raw& R, int i) {
        const int sg = 4 * ((xg0 + i * a.W) & 7);
        const uint32_t m0 = kst ? mg[1][0] : mg[0][0], m1 = kst ? mg[1][1] : mg[0][1];
        uint32_t w[4];
        if constexpr (NS == 1) {
          const uint32_t x0 = __builtin_amdgcn_alignbit(R.g[0][1], R.g[0][0], sg) & m0;
          const uint32_t x1 = __builtin_amdgcn_alignbit(R.g[0][2], R.g[0][1], sg) & m1;
          expand_luq(x0, w[0], w[1]);
          expand_luq(x1, w[2], w[3]);
        } else {
#pragma unroll
          for (int d = 0; d < 2; ++d) {
            const uint32_t m = d ? m1 : m0;
            const uint32_t p0 = __builtin_amdgcn_alignbit(R.g[0][d + 1], R.g[0][d], sg) & m;
            const uint32_t p1 = __builtin_amdgcn_alignbit(R.g[1][d + 1], R.g[1][d], sg) & m;
            uint32_t l0, h0, l1, h1;
            expand_luq_excess64(p0, l0, h0);
            expand_luq_excess64(p1, l1, h1);
            w[2 * d] = (l0 + l1) ^ 0x80808080u;
            w[2 * d + 1] = (h0 + h1) ^ 0x80808080u;
          }
        }
        return v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
      };
      // step i: expand the activation window into wj; for a gradient row
      // (i >= 2) multiply it with the windows of rows r - 1 (w0), r (w1) and
      // r + 1 (wj)
      auto step = [&](int i, v4i (&wj)[3], const v4i (&w0)[3], const v4i (&w1)[3]) {
        if (i >= per) return;
        Raw R;
        load(R, i);
        expand_x(R, wj, i);
        v4i fa = v4i{};
        if (i >= 2) fa = expand_g(R, i);
        if (i >= 2) {
          const int y = yy;
          yy = y + 1 == a.H ? 0 : y + 1;
          if (y > 0) {
#pragma unroll
            for (int kw = 0; kw < 3; ++kw)
              acc[kw] = __builtin_amdgcn_mfma_i32_32x32x32_i8(w0[kw], fa, acc[kw], 0, 0, 0);
          }
#pragma unroll
          for (int kw = 0; kw < 3; ++kw)
            acc[3 + kw] = __builtin_amdgcn_mfma_i32_32x32x32_i8(w1[kw], fa, acc[3 + kw], 0, 0, 0);
          if (y < a.H - 1) {
#pragma unroll
            for (int kw = 0; kw < 3; ++kw)
              acc[6 + kw] = __builtin_amdgcn_mfma_i32_32x32x32_i8(wj[kw], fa, acc[6 + kw], 0, 0, 0);
          }
        }
      };

      v4i win[3][3];
      for (int i = 0; i < per; i += 3) {
        step(i, win[0], win[1], win[2]);
        step(i + 1, win[1], win[2], win[0]);
        step(i + 2, win[2], win[0], win[1]);
      }
    }
  }

  // add the eight waves' tiles through LDS in two rounds, each over half of
  // the 36 (tap, quad) pairs (eight waves' halves fill the LDS): every wave
  // writes its half, then every thread adds the eight values of its share of
  // the round's outputs and stores them
  v4i* red = reinterpret_cast<v4i*>(lds);   // [8][18][64]
  constexpr int kHalfV4 = 18 * 64;          // one wave's half in 16-byte entries
  const bool part = a.partial != nullptr;
  const float sc = part ? 0.0f : epilogue_scale<kAcLuq, NS, ASIGNED>(*a.alpha, *a.ascale);
  const int64_t ncol = 9LL * a.C;
  uint32_t* out = part ? reinterpret_cast<uint32_t*>(a.partial + (int64_t)range * a.Cout * ncol)
                       : reinterpret_cast<uint32_t*>(a.dw);
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    __syncthreads();  // the staging is consumed, or the previous round read
#pragma unroll
    for (int u = 0; u < 18; ++u) {
      const int tq = 18 * r + u, t = tq >> 2, q = tq & 3;
      red[(wave * 18 + u) * 64 + lane] = v4i{acc[t][4 * q], acc[t][4 * q + 1], acc[t][4 * q + 2], acc[t][4 * q + 3]};
    }
    __syncthreads();
    // entry e = u * 64 + l: (tap, quad) pair 18r + u; output channel
    // o = l % 32, input channels c0 + 8q + 4(l / 32) .. +3 of the tap
    for (int e = tid; e < kHalfV4; e += kWrThreads) {
      v4i s4 = red[e];
#pragma unroll
      for (int w = 1; w < kWrWaves; ++w) s4 += red[w * kHalfV4 + e];
      const int tq = 18 * r + (e >> 6), t = tq >> 2, q = tq & 3, l = e & 63;
      const int o = obk * 32 + (l & 31);
      v4u v;
#pragma unroll
      for (int k = 0; k < 4; ++k) v[k] = part ? (uint32_t)s4[k] : __float_as_uint(__fmul_rn((float)s4[k], sc));
      uint32_t* dst = out + (int64_t)o * ncol + t * a.C + cbk * 32 + 8 * q + 4 * (l >> 5);
      if (a.vec) {
        *reinterpret_cast<v4u*>(dst) = v;
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) dst[k] = v[k];
      }
    }
  }
}

// rows per staged chunk: the gradient planes and the activation rows of a
// chunk fit the kernel's LDS
static int conv_wr_chunk_rows(int64_t W, int ns) {
  // the staged pieces: each operand rounded up to whole wave loads of 64
  auto bytes = [&](int n) {
    const int rg = (32 * (wr_pitch(wr_seg_dwords(n, (int)W)) / 4) + 63) / 64 * 64;
    const int ra = (32 * (wr_pitch(wr_seg_dwords(n + 2, (int)W)) / 4) + 63) / 64 * 64;
    return 16 * (ns * rg + ra);
  };
  int ch = 1;
  while (bytes(ch + 1) <= kWrLdsBytes) ++ch;
  return ch;
}

// row ranges of the row form: about one workgroup per CU, and at most
// kWrMaxPixels pixels per range (rows <= 0: an upper bound for any row count)
static int64_t conv_wr_ranges(int64_t T, int64_t C, int64_t Cout, int64_t rows) {
  const int64_t blocks = (C / 32) * (Cout / 32);
  int64_t nr = 256 / blocks;
  if (nr < 1) nr = 1;
  const int64_t need = (T + kWrMaxPixels - 1) / kWrMaxPixels;
  if (nr < need) nr = need;
  if (rows > 0 && nr > rows) nr = rows;  // rows >= T / 64 >= need
  return nr;
}

static bool conv_wr_eligible(int64_t W, int64_t C, int64_t Cout) {
  return W >= 1 && W <= 64 && C % 32 == 0 && Cout % 32 == 0;
}

struct ConvWgPlan {
  int lg, nranges, nsplit;
};

static ConvWgPlan plan_conv_wgrad(int64_t T, int64_t C, int64_t Cout) {
  const int64_t tiles = ((Cout + 63) / 64) * ((C + 63) / 64);
  // about one workgroup per CU: 3 kernel rows x tiles x nsplit ~ 256
  int64_t want = 256 / (3 * tiles);
  if (want < 1) want = 1;
  int64_t lg = (T + want * kWgKG - 1) / (want * kWgKG);
  lg = (lg + 2 * kWgBK - 1) / (2 * kWgBK) * (2 * kWgBK);  // an even number of stages
  if (lg > kWgMaxLg) lg = kWgMaxLg;
  const int64_t nranges = (T + kWgKG * lg - 1) / (kWgKG * lg);
  // each workgroup sums at most kWgMaxWgPixels pixels, so its int32 sums
  // cannot overflow (|term| <= 64 * 120)
  const int64_t per = kWgMaxWgPixels / (kWgKG * lg);
  int64_t nsplit = want;
  if (nsplit < (nranges + per - 1) / per) nsplit = (nranges + per - 1) / per;
  if (nsplit > nranges) nsplit = nranges;
  ConvWgPlan p;
  p.lg = (int)lg;
  p.nranges = (int)nranges;
  p.nsplit = (int)nsplit;
  return p;
}

size_t conv3x3_wgrad_workspace_bytes(int64_t T, int64_t C, int64_t Cout) {
  const ConvWgPlan p = plan_conv_wgrad(T, C, Cout);
  int64_t parts = p.nsplit > 1 ? p.nsplit : 0;
  // the row form (taken for W <= 64, which the workspace query does not see)
  if (conv_wr_eligible(1, C, Cout)) {
    const int64_t nr = conv_wr_ranges(T, C, Cout, 0);
    if (nr > 1 && nr > parts) parts = nr;
  }
  return (size_t)parts * (size_t)Cout * (size_t)(9 * C) * sizeof(int32_t);
}

int64_t conv3x3_wgrad_blocks(int64_t T, int64_t C, int64_t Cout) {
  const ConvWgPlan p = plan_conv_wgrad(T, C, Cout);
  return ((Cout + 63) / 64) * ((C + 63) / 64) * 24 * ((p.nsplit + 7) / 8);
}

template <int NS, bool ASIGNED>
static void conv_wgrad_launch_t(const ConvWgArgs& a, unsigned blocks, hipStream_t st) {
  hipLaunchKernelGGL((conv3x3_wgrad_kernel<NS, ASIGNED>), dim3(blocks), dim3(kWgThreads), 0, st, a);
  if (a.partial) {
    const int64_t MN = (int64_t)a.Cout * 9 * a.C;
    const int vec = (MN % 4) == 0;
    hipLaunchKernelGGL((conv_wgrad_reduce_kernel<NS, ASIGNED>), dim3((unsigned)((MN + 255) / 256)),
                       dim3(kRedThreads), 0, st, a.partial, a.nsplit, MN, vec, a.alpha, a.ascale, a.dw);
  }
}

template <int NS, bool ASIGNED>
static void conv_wr_launch_t(const ConvWrArgs& a, unsigned blocks, hipStream_t st) {
  hipLaunchKernelGGL((conv3x3_wgrad_rows_kernel<NS, ASIGNED>), dim3(blocks), dim3(kWrThreads), 0, st, a);
  if (a.partial) {
    const int64_t MN = (int64_t)a.Cout * 9 * a.C;
    hipLaunchKernelGGL((conv_wgrad_reduce_kernel<NS, ASIGNED>), dim3((unsigned)((MN + 255) / 256)),
                       dim3(kRedThreads), 0, st, a.partial, a.nr, MN, 1, a.alpha, a.ascale, a.dw);
  }
}

hipError_t launch_conv3x3_wgrad(const uint8_t* g, int64_t g_plane, int ns, const float* alpha, const uint8_t* act,
                                const float* ascale, int a_signed, int64_t B, int64_t H, int64_t W, int64_t C,
                                int64_t Cout, float* dw, void* ws, hipStream_t st) {
  const int64_t T = B * H * W;
  const ConvWgPlan p = plan_conv_wgrad(T, C, Cout);
  ConvWgArgs a;
  a.g = g;
  a.g_plane = g_plane;
  a.a = act;
  a.alpha = alpha;
  a.ascale = ascale;
  a.dw = dw;
  a.partial = p.nsplit > 1 ? static_cast<int32_t*>(ws) : nullptr;
  a.T = (int)T;
  a.H = (int)H;
  a.W = (int)W;
  a.C = (int)C;
  a.Cout = (int)Cout;
  a.lg = p.lg;
  a.nranges = p.nranges;
  a.nsplit = p.nsplit;
  a.nblk = 24 * ((p.nsplit + 7) / 8);
  a.ctiles = (int)((C + 63) / 64);
  a.vec = (C % 4) == 0 && (((uintptr_t)(a.partial ? (void*)a.partial : (void*)dw)) & 15) == 0;
  if (conv_wr_eligible(W, C, Cout)) {
    ConvWrArgs r;
    r.g = g;
    r.g_plane = g_plane;
    r.a = act;
    r.alpha = alpha;
    r.ascale = ascale;
    r.dw = dw;
    r.T = (int)T;
    r.H = (int)H;
    r.W = (int)W;
    r.C = (int)C;
    r.Cout = (int)Cout;
    r.rows = (int)(B * H);
    r.nr = (int)conv_wr_ranges(T, C, Cout, B * H);
    r.ch = conv_wr_chunk_rows(W, ns);
    r.oblk = (int)(Cout / 32);
    r.cblk = (int)(C / 32);
    r.partial = r.nr > 1 ? static_cast<int32_t*>(ws) : nullptr;
    r.vec = (((uintptr_t)(r.partial ? (void*)r.partial : (void*)dw)) & 15) == 0;
    const unsigned blocks = (unsigned)((int64_t)r.nr * r.oblk * r.cblk);
    if (ns == 1)
      a_signed ? conv_wr_launch_t<1, true>(r, blocks, st) : conv_wr_launch_t<1, false>(r, blocks, st);
    else
      a_signed ? conv_wr_launch_t<2, true>(r, blocks, st) : conv_wr_launch_t<2, false>(r, blocks, st);
    return hipGetLastError();
  }
  const unsigned blocks = (unsigned)conv3x3_wgrad_blocks(T, C, Cout);
  if (ns == 1)
    a_signed ? conv_wgrad_launch_t<1, true>(a, blocks, st) : conv_wgrad_launch_t<1, false>(a, blocks, st);
  else
    a_signed ? conv_wgrad_launch_t<2, true>(a, blocks, st) : conv_wgrad_launch_t<2, false>(a, blocks, st);
  return hipGetLastError();
}

}  // namespace luq

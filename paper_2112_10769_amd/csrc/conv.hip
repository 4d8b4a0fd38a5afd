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
// A workgroup owns kBM consecutive pixels and 64 channels.  For each 64-deep
// chunk of Cout it expands, once, into LDS:
//   - the gradient codes of its pixels and of the W + 1 pixels on either
//     side (every tap of every pixel reads inside that halo, because a tap
//     shifts the flat pixel index by (1 - kh) * W + (1 - kw)),
//   - the 9 x 64 x 64 weight codes of the chunk;
// then multiplies nine taps of two 32-deep k-steps.  A tap's A fragment is
// the halo shifted by the tap's pixel offset; a lane whose pixel's tap falls
// off the image reads a zero row instead.  Expansion and MFMA carrier are
// those of the GEMMs (gemm_kernel.hpp): exact int32 sums, scales applied once.
#include "gemm_kernel.hpp"

namespace luq {

constexpr int kConvThreads = 256;
constexpr int kConvBM = 256;       // pixels per workgroup (4 waves x 64)
constexpr int kConvBN = 64;        // channels per workgroup
constexpr int kConvPitch = 80;     // LDS row pitch (64 int8 + 16 pad)

template <int MAXW>
struct ConvLds {
  static constexpr int kHalo = kConvBM + 2 * (MAXW + 1);        // halo rows
  static constexpr int kZeroRow = kHalo;                         // an all-zero row
  static constexpr int kABytes = (kHalo + 1) * kConvPitch;
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
  int tiles_m;
  int vec;               // dact rows 16-byte aligned with C % 4 == 0
};

template <int MAXW, int NS, bool WSIGNED>
__global__ __launch_bounds__(kConvThreads, MAXW <= 64 ? 2 : 1) void conv3x3_dgrad_kernel(ConvArgs a) {
  using Lds = ConvLds<MAXW>;
  __shared__ __attribute__((aligned(16))) uint8_t lds[Lds::kBytes];
  uint8_t* As = lds;
  uint8_t* Bs = lds + Lds::kABytes;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // tiles of consecutive pixels go to one XCD (blocks are dealt round-robin
  // over the 8 XCDs), so the halos two neighbours share hit the same L2
  int L = blockIdx.x;
  if ((a.tiles_m & 7) == 0) L = (L & 7) * (a.tiles_m >> 3) + (L >> 3);
  const int t0 = L * kConvBM;
  const int c0 = blockIdx.y * kConvBN;
  const int hoff = a.W + 1;                       // halo rows before t0
  const int hrows = kConvBM + 2 * hoff;
  const int rowb = a.Cout >> 1;                   // bytes per code row (both operands)

  __amdgpu_buffer_rsrc_t rsg[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s)
    rsg[s] = __builtin_amdgcn_make_buffer_rsrc((void*)(a.g + s * a.g_plane), (short)0, a.T * rowb, kBufferFlags);
  const __amdgpu_buffer_rsrc_t rsw =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.w, (short)0, 9 * a.C * rowb, kBufferFlags);

  // the zero row (read by taps off the image)
  if (tid < 4) reinterpret_cast<uint4*>(As + Lds::kZeroRow * kConvPitch)[tid] = make_uint4(0, 0, 0, 0);

  // Per lane: the LDS byte offsets of its two A-fragment rows (pixel rows
  // wave*64 + i*32 + lane%32 of the tile) and which of the nine taps of each
  // stay on the image.
  int abase[2];
  uint32_t tapok[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = wave * 64 + i * 32 + (lane & 31);
    const int t = t0 + r;
    abase[i] = (r + hoff) * kConvPitch + (lane >> 5) * 16;
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
  const int zbase = Lds::kZeroRow * kConvPitch + (lane >> 5) * 16;

  v16i acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = v16i{};

  const int nchunks = (a.Cout + 63) >> 6;
  for (int cc = 0; cc < nchunks; ++cc) {
    if (cc > 0) __syncthreads();  // the previous chunk's fragments are consumed
    // ---- load: halo pieces (row h, half hf: 32 codes of o) and weight pieces
    v4u ga[Lds::kAPieces][NS];
    v4u wb[Lds::kBPieces];
#pragma unroll
    for (int q = 0; q < Lds::kAPieces; ++q) {
      const int p = tid + q * kConvThreads;
      const int h = p >> 1, hf = p & 1;
      const int pix = t0 - hoff + h;
      const bool in = p < 2 * hrows && pix >= 0 && pix < a.T && cc * 64 + hf * 32 < a.Cout;
      const int off = in ? pix * rowb + cc * 32 + hf * 16 : kOutOfRange;
#pragma unroll
      for (int s = 0; s < NS; ++s) ga[q][s] = __builtin_amdgcn_raw_buffer_load_b128(rsg[s], off, 0, 0);
    }
#pragma unroll
    for (int q = 0; q < Lds::kBPieces; ++q) {
      const int p = tid + q * kConvThreads;
      const int row = p >> 1, hf = p & 1;              // row = tap * 64 + c
      const int tap = row >> 6, c = row & 63;
      const bool in = p < 2 * 9 * kConvBN && c0 + c < a.C && cc * 64 + hf * 32 < a.Cout;
      const int off = in ? (tap * a.C + c0 + c) * rowb + cc * 32 + hf * 16 : kOutOfRange;
      wb[q] = __builtin_amdgcn_raw_buffer_load_b128(rsw, off, 0, 0);
    }
    // ---- expand to int8 in LDS (even-k nibbles of a word in one word, odd-k
    // in the next; both operands alike)
#pragma unroll
    for (int q = 0; q < Lds::kAPieces; ++q) {
      const int p = tid + q * kConvThreads;
      if (p >= 2 * hrows) continue;
      const int h = p >> 1, hf = p & 1;
      uint32_t w[8];
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        if constexpr (NS == 1) {
          expand_luq(ga[q][0][d], w[2 * d], w[2 * d + 1]);
        } else {
          uint32_t l0, h0, l1, h1;
          expand_luq_excess64(ga[q][0][d], l0, h0);
          expand_luq_excess64(ga[q][1][d], l1, h1);
          w[2 * d] = (l0 + l1) ^ 0x80808080u;
          w[2 * d + 1] = (h0 + h1) ^ 0x80808080u;
        }
      }
      uint4* dst = reinterpret_cast<uint4*>(As + h * kConvPitch + hf * 32);
      dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
      dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
    }
#pragma unroll
    for (int q = 0; q < Lds::kBPieces; ++q) {
      const int p = tid + q * kConvThreads;
      if (p >= 2 * 9 * kConvBN) continue;
      const int row = p >> 1, hf = p & 1;
      uint32_t w[8];
#pragma unroll
      for (int d = 0; d < 4; ++d) expand_int4<WSIGNED>(wb[q][d], w[2 * d], w[2 * d + 1]);
      uint4* dst = reinterpret_cast<uint4*>(Bs + row * kConvPitch + hf * 32);
      dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
      dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
    }
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
  }

  // ---- epilogue through LDS: lane l of MFMA tile (i, j) holds pixel row l%32
  // and, in registers 4q..4q+3, channels 8q + 4*(l/32) + 0..3 of the 32.  Each
  // wave stages 32 rows x 64 channels, then stores 16-byte row segments
  // (16 lanes per row, 4 rows per instruction).
  constexpr int EP = 64 + 4;  // slab pitch in words
  static_assert(4 * 32 * EP * 4 <= Lds::kBytes, "epilogue slabs fit");
  uint32_t* E = reinterpret_cast<uint32_t*>(lds) + wave * 32 * EP;
  const float sc = epilogue_scale<kAcLuq, NS, WSIGNED>(*a.alpha, *a.wscale);
  const int srow = lane >> 4, scol = (lane & 15) * 4;
  __syncthreads();  // every wave is done with the operands in LDS
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v4u v;
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = __float_as_uint(__fmul_rn((float)acc[i][j][4 * q + r], sc));
        *reinterpret_cast<v4u*>(E + (lane & 31) * EP + j * 32 + 8 * q + 4 * (lane >> 5)) = v;
      }
    __syncthreads();
#pragma unroll
    for (int rr = 0; rr < 32; rr += 4) {
      const int t = t0 + wave * 64 + i * 32 + rr + srow;
      const int c = c0 + scol;
      if (t < a.T && c < a.C) {
        const v4u v = *reinterpret_cast<const v4u*>(E + (rr + srow) * EP + scol);
        float* dst = a.dact + (int64_t)t * a.C + c;
        if (a.vec) {
          *reinterpret_cast<v4u*>(dst) = v;
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (c + r < a.C) dst[r] = __uint_as_float(v[r]);
        }
      }
    }
    __syncthreads();
  }
}

template <int MAXW, int NS>
static void conv_launch_w(const ConvArgs& a, int wsigned, dim3 grid, hipStream_t st) {
  if (wsigned)
    hipLaunchKernelGGL((conv3x3_dgrad_kernel<MAXW, NS, true>), grid, dim3(kConvThreads), 0, st, a);
  else
    hipLaunchKernelGGL((conv3x3_dgrad_kernel<MAXW, NS, false>), grid, dim3(kConvThreads), 0, st, a);
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
  const dim3 grid((unsigned)a.tiles_m, (unsigned)((C + kConvBN - 1) / kConvBN));
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
// with t' = (b, y + kh - 1, x + kw - 1) for t = (b, y, x), terms whose t' lies
// off the image left out.  Operands are the transposed code layouts (pixels
// innermost): g^T [Cout][T] and a^T [C][T].
//
// A workgroup owns 64 output channels o, 64 input channels c and a range of
// pixels t, for all nine taps (the reduction is split over pixel ranges; the
// int32 chunk sums are combined by splitk_reduce_kernel).  Per stage of 128
// pixels it expands into LDS, in element order (one int8 per pixel):
//   - the gradient codes of its 64 output channels at those pixels, three
//     times: for the taps kw = 0, 1, 2, the first and last with the pixels at
//     x = 0 and x = W - 1 zeroed (a tap that leaves the image sideways lands,
//     in the flat pixel index, on the neighbouring row, whose product must
//     not count);
//   - a window of the activation codes of its 64 input channels covering
//     every pixel a tap reads: in the flat pixel index the tap (kh, kw) is the
//     shift (kh - 1) * W + kw - 1, so the window spans 2W + 2 pixels more.
// Twelve waves, one per kernel row kh, half of the input and half of the
// output channels, multiply the three taps kw of their row: a tap's B
// fragment is the window read at its shift (dword-aligned LDS reads and
// v_alignbyte, the shift being wave-uniform); for kh = 0 and 2 the A
// fragment is and-ed with the byte mask of y = 0 or y = H - 1 (mask tables
// built once per workgroup for its pixels).  Operands are double-buffered in
// LDS: the expansion of stage t+1 is cut into one piece per 32-deep k-step
// and issued after that k-step's MFMAs of stage t, one barrier per stage.
// ---------------------------------------------------------------------------

constexpr int kWgThreads = 768;
constexpr int kWgBK = 128;                     // pixels per stage
constexpr int kWgMaxChunk = 2048;              // pixels per split (mask table bytes)
constexpr int kWgApitch = kWgBK + 16;          // A rows (bytes)
constexpr int kWgAcopy = 64 * kWgApitch;       // one masked copy of the A stage

template <int MAXW>
struct WgLds {
  // window pixels: a tap reads up to 145 + 2W bytes into it, 20 at a time
  static constexpr int kWin = (165 + 2 * MAXW + 31) / 32 * 32;
  static constexpr int kBpitch = kWin + 4;     // odd number of dwords per row
  static constexpr int kWinChunks = 64 * (kWin / 32);
  static constexpr int kStage = 3 * kWgAcopy + 64 * kBpitch;
};

struct ConvWgArgs {
  const uint8_t* g;      // LUQ codes [Cout][T], ns planes
  int64_t g_plane;
  const uint8_t* a;      // INT4 codes [C][T]
  const float* alpha;
  const float* ascale;
  float* dw;             // [Cout][9C]
  int32_t* partial;      // [splits][Cout][9C] chunk sums, or null
  int T, H, W, C, Cout;
  int kchunk;            // pixels per split, a multiple of kWgBK, <= kWgMaxChunk
  int ctiles;            // ceil(C / 64)
  int vec;               // 16-byte stores of dW rows
};

// Element-order bytes from the even / odd split of the GEMM expansions:
// e holds elements 0, 2, 4, 6 and o elements 1, 3, 5, 7.
__device__ __forceinline__ void interleave_bytes(uint32_t e, uint32_t o, uint32_t& lo, uint32_t& hi) {
  lo = __builtin_amdgcn_perm(o, e, 0x05010400u);
  hi = __builtin_amdgcn_perm(o, e, 0x07030602u);
}

template <int MAXW, int NS, bool ASIGNED>
__global__ __launch_bounds__(kWgThreads, 1) void conv3x3_wgrad_kernel(ConvWgArgs a) {
  using Lds = WgLds<MAXW>;
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * Lds::kStage];
  __shared__ __attribute__((aligned(16))) uint8_t vmask[4][kWgMaxChunk];  // 0xFF: y != 0, y != H-1, x != 0, x != W-1

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ct = blockIdx.x % a.ctiles;
  const int ot = blockIdx.x / a.ctiles;
  const int o0 = ot * 64, c0 = ct * 64;
  const int kb = blockIdx.y * a.kchunk;
  const int ke = min(kb + a.kchunk, a.T);
  const int nst = (ke - kb + kWgBK - 1) / kWgBK;
  const int rowb = a.T >> 1;  // bytes per code row of either operand
  // the smallest tap shift is -(W + 1); the window starts at the 32-pixel
  // boundary at or below it
  const int smin = -(a.W + 1);
  const int wq = -(((-smin) + 31) >> 5) * 32;
  const int wr = smin - wq;  // 0..31

  for (int p = tid; p < nst * kWgBK; p += kWgThreads) {
    const int t = kb + p;
    uint32_t my0 = 0, my2 = 0, mx0 = 0, mx2 = 0;
    if (t < ke) {
      const int r = t / a.W, x = t - r * a.W;
      const int y = r % a.H;
      my0 = y != 0 ? 0xFFu : 0u;
      my2 = y != a.H - 1 ? 0xFFu : 0u;
      mx0 = x != 0 ? 0xFFu : 0u;
      mx2 = x != a.W - 1 ? 0xFFu : 0u;
    }
    vmask[0][p] = (uint8_t)my0;
    vmask[1][p] = (uint8_t)my2;
    vmask[2][p] = (uint8_t)mx0;
    vmask[3][p] = (uint8_t)mx2;
  }

  __amdgpu_buffer_rsrc_t rsg[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s)
    rsg[s] = __builtin_amdgcn_make_buffer_rsrc((void*)(a.g + s * a.g_plane), (short)0, a.Cout * rowb, kBufferFlags);
  const __amdgpu_buffer_rsrc_t rsa =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.a, (short)0, a.C * rowb, kBufferFlags);

  // load slots: threads 0..255 one A chunk (row tid/4, 32 pixels tid%4);
  // window chunks q = tid, tid + 768, ... (row q / (kWin/32), 32 pixels)
  constexpr int WC = Lds::kWin / 32;
  constexpr int BQ = (Lds::kWinChunks + kWgThreads - 1) / kWgThreads;
  static_assert(BQ <= 3, "window chunks fit three expansion pieces");
  const bool has_a = tid < 256;
  const int arow = (tid & 255) >> 2, ajc = tid & 3;
  const bool aok = has_a && o0 + arow < a.Cout;
  struct Regs {
    v4u g[NS];
    v4u b[BQ];
  };
  auto load = [&](Regs& r, int t) {
    const int k0 = kb + t * kWgBK;
    const int ka = k0 + ajc * 32;
    const int offa = aok && ka < ke ? (o0 + arow) * rowb + (ka >> 1) : kOutOfRange;
#pragma unroll
    for (int s = 0; s < NS; ++s) r.g[s] = __builtin_amdgcn_raw_buffer_load_b128(rsg[s], offa, 0, 0);
#pragma unroll
    for (int u = 0; u < BQ; ++u) {
      const int q = tid + u * kWgThreads;
      const int row = q / WC, jc = q - (q / WC) * WC;
      const int kw0 = k0 + wq + jc * 32;
      const bool ok = q < Lds::kWinChunks && c0 + row < a.C && kw0 >= 0 && kw0 < a.T;
      r.b[u] = __builtin_amdgcn_raw_buffer_load_b128(rsa, ok ? (c0 + row) * rowb + (kw0 >> 1) : kOutOfRange, 0, 0);
    }
  };
  // expansion piece 0: the A chunk (three copies); pieces 1..BQ: window chunks
  auto expand_piece = [&](const Regs& r, int t, uint8_t* stage, int piece) {
    uint32_t w[8];
    if (piece == 0) {
      if (!has_a) return;
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        uint32_t e, o;
        if constexpr (NS == 1) {
          expand_luq(r.g[0][d], e, o);
        } else {
          uint32_t e0, o0_, e1, o1;
          expand_luq_excess64(r.g[0][d], e0, o0_);
          expand_luq_excess64(r.g[1][d], e1, o1);
          e = (e0 + e1) ^ 0x80808080u;
          o = (o0_ + o1) ^ 0x80808080u;
        }
        interleave_bytes(e, o, w[2 * d], w[2 * d + 1]);
      }
      const int mp = t * kWgBK + ajc * 32;
      const uint4* m0 = reinterpret_cast<const uint4*>(&vmask[2][mp]);
      const uint4* m2 = reinterpret_cast<const uint4*>(&vmask[3][mp]);
      const uint4 a0 = m0[0], a1 = m0[1], b0 = m2[0], b1 = m2[1];
      uint4* d0 = reinterpret_cast<uint4*>(stage + arow * kWgApitch + ajc * 32);
      uint4* d1 = reinterpret_cast<uint4*>(stage + kWgAcopy + arow * kWgApitch + ajc * 32);
      uint4* d2 = reinterpret_cast<uint4*>(stage + 2 * kWgAcopy + arow * kWgApitch + ajc * 32);
      d0[0] = make_uint4(w[0] & a0.x, w[1] & a0.y, w[2] & a0.z, w[3] & a0.w);
      d0[1] = make_uint4(w[4] & a1.x, w[5] & a1.y, w[6] & a1.z, w[7] & a1.w);
      d1[0] = make_uint4(w[0], w[1], w[2], w[3]);
      d1[1] = make_uint4(w[4], w[5], w[6], w[7]);
      d2[0] = make_uint4(w[0] & b0.x, w[1] & b0.y, w[2] & b0.z, w[3] & b0.w);
      d2[1] = make_uint4(w[4] & b1.x, w[5] & b1.y, w[6] & b1.z, w[7] & b1.w);
      return;
    }
    const int u = piece - 1;
    if (u >= BQ) return;
    const int q = tid + u * kWgThreads;
    if (q >= Lds::kWinChunks) return;
    const int row = q / WC, jc = q - (q / WC) * WC;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      uint32_t e, o;
      expand_int4<ASIGNED>(r.b[u][d], e, o);
      interleave_bytes(e, o, w[2 * d], w[2 * d + 1]);
    }
    uint32_t* db = reinterpret_cast<uint32_t*>(stage + 3 * kWgAcopy + row * Lds::kBpitch + jc * 32);
#pragma unroll
    for (int k = 0; k < 8; ++k) db[k] = w[k];
  };

  // wave: kernel row kh, input channels cj*32 .. +31, output channels oi*32 .. +31
  const int kh = wave >> 2, cj = (wave >> 1) & 1, oi = wave & 1;
  const int r32 = lane & 31, h = lane >> 5;
  const int sh = wr + kh * a.W;  // window offset of the tap (kh, 0)
  const int aoff = (oi * 32 + r32) * kWgApitch;
  const int boff = 3 * kWgAcopy + (cj * 32 + r32) * Lds::kBpitch;
  v16i acc[3];
#pragma unroll
  for (int kw = 0; kw < 3; ++kw) acc[kw] = v16i{};
  auto mfma_kstep = [&](const uint8_t* stage, int t, int kk) {
    const int p = kk * 32 + 16 * h;
    v4u ym = v4u{0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu};
    if (kh != 1) ym = *reinterpret_cast<const v4u*>(&vmask[kh >> 1][t * kWgBK + p]);
#pragma unroll
    for (int kw = 0; kw < 3; ++kw) {
      const v4u fa = *reinterpret_cast<const v4u*>(stage + kw * kWgAcopy + aoff + p) & ym;
      const int s = p + sh + kw;
      const uint32_t* src = reinterpret_cast<const uint32_t*>(stage + boff + (s & ~3));
      uint32_t x[5];
#pragma unroll
      for (int d = 0; d < 5; ++d) x[d] = src[d];
      v4i fb;
#pragma unroll
      for (int d = 0; d < 4; ++d) fb[d] = (int)__builtin_amdgcn_alignbyte(x[d + 1], x[d], (uint32_t)(s & 3));
      acc[kw] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fb, (v4i)fa, acc[kw], 0, 0, 0);
    }
  };
  // one pipeline step: multiply stage t (buffer cb) while expanding stage t+1
  // (registers r) into the other buffer, then refill r with stage t+3
  auto step = [&](int cb, int t, Regs& r) {
    uint8_t* cur = lds + cb * Lds::kStage;
    uint8_t* nxt = lds + (cb ^ 1) * Lds::kStage;
    const bool more = t + 1 < nst;
#pragma unroll
    for (int kk = 0; kk < kWgBK / 32; ++kk) {
      mfma_kstep(cur, t, kk);
      if (more) expand_piece(r, t + 1, nxt, kk);
    }
    if (t + 3 < nst) load(r, t + 3);
    __syncthreads();
  };

  __syncthreads();  // the mask tables are written
  Regs r0, r1;
  load(r0, 0);
  if (1 < nst) load(r1, 1);
#pragma unroll
  for (int piece = 0; piece < 4; ++piece) expand_piece(r0, 0, lds, piece);
  if (2 < nst) load(r0, 2);
  __syncthreads();
  for (int t = 0; t < nst; t += 2) {
    step(0, t, r1);                     // multiply t, expand t+1 (r1), reload r1 with t+3
    if (t + 1 < nst) step(1, t + 1, r0);  // multiply t+1, expand t+2 (r0), reload r0 with t+4
  }

  // lane holds output channel o0 + oi*32 + l%32 and input channels
  // c0 + cj*32 + 8q + 4*(l/32) + 0..3 of tap (kh, kw) in registers 4q..4q+3
  const bool part = a.partial != nullptr;
  const float sc = part ? 0.0f : epilogue_scale<kAcLuq, NS, ASIGNED>(*a.alpha, *a.ascale);
  const int64_t ncol = 9LL * a.C;
  uint32_t* out = part ? reinterpret_cast<uint32_t*>(a.partial + (int64_t)blockIdx.y * a.Cout * ncol)
                       : reinterpret_cast<uint32_t*>(a.dw);
  const int o = o0 + oi * 32 + r32;
  if (o < a.Cout) {
#pragma unroll
    for (int kw = 0; kw < 3; ++kw)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c = c0 + cj * 32 + 8 * q + 4 * h;
        if (c >= a.C) continue;
        v4u v;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int32_t x = acc[kw][4 * q + r];
          v[r] = part ? (uint32_t)x : __float_as_uint(__fmul_rn((float)x, sc));
        }
        uint32_t* dst = out + (int64_t)o * ncol + (kh * 3 + kw) * a.C + c;
        if (a.vec) {
          *reinterpret_cast<v4u*>(dst) = v;
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (c + r < a.C) dst[r] = v[r];
        }
      }
  }
}

struct ConvWgPlan {
  int kchunk, splits;
};

static ConvWgPlan plan_conv_wgrad(int64_t T, int64_t C, int64_t Cout) {
  const int64_t tiles = ((Cout + 63) / 64) * ((C + 63) / 64);
  const int64_t want = (256 + tiles - 1) / tiles;  // one workgroup per CU
  int64_t kc = (T + want - 1) / want;
  kc = (kc + kWgBK - 1) / kWgBK * kWgBK;
  if (kc < 4 * kWgBK) kc = 4 * kWgBK;              // at least 4 stages per split
  if (kc > kWgMaxChunk) kc = kWgMaxChunk;
  ConvWgPlan p;
  p.kchunk = (int)kc;
  p.splits = (int)((T + kc - 1) / kc);
  return p;
}

size_t conv3x3_wgrad_workspace_bytes(int64_t T, int64_t C, int64_t Cout) {
  const ConvWgPlan p = plan_conv_wgrad(T, C, Cout);
  return p.splits > 1 ? (size_t)p.splits * (size_t)Cout * (size_t)(9 * C) * sizeof(int32_t) : 0;
}

template <int MAXW, int NS, bool ASIGNED>
static void conv_wgrad_launch_t(const ConvWgArgs& a, dim3 grid, hipStream_t st) {
  hipLaunchKernelGGL((conv3x3_wgrad_kernel<MAXW, NS, ASIGNED>), grid, dim3(kWgThreads), 0, st, a);
  if (a.partial) {
    const int64_t MN = (int64_t)a.Cout * 9 * a.C;
    hipLaunchKernelGGL((splitk_reduce_kernel<kAcLuq, NS, ASIGNED>), dim3((unsigned)((MN + 63) / 64)), dim3(256), 0, st,
                       a.partial, (int)grid.y, MN, a.alpha, a.ascale, a.dw);
  }
}

template <int MAXW>
static void conv_wgrad_launch_w(const ConvWgArgs& a, int ns, int a_signed, dim3 grid, hipStream_t st) {
  if (ns == 1)
    a_signed ? conv_wgrad_launch_t<MAXW, 1, true>(a, grid, st) : conv_wgrad_launch_t<MAXW, 1, false>(a, grid, st);
  else
    a_signed ? conv_wgrad_launch_t<MAXW, 2, true>(a, grid, st) : conv_wgrad_launch_t<MAXW, 2, false>(a, grid, st);
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
  a.partial = p.splits > 1 ? static_cast<int32_t*>(ws) : nullptr;
  a.T = (int)T;
  a.H = (int)H;
  a.W = (int)W;
  a.C = (int)C;
  a.Cout = (int)Cout;
  a.kchunk = p.kchunk;
  a.ctiles = (int)((C + 63) / 64);
  a.vec = (C % 4) == 0 && (((uintptr_t)(a.partial ? (void*)a.partial : (void*)dw)) & 15) == 0;
  const dim3 grid((unsigned)(((Cout + 63) / 64) * a.ctiles), (unsigned)p.splits);
  if (W <= 64)
    conv_wgrad_launch_w<64>(a, ns, a_signed, grid, st);
  else
    conv_wgrad_launch_w<256>(a, ns, a_signed, grid, st);
  return hipGetLastError();
}

}  // namespace luq

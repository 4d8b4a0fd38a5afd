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

}  // namespace luq

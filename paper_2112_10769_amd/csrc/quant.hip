// LUQ and INT4 quantizer kernels (gfx950).
//
// Both quantizers are two passes over the input, because every code depends
// on a tensor-wide maximum (Eq. alpha of the paper for LUQ; the INT4 range of
// Appendix A.1):
//   1. max pass   -- grid-stride 16-byte loads, one partial max per block.
//   2. encode     -- every block first folds the partials (<= 1024 words,
//                    L2 resident) into the tensor maximum, then encodes a
//                    grid-stride share of the tensor.
// Keys are float32 bit patterns of |x|, whose unsigned order is the float
// order; NaN / Inf land above every finite key and mark the tensor
// non-finite.
//
// LUQ encode (Section 4): one Philox4x32-10 call yields the 16-bit uniforms
// of 8 consecutive elements.  The rounding decision j * w < d * 2^16 is made
// exactly as the sign of fmaf(j, w * 2^-16, -d): d is exact (Sterbenz), j*w
// has at most 40 significant bits and the fused result is rounded once, so
// its sign is the sign of the exact difference as long as w * 2^-16 is a
// normal float.  When max|g| < 2^-90 every magnitude and level is first
// multiplied by 2^100 (exact: scaling up by a power of two) so that this
// holds for any finite input.
//
// The "tile" encoders also write the transposed code matrix: each lane owns
// an 8x8 element block, packs its 8 row words and transposes them with a
// 4-bit field-swap network in registers.
#include "luq_device.hpp"
#include "luq_launch.hpp"

namespace luq {

constexpr int kThreads = 256;
constexpr int kMaxPartials = 1024;
constexpr int kMaxEncodeBlocks = 4096;

// Max-pass keys.  MODE 0: |x| (LUQ, signed INT4).  MODE 1: max(x, 0) with
// non-finite values of either sign kept (unsigned INT4).
template <int MODE>
__device__ __forceinline__ uint32_t max_key(uint32_t b) {
  const uint32_t a = b & 0x7FFFFFFFu;
  if constexpr (MODE == 0) return a;
  return (a >= 0x7F800000u) ? a : ((b >> 31) ? 0u : b);
}

template <bool BF16, int MODE>
__global__ __launch_bounds__(kThreads) void max_partial_kernel(const void* __restrict__ x, int64_t n,
                                                              uint32_t* __restrict__ partial) {
  __shared__ uint32_t scratch[kThreads / kWave];
  const int64_t ngroups = n >> 3;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  uint32_t m0 = 0, m1 = 0;
  int64_t g = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  // two groups per trip keep four 16-byte loads in flight for float32
  for (; g + stride < ngroups; g += 2 * stride) {
    const U8 a = load8<BF16>(x, g * 8);
    const U8 b = load8<BF16>(x, (g + stride) * 8);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      m0 = max(m0, max_key<MODE>(a.v[i]));
      m1 = max(m1, max_key<MODE>(b.v[i]));
    }
  }
  if (g < ngroups) {
    const U8 a = load8<BF16>(x, g * 8);
#pragma unroll
    for (int i = 0; i < 8; ++i) m0 = max(m0, max_key<MODE>(a.v[i]));
  }
  if (blockIdx.x == 0 && threadIdx.x == 0 && (n & 7)) {
    const U8 a = load8_tail<BF16>(x, ngroups * 8, n);  // missing elements read +0 (key 0)
#pragma unroll
    for (int i = 0; i < 8; ++i) m0 = max(m0, max_key<MODE>(a.v[i]));
  }
  const uint32_t m = block_max_u32(max(m0, m1), scratch);
  if (threadIdx.x == 0) partial[blockIdx.x] = m;
}

// ------------------------------- LUQ ---------------------------------------

struct LuqParams {
  float alpha_s;    // alpha * S
  float alpha16_s;  // alpha * S * 2^-16
  float ltop_s;     // alpha * S * 2^R
  float S;          // 1 or 2^100
  uint32_t a_bits;  // bits of alpha_s
  uint32_t a16_bits;
  uint32_t e_alpha;  // biased exponent of alpha_s
  uint32_t m_alpha;  // mantissa field of alpha_s
  uint32_t top_field;
  bool zero;  // every code is 0 (alpha == 0, or non-finite input)
};

// Eq. alpha: alpha = fl32(m * 2^-R).  `alpha_out` gets the unscaled alpha.
__device__ __forceinline__ LuqParams luq_params(uint32_t mbits, int R, float* alpha_out) {
  LuqParams p;
  const float m = __uint_as_float(mbits);
  float alpha;
  if (mbits >= 0x7F800000u) {
    alpha = __uint_as_float(0x7FC00000u);  // NaN
    p.zero = true;
  } else {
    alpha = m * __uint_as_float((uint32_t)(127 - R) << 23);  // exact 2^-R scale, one rounding
    p.zero = (alpha == 0.0f);
  }
  *alpha_out = alpha;
  p.S = (m < 0x1p-90f) ? 0x1p100f : 1.0f;
  p.alpha_s = alpha * p.S;
  p.alpha16_s = p.alpha_s * 0x1p-16f;
  p.ltop_s = p.alpha_s * __uint_as_float((uint32_t)(127 + R) << 23);
  p.a_bits = __float_as_uint(p.alpha_s);
  p.a16_bits = __float_as_uint(p.alpha16_s);
  p.e_alpha = p.a_bits >> 23;
  p.m_alpha = p.a_bits & 0x7FFFFFu;
  p.top_field = (uint32_t)R + 1;
  return p;
}

// One element's 4-bit LUQ code from its float32 bits and 16-bit uniform.
__device__ __forceinline__ uint32_t luq_nibble(uint32_t b, uint32_t j, const LuqParams& p) {
  const float as = __uint_as_float(b & 0x7FFFFFFFu) * p.S;
  const uint32_t ab = __float_as_uint(as);
  const bool under = as < p.alpha_s;  // stochastic underflow bin [0, alpha)
  const bool top = as >= p.ltop_s;    // the largest level
  // bin index n: the largest n with alpha * 2^n <= |x| (meaningful when
  // neither under nor top, where |x| and alpha are normal floats)
  const uint32_t n = (ab >> 23) - p.e_alpha - ((ab & 0x7FFFFFu) < p.m_alpha ? 1u : 0u);
  const float lo = under ? 0.0f : __uint_as_float(p.a_bits + (n << 23));
  const float w16 = under ? p.alpha16_s : __uint_as_float(p.a16_bits + (n << 23));
  const float d = as - lo;  // exact
  const bool up = fmaf((float)j, w16, -d) < 0.0f;
  const uint32_t field = top ? p.top_field : (under ? (uint32_t)up : n + 1u + (uint32_t)up);
  const uint32_t sgn = (field != 0u) ? ((b >> 31) << 3) : 0u;
  return field | sgn;
}

// Codes of 8 consecutive elements (bits in v) for Philox block `blk`.
__device__ __forceinline__ uint32_t luq_word(const U8& v, uint64_t blk, uint32_t sample,
                                             uint32_t counter, uint32_t k0, uint32_t k1,
                                             const LuqParams& p) {
  const U4 y = philox4x32_10(U4{(uint32_t)blk, (uint32_t)(blk >> 32), sample, counter}, k0, k1);
  const uint32_t w[4] = {y.x, y.y, y.z, y.w};
  uint32_t out = 0;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint32_t j = (e & 1) ? (w[e >> 1] >> 16) : (w[e >> 1] & 0xFFFFu);
    out |= luq_nibble(v.v[e], j, p) << (4 * e);
  }
  return out;
}

struct LuqArgs {
  const void* g;
  int64_t rows, cols, n;
  int R;
  uint32_t k0, k1, counter;
  const uint32_t* partial;
  int nparts;
  uint8_t* codes;
  uint8_t* codes_t;
  int64_t plane;
  float* alpha_out;
  float* max_out;
};

__device__ __forceinline__ LuqParams luq_block_params(const LuqArgs& a) {
  __shared__ uint32_t scratch[kThreads / kWave];
  const uint32_t mbits = reduce_partials(a.partial, a.nparts, scratch);
  float alpha;
  const LuqParams p = luq_params(mbits, a.R, &alpha);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    *a.alpha_out = alpha;
    if (a.max_out) *a.max_out = __uint_as_float(mbits);
  }
  return p;
}

// Flat row-major codes; groups of 8 elements along the flattened tensor.
template <bool BF16, int NS>
__global__ __launch_bounds__(kThreads) void luq_encode_flat_kernel(LuqArgs a) {
  const LuqParams p = luq_block_params(a);
  const int64_t ngroups = (a.n + 7) >> 3;
  for (int64_t g = (int64_t)blockIdx.x * kThreads + threadIdx.x; g < ngroups;
       g += (int64_t)gridDim.x * kThreads) {
    const bool full = (g * 8 + 8) <= a.n;
    const U8 v = full ? load8<BF16>(a.g, g * 8) : load8_tail<BF16>(a.g, g * 8, a.n);
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const uint32_t word = p.zero ? 0u : luq_word(v, (uint64_t)g, s, a.counter, a.k0, a.k1, p);
      uint8_t* dst = a.codes + s * a.plane + g * 4;
      if (full)
        *reinterpret_cast<uint32_t*>(dst) = word;
      else
        store_bytes(dst, word, (int)((a.n - g * 8 + 1) >> 1));
    }
  }
}

// Tile encoder: rows % 8 == 0 and cols % 8 == 0.  A block covers 128 x 128
// elements as 2 x 2 wave tiles of 8 x 8 lanes, each lane an 8 x 8 block.
template <bool BF16, int NS>
__global__ __launch_bounds__(kThreads) void luq_encode_tile_kernel(LuqArgs a) {
  const LuqParams p = luq_block_params(a);
  const int64_t RB = a.rows >> 3, CB = a.cols >> 3;
  const int64_t ntr = (RB + 15) >> 4, ntc = (CB + 15) >> 4;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = (wave >> 1) * 8 + (lane >> 3), lc = (wave & 1) * 8 + (lane & 7);
  for (int64_t t = blockIdx.x; t < ntr * ntc; t += gridDim.x) {
    const int64_t R = (t / ntc) * 16 + lr, C = (t % ntc) * 16 + lc;
    if (R >= RB || C >= CB) continue;
    uint32_t rw[NS][8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int64_t e0 = (R * 8 + r) * a.cols + C * 8;
      const U8 v = load8<BF16>(a.g, e0);
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        rw[s][r] = p.zero ? 0u : luq_word(v, (uint64_t)(e0 >> 3), s, a.counter, a.k0, a.k1, p);
        if (a.codes) *reinterpret_cast<uint32_t*>(a.codes + s * a.plane + (e0 >> 1)) = rw[s][r];
      }
    }
    if (a.codes_t) {
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        transpose8x8_nibbles(rw[s]);
#pragma unroll
        for (int c = 0; c < 8; ++c)
          *reinterpret_cast<uint32_t*>(a.codes_t + s * a.plane + (C * 8 + c) * (a.rows >> 1) + R * 4) =
              rw[s][c];
      }
    }
  }
}

__global__ void write_two_floats_kernel(float* a, float va, float* b, float vb) {
  if (a) *a = va;
  if (b) *b = vb;
}

// ------------------------------- INT4 --------------------------------------

struct Int4Params {
  float inv;
  float lo, hi;
  bool zero;
};

struct Int4Args {
  const void* x;
  int64_t rows, cols, n;
  int is_signed;
  float clip;
  const uint32_t* partial;
  int nparts;
  uint8_t* codes;
  uint8_t* codes_t;
  float* scale_out;
};

__device__ __forceinline__ Int4Params int4_block_params(const Int4Args& a) {
  __shared__ uint32_t scratch[kThreads / kWave];
  Int4Params p;
  const float Q = a.is_signed ? 7.0f : 15.0f;
  float m, s;
  bool nonfinite = false;
  if (a.clip > 0.0f) {
    m = a.clip;
  } else {
    const uint32_t mbits = reduce_partials(a.partial, a.nparts, scratch);
    nonfinite = mbits >= 0x7F800000u;
    m = __uint_as_float(mbits);
  }
  if (nonfinite) {
    s = __uint_as_float(0x7FC00000u);
    p.zero = true;
    p.inv = 0.0f;
  } else if (m == 0.0f) {
    s = 0.0f;
    p.zero = true;
    p.inv = 0.0f;
  } else {
    p.inv = __fdiv_rn(Q, m);
    s = __fdiv_rn(m, Q);
    p.zero = false;
  }
  p.lo = a.is_signed ? -7.0f : 0.0f;
  p.hi = Q;
  if (blockIdx.x == 0 && threadIdx.x == 0) *a.scale_out = s;
  return p;
}

__device__ __forceinline__ uint32_t int4_nibble(uint32_t b, const Int4Params& p) {
  const float v = __uint_as_float(b) * p.inv;
  float q = rintf(v);  // round half to even
  q = fminf(fmaxf(q, p.lo), p.hi);
  q = (v != v) ? 0.0f : q;
  return (uint32_t)(int)q & 0xFu;
}

__device__ __forceinline__ uint32_t int4_word(const U8& v, const Int4Params& p) {
  uint32_t out = 0;
#pragma unroll
  for (int e = 0; e < 8; ++e) out |= int4_nibble(v.v[e], p) << (4 * e);
  return out;
}

template <bool BF16>
__global__ __launch_bounds__(kThreads) void int4_encode_flat_kernel(Int4Args a) {
  const Int4Params p = int4_block_params(a);
  const int64_t ngroups = (a.n + 7) >> 3;
  for (int64_t g = (int64_t)blockIdx.x * kThreads + threadIdx.x; g < ngroups;
       g += (int64_t)gridDim.x * kThreads) {
    const bool full = (g * 8 + 8) <= a.n;
    const U8 v = full ? load8<BF16>(a.x, g * 8) : load8_tail<BF16>(a.x, g * 8, a.n);
    const uint32_t word = p.zero ? 0u : int4_word(v, p);
    if (full)
      *reinterpret_cast<uint32_t*>(a.codes + g * 4) = word;
    else
      store_bytes(a.codes + g * 4, word, (int)((a.n - g * 8 + 1) >> 1));
  }
}

template <bool BF16>
__global__ __launch_bounds__(kThreads) void int4_encode_tile_kernel(Int4Args a) {
  const Int4Params p = int4_block_params(a);
  const int64_t RB = a.rows >> 3, CB = a.cols >> 3;
  const int64_t ntr = (RB + 15) >> 4, ntc = (CB + 15) >> 4;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = (wave >> 1) * 8 + (lane >> 3), lc = (wave & 1) * 8 + (lane & 7);
  for (int64_t t = blockIdx.x; t < ntr * ntc; t += gridDim.x) {
    const int64_t R = (t / ntc) * 16 + lr, C = (t % ntc) * 16 + lc;
    if (R >= RB || C >= CB) continue;
    uint32_t rw[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int64_t e0 = (R * 8 + r) * a.cols + C * 8;
      const U8 v = load8<BF16>(a.x, e0);
      rw[r] = p.zero ? 0u : int4_word(v, p);
      if (a.codes) *reinterpret_cast<uint32_t*>(a.codes + (e0 >> 1)) = rw[r];
    }
    if (a.codes_t) {
      transpose8x8_nibbles(rw);
#pragma unroll
      for (int c = 0; c < 8; ++c)
        *reinterpret_cast<uint32_t*>(a.codes_t + (C * 8 + c) * (a.rows >> 1) + R * 4) = rw[c];
    }
  }
}

// ------------------------------- launchers ---------------------------------

static int max_pass_blocks(int64_t n) {
  const int64_t groups = (n + 7) >> 3;
  int64_t b = (groups + kThreads * 4 - 1) / (kThreads * 4);
  if (b < 1) b = 1;
  if (b > kMaxPartials) b = kMaxPartials;
  return (int)b;
}

size_t quant_workspace_bytes(int64_t /*n*/) { return kMaxPartials * sizeof(uint32_t); }

static int encode_blocks_flat(int64_t n) {
  const int64_t groups = (n + 7) >> 3;
  int64_t b = (groups + kThreads - 1) / kThreads;
  if (b < 1) b = 1;
  if (b > kMaxEncodeBlocks) b = kMaxEncodeBlocks;
  return (int)b;
}

static int encode_blocks_tile(int64_t rows, int64_t cols) {
  const int64_t tiles = (((rows >> 3) + 15) >> 4) * (((cols >> 3) + 15) >> 4);
  int64_t b = tiles < 1 ? 1 : tiles;
  if (b > kMaxEncodeBlocks) b = kMaxEncodeBlocks;
  return (int)b;
}

template <bool BF16>
static hipError_t luq_launch_t(const LuqArgs& a, int ns, int nmax, hipStream_t st) {
  hipLaunchKernelGGL((max_partial_kernel<BF16, 0>), dim3(nmax), dim3(kThreads), 0, st, a.g, a.n,
                     const_cast<uint32_t*>(a.partial));
  if (a.codes_t) {
    const int nb = encode_blocks_tile(a.rows, a.cols);
    if (ns == 1)
      hipLaunchKernelGGL((luq_encode_tile_kernel<BF16, 1>), dim3(nb), dim3(kThreads), 0, st, a);
    else
      hipLaunchKernelGGL((luq_encode_tile_kernel<BF16, 2>), dim3(nb), dim3(kThreads), 0, st, a);
  } else {
    const int nb = encode_blocks_flat(a.n);
    if (ns == 1)
      hipLaunchKernelGGL((luq_encode_flat_kernel<BF16, 1>), dim3(nb), dim3(kThreads), 0, st, a);
    else
      hipLaunchKernelGGL((luq_encode_flat_kernel<BF16, 2>), dim3(nb), dim3(kThreads), 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_luq_quantize(const void* g, int bf16, int64_t rows, int64_t cols, int R,
                               uint64_t seed, uint32_t counter, int ns, uint8_t* codes,
                               uint8_t* codes_t, float* alpha, float* maxabs, void* ws,
                               hipStream_t st) {
  const int64_t n = rows * cols;
  if (n == 0) {
    hipLaunchKernelGGL(write_two_floats_kernel, dim3(1), dim3(1), 0, st, alpha, 0.0f, maxabs, 0.0f);
    return hipGetLastError();
  }
  LuqArgs a;
  a.g = g;
  a.rows = rows;
  a.cols = cols;
  a.n = n;
  a.R = R;
  a.k0 = (uint32_t)seed;
  a.k1 = (uint32_t)(seed >> 32);
  a.counter = counter;
  a.partial = static_cast<uint32_t*>(ws);
  a.nparts = max_pass_blocks(n);
  a.codes = codes;
  a.codes_t = codes_t;
  a.plane = (int64_t)plane_bytes(n);
  a.alpha_out = alpha;
  a.max_out = maxabs;
  return bf16 ? luq_launch_t<true>(a, ns, a.nparts, st) : luq_launch_t<false>(a, ns, a.nparts, st);
}

template <bool BF16>
static hipError_t int4_launch_t(const Int4Args& a, hipStream_t st) {
  if (a.clip <= 0.0f) {
    if (a.is_signed)
      hipLaunchKernelGGL((max_partial_kernel<BF16, 0>), dim3(a.nparts), dim3(kThreads), 0, st, a.x,
                         a.n, const_cast<uint32_t*>(a.partial));
    else
      hipLaunchKernelGGL((max_partial_kernel<BF16, 1>), dim3(a.nparts), dim3(kThreads), 0, st, a.x,
                         a.n, const_cast<uint32_t*>(a.partial));
  }
  if (a.codes_t)
    hipLaunchKernelGGL((int4_encode_tile_kernel<BF16>), dim3(encode_blocks_tile(a.rows, a.cols)),
                       dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL((int4_encode_flat_kernel<BF16>), dim3(encode_blocks_flat(a.n)),
                       dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_int4_quantize(const void* x, int bf16, int64_t rows, int64_t cols, int is_signed,
                                float clip, uint8_t* codes, uint8_t* codes_t, float* scale,
                                void* ws, hipStream_t st) {
  const int64_t n = rows * cols;
  if (n == 0) {
    hipLaunchKernelGGL(write_two_floats_kernel, dim3(1), dim3(1), 0, st, scale, 0.0f,
                       (float*)nullptr, 0.0f);
    return hipGetLastError();
  }
  Int4Args a;
  a.x = x;
  a.rows = rows;
  a.cols = cols;
  a.n = n;
  a.is_signed = is_signed;
  a.clip = clip;
  a.partial = static_cast<uint32_t*>(ws);
  a.nparts = max_pass_blocks(n);
  a.codes = codes;
  a.codes_t = codes_t;
  a.scale_out = scale;
  return bf16 ? int4_launch_t<true>(a, st) : int4_launch_t<false>(a, st);
}

}  // namespace luq

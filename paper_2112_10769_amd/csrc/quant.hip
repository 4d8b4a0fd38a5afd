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
// The "tile" encoders also write the transposed code matrix (see
// encode_tiles below).
#include <atomic>

#include "luq_device.hpp"
#include "luq_launch.hpp"

namespace luq {

constexpr int kThreads = 256;
// Partials of the max pass.  Up to kDirectPartials, every encode block
// folds them itself; beyond that (large tensors, more max-pass blocks in
// flight) one extra block folds them into the word after the partials.
constexpr int kDirectPartials = 2048;
constexpr int kMaxPartials = 16384;
constexpr int kMaxEncodeBlocks = 4096;
// Word of the quantizer workspace after the partials and their fold: the
// status of the last call (kStatusTag | LUQ_OK or LUQ_ERR_NONFINITE).
constexpr int kStatusWord = kMaxPartials + 1;
constexpr uint32_t kStatusNonfinite = 8;  // LUQ_ERR_NONFINITE
// Tensors above kCacheBytes (the 256 MB last-level cache) are streamed: the
// max pass reads all but the last kKeepBytes of them non-temporally and the
// encode pass, whose loads (and LUQ code stores) are then non-temporal too,
// walks the tensor from its end, so that it starts on the part the max pass
// left in the cache.
constexpr int64_t kCacheBytes = 256LL << 20;
constexpr int64_t kKeepBytes = 192LL << 20;
// INT4 tensors stream from a lower size: a tensor as large as the cache does not
// stay in it beside the other data of a training step, and the INT4 encode is
// bound by memory (the LUQ encode, bound by its ALU work, keeps kCacheBytes).
// Their max pass keeps no tail cached: read through the cache, that tail
// evicted (and waited for the write-back of) what the step's earlier kernels
// left there.
constexpr int64_t kInt4StreamBytes = 160LL << 20;

// Max-pass keys.  MODE 0: |x| (LUQ, signed INT4).  MODE 1: max(x, 0) with
// non-finite values of either sign kept (unsigned INT4).
template <int MODE>
__device__ __forceinline__ uint32_t max_key(uint32_t b) {
  const uint32_t a = b & 0x7FFFFFFFu;
  if constexpr (MODE == 0) return a;
  return (a >= 0x7F800000u) ? a : ((b >> 31) ? 0u : b);
}

// Max key |x| over 8 elements.
__device__ __forceinline__ uint32_t max_key8(const U8& v) {
  uint32_t m = v.v[0] & 0x7FFFFFFFu;
#pragma unroll
  for (int e = 1; e < 8; ++e) m = max(m, v.v[e] & 0x7FFFFFFFu);
  return m;
}

template <bool BF16, int MODE, bool NT>
__global__ __launch_bounds__(kThreads) void max_partial_kernel(const void* __restrict__ x, int64_t n,
                                                              uint32_t* __restrict__ partial, int64_t keep) {
  // groups of 8 elements per trip: eight 16-byte loads in flight per thread
  constexpr int G = BF16 ? 8 : 4;
  __shared__ uint32_t scratch[kThreads / kWave];
  const int64_t ngroups = n >> 3;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  uint32_t m[G];
#pragma unroll
  for (int i = 0; i < G; ++i) m[i] = 0;
  int64_t g = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if constexpr (NT) {
    // streamed tensor: all but its last keep bytes bypass the caches; that
    // tail, read last, is left in the last-level cache for the encode pass,
    // which starts there
    const int64_t cut = ngroups - keep / (BF16 ? 16 : 32);
    for (; g + (G - 1) * stride < cut; g += G * stride) {
      U8 v[G];
#pragma unroll
      for (int i = 0; i < G; ++i) v[i] = load8<BF16, true>(x, (g + i * stride) * 8);
#pragma unroll
      for (int i = 0; i < G; ++i)
#pragma unroll
        for (int e = 0; e < 8; ++e) m[i] = max(m[i], max_key<MODE>(v[i].v[e]));
    }
  }
  for (; g + (G - 1) * stride < ngroups; g += G * stride) {
    U8 v[G];
#pragma unroll
    for (int i = 0; i < G; ++i) v[i] = load8<BF16, false>(x, (g + i * stride) * 8);
#pragma unroll
    for (int i = 0; i < G; ++i)
#pragma unroll
      for (int e = 0; e < 8; ++e) m[i] = max(m[i], max_key<MODE>(v[i].v[e]));
  }
  for (; g < ngroups; g += stride) {
    const U8 a = load8<BF16>(x, g * 8);
#pragma unroll
    for (int e = 0; e < 8; ++e) m[0] = max(m[0], max_key<MODE>(a.v[e]));
  }
  if (blockIdx.x == 0 && threadIdx.x == 0 && (n & 7)) {
    const U8 a = load8_tail<BF16>(x, ngroups * 8, n);  // missing elements read +0 (key 0)
#pragma unroll
    for (int e = 0; e < 8; ++e) m[0] = max(m[0], max_key<MODE>(a.v[e]));
  }
#pragma unroll
  for (int i = 1; i < G; ++i) m[0] = max(m[0], m[i]);
  const uint32_t r = block_max_u32(m[0], scratch);
  if (threadIdx.x == 0) partial[blockIdx.x] = r;
}

// Folds `nparts` (1 .. 16 * 1024) partial keys into one (one block): each
// thread reads 16 keys with independent loads (indices past the end are
// clamped to the last key, which leaves the maximum unchanged).
__global__ __launch_bounds__(1024) void fold_partials_kernel(const uint32_t* __restrict__ partial, int nparts,
                                                            uint32_t* __restrict__ out) {
  __shared__ uint32_t scratch[1024 / kWave];
  const int i0 = threadIdx.x;
  uint32_t v[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) v[k] = partial[min(i0 + k * 1024, nparts - 1)];
  uint32_t m = 0;
#pragma unroll
  for (int k = 0; k < 16; ++k) m = max(m, v[k]);
  m = block_max_u32(m, scratch);
  if (threadIdx.x == 0) *out = m;
}

// ---------------------------- transposing tiles ----------------------------
//
// When the transposed code layout is requested, work goes by tiles of
// TW = 2^lt code words: TG = 2^lg column groups (8 columns each) by
// TR = TW / TG rows.  TG is 32, or the next power of two above the number of
// column groups for narrow matrices; TW is 4096 (LUQ) or 8192 (INT4), or
// smaller (down to 1024) when that leaves too few tiles to fill the chip.
//   Phase A: consecutive lanes take consecutive column groups of a row, so
//            the loads and the row-major code stores of a row are contiguous;
//            every 8-element code word also goes to LDS at [group][row].
//   Phase B: consecutive lanes take consecutive 8-row blocks of one column
//            group, read the block's 8 words (two 16-byte LDS reads),
//            transpose them in registers and store one word per column, so
//            consecutive lanes write consecutive words of a transposed row.
// Largest tiles (words): the LUQ encoder is ALU-bound and prefers more,
// smaller tiles in flight; the INT4 encoder is bound by memory and prefers
// longer contiguous stores.
constexpr int kLuqTileLg = 12, kInt4TileLg = 13;
constexpr int kTilePad = 4;  // LDS words between column groups (keeps 16-byte alignment)

//
// SUM (two SMP samples stored as one int8 per element): the two code words
// of an item become 8 bytes of sums (elements 0..3 in the first word), which
// take the places of the two planes in LDS; phase B transposes 4x4 byte
// blocks and stores 8 bytes (8 rows) per column.
template <int NS, typename Enc, bool SUM = false>
__device__ __forceinline__ void encode_tiles(const Enc& enc, int64_t rows, int64_t cols, int lg,
                                             int lt, uint8_t* codes, uint8_t* codes_t,
                                             int64_t plane, uint32_t* lds, uint32_t& mx) {
  static_assert(!SUM || NS == 2, "the summed operand takes two samples");
  const int tw = 1 << lt, tg = 1 << lg, tr = tw >> lg, pitch = tr + kTilePad;
  const int64_t cgs = cols >> 3;
  const int64_t ntr = (rows + tr - 1) / tr, ntc = (cgs + tg - 1) / tg;
  for (int64_t k = blockIdx.x; k < ntr * ntc; k += gridDim.x) {
    const int64_t t = Enc::kNT ? ntr * ntc - 1 - k : k;  // a streamed tensor is walked from its end
    const int64_t r0 = (t / ntc) * tr, g0 = (t % ntc) * tg;
    if constexpr (Enc::kPipeline) {
      // two items per trip (tw is a multiple of 2 * kThreads, so the trip count
      // is even): the next trip's loads are issued before this trip's items are
      // encoded, so one trip's encode hides the next one's memory latency.  The
      // fetch after the last trip re-reads the first one (in bounds, ignored):
      // every trip issues the same loads and the wait counts stay static.
      constexpr int U = 2;
      const int ntrips = tw / (U * kThreads);
      struct Trip {
        int g[U], r[U];
        bool ok[U];
        int64_t e0[U];
        U8 v[U];
      };
      auto fetch = [&](Trip& T, int trip) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int q = threadIdx.x + (trip * U + u) * kThreads;
          T.g[u] = q & (tg - 1);
          T.r[u] = q >> lg;
          const int64_t row = r0 + T.r[u], cg = g0 + T.g[u];
          T.ok[u] = row < rows && cg < cgs;
          T.e0[u] = row * cols + cg * 8;
          T.v[u] = enc.load(T.ok[u] ? T.e0[u] : 0);  // no branch: an item off the tensor reads element 0
        }
      };
      auto encode = [&](const Trip& T) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
          if constexpr (Enc::kTrack) {
            if (T.ok[u]) mx = max(mx, max_key8(T.v[u]));
          }
          uint32_t w[NS];
#pragma unroll
          for (int s = 0; s < NS; ++s) w[s] = 0;
          if (T.ok[u]) {
#pragma unroll
            for (int s = 0; s < NS; ++s) w[s] = enc.word(T.v[u], (uint64_t)(T.e0[u] >> 3), s);
            if constexpr (SUM) {
              uint32_t lo, hi;
              smp_sum_bytes(w[0], w[1], lo, hi);
              w[0] = lo;
              w[1] = hi;
              if (codes) store_word2<Enc::kNTStore>(codes + T.e0[u], lo, hi);
            } else {
#pragma unroll
              for (int s = 0; s < NS; ++s)
                if (codes) store_word<Enc::kNTStore>(codes + s * plane + (T.e0[u] >> 1), w[s]);
            }
          }
#pragma unroll
          for (int s = 0; s < NS; ++s) lds[(s * tg + T.g[u]) * pitch + T.r[u]] = w[s];
        }
      };
      Trip ta, tb;
      fetch(ta, 0);
      for (int trip = 0; trip < ntrips; trip += 2) {
        fetch(tb, trip + 1);
        encode(ta);
        fetch(ta, trip + 2 < ntrips ? trip + 2 : 0);
        encode(tb);
      }
    } else {
      // two items per trip (tw is a multiple of 2 * kThreads): both loads are
      // in flight before either is encoded
      constexpr int U = 2;
      for (int q0 = threadIdx.x; q0 < tw; q0 += U * kThreads) {
        int g[U], r[U];
        bool ok[U];
        int64_t e0[U];
        U8 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int q = q0 + u * kThreads;
          g[u] = q & (tg - 1);
          r[u] = q >> lg;
          const int64_t row = r0 + r[u], cg = g0 + g[u];
          ok[u] = row < rows && cg < cgs;
          e0[u] = row * cols + cg * 8;
          if (ok[u]) {
            v[u] = enc.load(e0[u]);
            if constexpr (Enc::kTrack) mx = max(mx, max_key8(v[u]));
          }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          uint32_t w[NS];
#pragma unroll
          for (int s = 0; s < NS; ++s) w[s] = 0;
          if (ok[u]) {
#pragma unroll
            for (int s = 0; s < NS; ++s) w[s] = enc.word(v[u], (uint64_t)(e0[u] >> 3), s);
            if constexpr (SUM) {
              uint32_t lo, hi;
              smp_sum_bytes(w[0], w[1], lo, hi);
              w[0] = lo;
              w[1] = hi;
              if (codes) store_word2<Enc::kNTStore>(codes + e0[u], lo, hi);
            } else {
#pragma unroll
              for (int s = 0; s < NS; ++s)
                if (codes) store_word<Enc::kNTStore>(codes + s * plane + (e0[u] >> 1), w[s]);
            }
          }
#pragma unroll
          for (int s = 0; s < NS; ++s) lds[(s * tg + g[u]) * pitch + r[u]] = w[s];
        }
      }
    }
    __syncthreads();
    const int rbs = tr >> 3;  // 8-row blocks per tile
    for (int q = threadIdx.x; q < (tw >> 3); q += kThreads) {
      const int rb = q & (rbs - 1), g = q / rbs;
      const int64_t row0 = r0 + rb * 8, cg = g0 + g;
      if (row0 >= rows || cg >= cgs) continue;
      if constexpr (SUM) {
        // lds plane 0: bytes of columns 0..3 of each row, plane 1: columns 4..7
        uint8_t* dst = codes_t + (cg * 8) * rows + row0;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const uint4* src = reinterpret_cast<const uint4*>(lds + (h * tg + g) * pitch + rb * 8);
          const uint4 a = src[0], b = src[1];
          const uint32_t ra[4] = {a.x, a.y, a.z, a.w}, rb4[4] = {b.x, b.y, b.z, b.w};
          uint32_t ca[4], cb[4];
          transpose4x4_bytes(ra, ca);   // rows 0..3
          transpose4x4_bytes(rb4, cb);  // rows 4..7
#pragma unroll
          for (int c = 0; c < 4; ++c) store_word2<Enc::kNTStore>(dst + (h * 4 + c) * rows, ca[c], cb[c]);
        }
        continue;
      }
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const uint4* src = reinterpret_cast<const uint4*>(lds + (s * tg + g) * pitch + rb * 8);
        const uint4 lo = src[0], hi = src[1];
        uint32_t w8[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
        transpose8x8_nibbles(w8);
        uint8_t* dst = codes_t + s * plane + (cg * 8) * (rows >> 1) + (row0 >> 1);
#pragma unroll
        for (int c = 0; c < 8; ++c) store_word<Enc::kNTStore>(dst + c * (rows >> 1), w8[c]);
      }
    }
    __syncthreads();
  }
}

// ------------------------------- LUQ ---------------------------------------

struct LuqParams {
  float alpha_s;     // alpha * S
  float S;           // 1 or 2^100
  uint32_t a1_bits;  // bits of alpha_s / 2
  uint32_t w16_bits;  // bits of alpha_s * 2^-17
  uint32_t top_field;
  bool zero;  // every code is 0 (alpha == 0, or non-finite input)
};

// Power-of-two alpha (Appendix, power-of-two LUQ): 2^(ceil(log2 m) - R) for
// a finite m > 0, from the bits of m: the exponent of a normal m, or the
// position of the top mantissa bit of a subnormal one, plus one unless m is
// a power of two.  Below the float32 subnormal range it is 0 (half the
// smallest subnormal rounds to 0 as well).
__device__ __forceinline__ float pw2_alpha(uint32_t mbits, int R) {
  if (mbits == 0) return 0.0f;
  const uint32_t e = mbits >> 23, mant = mbits & 0x7FFFFFu;
  const int c = e ? (int)e - 127 + (mant != 0) : (31 - __clz((int)mant)) - 149 + ((mant & (mant - 1)) != 0);
  const int k = c - R;
  if (k >= -126) return __uint_as_float((uint32_t)(k + 127) << 23);
  return k >= -149 ? __uint_as_float(1u << (k + 149)) : 0.0f;
}

// Eq. alpha: alpha = fl32(m * 2^-R), or with pw2 the power-of-two alpha.
// `alpha_out` gets the unscaled alpha.  alpha_s * 2^-17 is a normal float
// (alpha_s >= 2^-96 unscaled, and tiny maxima are scaled by 2^100).
__device__ __forceinline__ LuqParams luq_params(uint32_t mbits, int R, bool pw2, float* alpha_out) {
  LuqParams p;
  const float m = __uint_as_float(mbits);
  float alpha;
  if (mbits >= 0x7F800000u) {
    alpha = __uint_as_float(0x7FC00000u);  // NaN
    p.zero = true;
  } else {
    alpha = pw2 ? pw2_alpha(mbits, R)
                : m * __uint_as_float((uint32_t)(127 - R) << 23);  // exact 2^-R scale, one rounding
    p.zero = (alpha == 0.0f);
  }
  *alpha_out = alpha;
  p.S = (m < 0x1p-90f) ? 0x1p100f : 1.0f;
  p.alpha_s = alpha * p.S;
  p.a1_bits = __float_as_uint(p.alpha_s * 0.5f);
  p.w16_bits = __float_as_uint(p.alpha_s * 0x1p-17f);
  p.top_field = (uint32_t)R + 1;
  return p;
}

// Sign bits of 8 words at the sign position of their nibbles (bit 4e+3):
// the top bytes of the odd words are gathered as they are (bit 7 of byte k
// is word 2k+1's sign), those of the even words are gathered and rotated
// right by 4 bits.  Other bits are garbage and masked by the caller.
__device__ __forceinline__ uint32_t gather_signs(const U8& v) {
  const uint32_t odd = __builtin_amdgcn_perm(v.v[3], v.v[1], 0x0C0C0703u) |
                       __builtin_amdgcn_perm(v.v[7], v.v[5], 0x07030C0Cu);
  const uint32_t even = __builtin_amdgcn_perm(v.v[2], v.v[0], 0x0C0C0703u) |
                        __builtin_amdgcn_perm(v.v[6], v.v[4], 0x07030C0Cu);
  return (odd & 0x80808080u) | (__builtin_amdgcn_alignbit(even, even, 4) & 0x08080808u);
}

// [n >= 1] in one instruction (the compiler would otherwise emit a compare
// and a select).
__device__ __forceinline__ uint32_t med3_01(int32_t n) {
  uint32_t r;
  asm("v_med3_i32 %0, %1, 0, 1" : "=v"(r) : "v"(n));
  return r;
}

// Codes of 8 consecutive elements (bits in v) for Philox block `blk`.
//
// Per element, on the magnitude a (scaled by S when SCALED; both a and alpha
// normal once a >= alpha): the difference of the float bit patterns
// bits(a) - bits(alpha / 2), shifted right by 23, is n1 = n + 1 with
// n = floor(log2(a / alpha)) -- the exponent difference, less one when the
// mantissa of a is below that of alpha (the borrow).  n1 <= 0 is the
// underflow bin [0, alpha) (lower level 0), n1 >= 1 the bin
// [alpha 2^n, alpha 2^(n+1)) (lower level = width = alpha 2^n), and the base
// field is max(n1, 0).  With w16 = width * 2^-16 (alpha * 2^-17 with
// max(n1, 1) added to its exponent) and jj = j + 2^16 [n1 >= 1], the exact
// value jj * w16 - a equals (j * w - d * 2^16) * 2^-16 for the offset d of a
// above the lower level; the fused multiply-add rounds it once, so its sign
// is that of j * w - d * 2^16 and the value rounds up exactly when the sign
// bit is set (a zero result is +0: no round-up).  The round-up bits are
// gathered from the sign bits and added to the packed base fields.
//
// Unscaled, a <= max <= alpha * 2^R (equal for the plain alpha, which is
// exact there), so n1 <= R + 1 and at n1 = R + 1 the offset is 0: the field
// never exceeds R + 1.  Scaled, alpha may have been rounded (subnormal alpha), and
// with an estimated maximum (CAP) magnitudes, Inf and NaN may lie above the
// top level: there the base field is clamped to R + 1 and the round-up bit
// of top-level elements is dropped (the top code, with the element's sign).
// Each sign bit is then set where the field is non-zero (zero is always +0).
template <bool SCALED, bool CAP = false>
__device__ __forceinline__ uint32_t luq_word(const U8& v, uint64_t blk, uint32_t sample,
                                             uint32_t counter, uint32_t k0, uint32_t k1,
                                             const LuqParams& p) {
  constexpr bool kClamp = SCALED || CAP;
  const U4 y = philox4x32_10(U4{(uint32_t)blk, (uint32_t)(blk >> 32), sample, counter}, k0, k1);
  const uint32_t w[4] = {y.x, y.y, y.z, y.w};
  uint32_t base = 0;
  U8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint32_t ab = SCALED ? __float_as_uint(fabsf(__uint_as_float(v.v[e])) * p.S) : (v.v[e] & 0x7FFFFFFFu);
    const int32_t n1 = ((int32_t)ab - (int32_t)p.a1_bits) >> 23;
    const int32_t f0 = kClamp ? min(max(n1, 0), (int32_t)p.top_field) : max(n1, 0);
    const uint32_t ge = med3_01(n1);
    const float w16 = __uint_as_float(p.w16_bits + ((uint32_t)max(n1, 1) << 23));
    const uint32_t jj = (e & 1) ? __builtin_amdgcn_alignbit(ge, w[e >> 1], 16)
                                : __builtin_amdgcn_perm(ge, w[e >> 1], 0x05040100u);
    r.v[e] = __float_as_uint(fmaf((float)jj, w16, -__uint_as_float(ab)));
    base |= (uint32_t)f0 << (4 * e);
  }
  uint32_t up = (gather_signs(r) >> 3) & 0x11111111u;
  if constexpr (kClamp) {
    const uint32_t t = base ^ (0x11111111u * p.top_field);
    up &= (t | (t >> 1) | (t >> 2));  // bit 4e set unless field e is the top one
  }
  const uint32_t fields = base + up;
  const uint32_t nz = (fields | (fields >> 1) | (fields >> 2)) & 0x11111111u;
  return fields | (gather_signs(v) & (nz << 3));
}

typedef short s16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ s16x2 as_s16x2(uint32_t x) { return __builtin_bit_cast(s16x2, x); }
__device__ __forceinline__ uint32_t as_u32(s16x2 x) { return __builtin_bit_cast(uint32_t, x); }

// luq_word for bf16 input on the unscaled path (alpha >= 2^-96, so alpha and
// alpha/2 have zero low halves, as every bf16 magnitude does): the same codes,
// with the bin index, base field, [n1 >= 1] and max(n1, 1) computed for two
// elements at once with 16-bit packed integer operations.  Elements are
// paired (i, i+4), so a pair's base fields land in nibbles i and i+4 with one
// shift-or, and the 16-bit bin index equals the 32-bit one:
// ((a - a1) << 16) >> 23 = (a - a1) >> 7 for 16-bit a, a1 (|a - a1| < 2^15).
// The rounding decision per element is luq_word's fused multiply-add.  CAP
// (an estimated maximum) clamps the base fields to the top one and drops the
// round-up there, as luq_word does; the bin widths of elements above the top
// level are then garbage, but their round-up bits are the dropped ones.
template <bool CAP = false>
__device__ __forceinline__ uint32_t luq_word_bf16(const U8& v, uint64_t blk, uint32_t sample, uint32_t counter,
                                                  uint32_t k0, uint32_t k1, const LuqParams& p) {
  const U4 y = philox4x32_10(U4{(uint32_t)blk, (uint32_t)(blk >> 32), sample, counter}, k0, k1);
  const uint32_t w[4] = {y.x, y.y, y.z, y.w};
  // the loaded bf16 words: elements 2i (low half) and 2i+1 (high half)
  uint32_t q[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) q[i] = (v.v[2 * i] >> 16) | (v.v[2 * i + 1] & 0xFFFF0000u);
  const s16x2 a1 = as_s16x2((p.a1_bits >> 16) * 0x10001u);
  const s16x2 top = as_s16x2(p.top_field * 0x10001u);
  uint32_t base = 0, sg = 0;
  U8 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    // pair i: element i in the low half, element i + 4 in the high half
    const uint32_t pr = __builtin_amdgcn_perm(q[2 + (i >> 1)], q[i >> 1], (i & 1) ? 0x07060302u : 0x05040100u);
    sg |= ((pr >> 12) & 0x00080008u) << (4 * i);    // signs of elements i, i+4 at bits 4i+3, 4i+19
    const uint32_t pm = pr & 0x7FFF7FFFu;
    const s16x2 n1 = (as_s16x2(pm) - a1) >> 7;
    s16x2 f0 = __builtin_elementwise_max(n1, (s16x2){0, 0});
    if constexpr (CAP) f0 = __builtin_elementwise_min(f0, top);
    uint32_t ge;  // [n1 >= 1] per half, one packed min (the compiler would compare and select)
    asm("v_pk_min_i16 %0, %1, %2" : "=v"(ge) : "v"(as_u32(f0)), "s"(0x00010001u));
    const uint32_t m1 = as_u32(__builtin_elementwise_max(n1, (s16x2){1, 1}));
    base |= as_u32(f0) << (4 * i);                  // fields <= R + 1 <= 7: nibbles i and i + 4
    const float w16_lo = __uint_as_float(p.w16_bits + (m1 << 23));
    const float w16_hi = __uint_as_float(p.w16_bits + (__builtin_amdgcn_ubfe(m1, 16, 3) << 23));
    // jj = j + 2^16 [n1 >= 1]: j of element e is half e & 1 of word e >> 1
    const uint32_t jj_lo = __builtin_amdgcn_perm(ge, w[i >> 1], (i & 1) ? 0x0C040302u : 0x0C040100u);
    const uint32_t jj_hi = __builtin_amdgcn_perm(ge, w[2 + (i >> 1)], (i & 1) ? 0x0C060302u : 0x0C060100u);
    r.v[i] = __float_as_uint(fmaf((float)jj_lo, w16_lo, -__uint_as_float(pm << 16)));
    r.v[i + 4] = __float_as_uint(fmaf((float)jj_hi, w16_hi, -__uint_as_float(pm & 0xFFFF0000u)));
  }
  uint32_t up = (gather_signs(r) >> 3) & 0x11111111u;
  if constexpr (CAP) {
    const uint32_t t = base ^ (0x11111111u * p.top_field);
    up &= (t | (t >> 1) | (t >> 2));  // bit 4e set unless field e is the top one
  }
  const uint32_t fields = base + up;
  const uint32_t nz = (fields | (fields >> 1) | (fields >> 2)) & 0x11111111u;
  return fields | (sg & (nz << 3));
}

struct LuqArgs {
  const void* g;
  int64_t rows, cols, n;
  int R;
  bool pw2;  // power-of-two alpha
  uint32_t k0, k1, counter;
  const uint32_t* partial;
  int nparts;
  uint8_t* codes;
  uint8_t* codes_t;
  int64_t plane;
  float* alpha_out;
  float* max_out;
  // in-hindsight mode: the estimate read at the start, and one partial
  // maximum per encode block written at the end
  const float* state;
  uint32_t* part_out;
  uint32_t* status;  // status word, or null
};

// Key of the in-hindsight estimate: NaN stays NaN, anything not positive is 0.
__device__ __forceinline__ uint32_t estimate_key(float m) {
  return m != m ? 0x7FC00000u : (m > 0.0f ? __float_as_uint(m) : 0u);
}

// HS (in-hindsight): alpha comes from the estimate; the fold kernel that
// runs after the encode writes alpha and the measured maximum.
template <bool HS = false>
__device__ __forceinline__ LuqParams luq_block_params(const LuqArgs& a) {
  __shared__ uint32_t scratch[kThreads / kWave];
  const uint32_t mbits = HS ? estimate_key(*a.state) : reduce_partials(a.partial, a.nparts, scratch);
  float alpha;
  const LuqParams p = luq_params(mbits, a.R, a.pw2, &alpha);
  if (!HS && blockIdx.x == 0 && threadIdx.x == 0) {
    *a.alpha_out = alpha;
    if (a.max_out) *a.max_out = __uint_as_float(mbits);
    if (a.status) *a.status = kStatusTag | (mbits >= 0x7F800000u ? kStatusNonfinite : 0u);
  }
  return p;
}

// Codes of group g (elements 8g .. 8g+7): one word per sample plane, or with
// SUM the 8 int8 sums of the two samples.
// The code word of 8 elements: the bf16-specialised encoder on the common
// (unscaled, exact-maximum) bf16 path, luq_word otherwise.
template <bool BF16, bool SCALED, bool HS>
__device__ __forceinline__ uint32_t luq_code_word(const U8& v, uint64_t blk, uint32_t sample, const LuqArgs& a,
                                                  const LuqParams& p) {
  if constexpr (BF16 && !SCALED) return luq_word_bf16<HS>(v, blk, sample, a.counter, a.k0, a.k1, p);
  return luq_word<SCALED, HS>(v, blk, sample, a.counter, a.k0, a.k1, p);
}

template <bool BF16, bool NT, int NS, bool SUM, bool SCALED, bool HS>
__device__ __forceinline__ void luq_emit_group(const LuqArgs& a, const LuqParams& p, const U8& v, int64_t g) {
  if constexpr (SUM) {
    uint32_t lo, hi;
    smp_sum_bytes(luq_code_word<BF16, SCALED, HS>(v, (uint64_t)g, 0, a, p),
                  luq_code_word<BF16, SCALED, HS>(v, (uint64_t)g, 1, a, p), lo, hi);
    store_word2<NT>(a.codes + g * 8, lo, hi);
  } else {
#pragma unroll
    for (int s = 0; s < NS; ++s)
      store_word<NT>(a.codes + s * a.plane + g * 4, luq_code_word<BF16, SCALED, HS>(v, (uint64_t)g, s, a, p));
  }
}

// Flat row-major codes; groups of 8 elements along the flattened tensor.
// With HS the fields are capped and the thread's max key is returned.
template <bool BF16, bool NT, int NS, bool SCALED, bool HS = false, bool SUM = false>
__device__ __forceinline__ uint32_t luq_flat_body(const LuqArgs& a, const LuqParams& p) {
  uint32_t mx = 0;
  const int64_t nfull = a.n >> 3;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  // step k of the walk takes group k, or with NT (streamed tensor) group
  // nfull - 1 - k: the walk starts at the end of the tensor
  const auto at = [&](int64_t k) { return NT ? nfull - 1 - k : k; };
  int64_t g = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  // four groups per trip (then two): every load of a trip is in flight before
  // any of its groups is encoded
  for (; g + 3 * stride < nfull; g += 4 * stride) {
    U8 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = load8<BF16, NT>(a.g, at(g + u * stride) * 8);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (HS) mx = max(mx, max_key8(v[u]));
      luq_emit_group<BF16, NT, NS, SUM, SCALED, HS>(a, p, v[u], at(g + u * stride));
    }
  }
  for (; g + stride < nfull; g += 2 * stride) {
    const U8 v0 = load8<BF16, NT>(a.g, at(g) * 8);
    const U8 v1 = load8<BF16, NT>(a.g, at(g + stride) * 8);
    if (HS) mx = max(mx, max(max_key8(v0), max_key8(v1)));
    luq_emit_group<BF16, NT, NS, SUM, SCALED, HS>(a, p, v0, at(g));
    luq_emit_group<BF16, NT, NS, SUM, SCALED, HS>(a, p, v1, at(g + stride));
  }
  if (g < nfull) {
    const U8 v = load8<BF16, NT>(a.g, at(g) * 8);
    if (HS) mx = max(mx, max_key8(v));
    luq_emit_group<BF16, NT, NS, SUM, SCALED, HS>(a, p, v, at(g));
  }
  if ((a.n & 7) && blockIdx.x == 0 && threadIdx.x == 0) {
    const U8 v = load8_tail<BF16>(a.g, nfull * 8, a.n);  // missing elements read +0
    if (HS) mx = max(mx, max_key8(v));
    const int tail = (int)(a.n & 7);
    if constexpr (SUM) {
      uint32_t lo, hi;
      smp_sum_bytes(luq_word<SCALED, HS>(v, (uint64_t)nfull, 0, a.counter, a.k0, a.k1, p),
                    luq_word<SCALED, HS>(v, (uint64_t)nfull, 1, a.counter, a.k0, a.k1, p), lo, hi);
      store_bytes(a.codes + nfull * 8, lo, min(tail, 4));
      store_bytes(a.codes + nfull * 8 + 4, hi, max(tail - 4, 0));
    } else {
#pragma unroll
      for (int s = 0; s < NS; ++s)
        store_bytes(a.codes + s * a.plane + nfull * 4,
                    luq_word<SCALED, HS>(v, (uint64_t)nfull, s, a.counter, a.k0, a.k1, p), (tail + 1) >> 1);
    }
  }
  return mx;
}

// Max key over the groups a flat-encode thread owns (in-hindsight mode with
// all codes 0: the measurement still covers the whole tensor).
template <bool BF16, bool NT>
__device__ __forceinline__ uint32_t flat_max_only(const LuqArgs& a) {
  uint32_t mx = 0;
  const int64_t nfull = a.n >> 3;
  for (int64_t g = (int64_t)blockIdx.x * kThreads + threadIdx.x; g < nfull; g += (int64_t)gridDim.x * kThreads)
    mx = max(mx, max_key8(load8<BF16, NT>(a.g, g * 8)));
  if ((a.n & 7) && blockIdx.x == 0 && threadIdx.x == 0) mx = max(mx, max_key8(load8_tail<BF16>(a.g, nfull * 8, a.n)));
  return mx;
}

// One partial maximum per block (in-hindsight mode).
__device__ __forceinline__ void write_block_max(uint32_t mx, uint32_t* part_out) {
  __shared__ uint32_t scratch[kThreads / kWave];
  const uint32_t m = block_max_u32(mx, scratch);
  if (threadIdx.x == 0) part_out[blockIdx.x] = m;
}

template <bool BF16, bool NT, int NS, bool HS = false, bool SUM = false>
__global__ __launch_bounds__(kThreads) void luq_encode_flat_kernel(LuqArgs a) {
  const LuqParams p = luq_block_params<HS>(a);
  if (p.zero) {  // alpha is 0 or NaN: every code (or sum) is 0
    const int64_t nbytes = SUM ? a.n : (a.n + 1) >> 1;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < nbytes; i += (int64_t)gridDim.x * kThreads)
      for (int s = 0; s < (SUM ? 1 : NS); ++s) a.codes[s * a.plane + i] = 0;
    if (HS) write_block_max(flat_max_only<BF16, NT>(a), a.part_out);
    return;
  }
  const uint32_t mx = p.S != 1.0f ? luq_flat_body<BF16, NT, NS, true, HS, SUM>(a, p)
                                  : luq_flat_body<BF16, NT, NS, false, HS, SUM>(a, p);
  if (HS) write_block_max(mx, a.part_out);
}

template <bool BF16, bool NT, bool SCALED, bool HS = false>
struct LuqEnc {
  static constexpr bool kTrack = HS;
  static constexpr bool kPipeline = true;  // ALU-heavy words: overlap the next loads with them
  static constexpr bool kNT = NT;
  static constexpr bool kNTStore = NT;
  const LuqArgs* a;
  const LuqParams* p;
  __device__ U8 load(int64_t e0) const { return load8<BF16, NT>(a->g, e0); }
  __device__ uint32_t word(const U8& v, uint64_t blk, int s) const {
    return p->zero ? 0u : luq_code_word<BF16, SCALED, HS>(v, blk, s, *a, *p);
  }
};

template <bool BF16, bool NT, int NS, bool HS = false, bool SUM = false>
__global__ __launch_bounds__(kThreads) void luq_encode_tile_kernel(LuqArgs a, int lg, int lt) {
  __shared__ __attribute__((aligned(16))) uint32_t lds[NS * ((1 << kLuqTileLg) + 32 * kTilePad)];
  const LuqParams p = luq_block_params<HS>(a);
  uint32_t mx = 0;
  if (p.S != 1.0f)
    encode_tiles<NS, LuqEnc<BF16, NT, true, HS>, SUM>(LuqEnc<BF16, NT, true, HS>{&a, &p}, a.rows, a.cols, lg, lt,
                                                      a.codes, a.codes_t, a.plane, lds, mx);
  else
    encode_tiles<NS, LuqEnc<BF16, NT, false, HS>, SUM>(LuqEnc<BF16, NT, false, HS>{&a, &p}, a.rows, a.cols, lg, lt,
                                                       a.codes, a.codes_t, a.plane, lds, mx);
  if (HS) write_block_max(mx, a.part_out);
}

// In-hindsight fold, after the encode: the measured maximum (from the encode
// blocks' partials), alpha of this step (from the estimate the encode read)
// and the next estimate, Eq. hindsight: m' = fl32(fl32(c1 max) + fl32(c0 m))
// with c1 = fl32(1 - eta), c0 = eta.  A step whose measured maximum is not
// finite (an overflowed gradient) leaves the estimate as it was, so that one
// such step does not make every later alpha NaN; it reports
// LUQ_ERR_NONFINITE, as does a non-finite estimate.
__global__ __launch_bounds__(1024) void hindsight_fold_kernel(const uint32_t* __restrict__ part, int nparts,
                                                             float* state, float c1, float c0, int R,
                                                             bool pw2, float* alpha_out, float* maxabs_out,
                                                             uint32_t* status) {
  __shared__ uint32_t scratch[1024 / kWave];
  const uint32_t m = reduce_partials(part, nparts, scratch);
  if (threadIdx.x == 0) {
    const uint32_t mkey = estimate_key(*state);
    float alpha;
    (void)luq_params(mkey, R, pw2, &alpha);
    const float mx = __uint_as_float(m);
    *alpha_out = alpha;
    if (maxabs_out) *maxabs_out = mx;
    const bool measured_ok = m < 0x7F800000u;
    if (measured_ok) *state = __fadd_rn(__fmul_rn(c1, mx), __fmul_rn(c0, __uint_as_float(mkey)));
    if (status) *status = kStatusTag | (measured_ok && mkey < 0x7F800000u ? 0u : kStatusNonfinite);
  }
}

// Empty tensors: the scalar outputs and the status word (when given).
__global__ void write_two_floats_kernel(float* a, float va, float* b, float vb, uint32_t* status) {
  if (a) *a = va;
  if (b) *b = vb;
  if (status) *status = kStatusTag;
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
  uint32_t* status;  // status word, or null
};

// Scale and rounding parameters from the range: clip when positive, else the
// max key mbits of the tensor (Section 3.3, Appendix A.1).
__device__ __forceinline__ Int4Params int4_params(const Int4Args& a, uint32_t mbits) {
  Int4Params p;
  const float Q = a.is_signed ? 7.0f : 15.0f;
  float m, s;
  bool nonfinite = false;
  if (a.clip > 0.0f) {
    m = a.clip;
  } else {
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
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    *a.scale_out = s;
    if (a.status) *a.status = kStatusTag | (nonfinite ? kStatusNonfinite : 0u);
  }
  return p;
}

__device__ __forceinline__ Int4Params int4_block_params(const Int4Args& a) {
  __shared__ uint32_t scratch[kThreads / kWave];
  return int4_params(a, a.clip > 0.0f ? 0u : reduce_partials(a.partial, a.nparts, scratch));
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

template <bool BF16, bool NT>
__global__ __launch_bounds__(kThreads) void int4_encode_flat_kernel(Int4Args a) {
  const Int4Params p = int4_block_params(a);
  const int64_t ngroups = (a.n + 7) >> 3;
  for (int64_t k = (int64_t)blockIdx.x * kThreads + threadIdx.x; k < ngroups;
       k += (int64_t)gridDim.x * kThreads) {
    const int64_t g = NT ? ngroups - 1 - k : k;  // a streamed tensor is walked from its end
    const bool full = (g * 8 + 8) <= a.n;
    const U8 v = full ? load8<BF16, NT>(a.x, g * 8) : load8_tail<BF16>(a.x, g * 8, a.n);
    const uint32_t word = p.zero ? 0u : int4_word(v, p);
    if (full)
      store_word<false>(a.codes + g * 4, word);
    else
      store_bytes(a.codes + g * 4, word, (int)((a.n - g * 8 + 1) >> 1));
  }
}

template <bool BF16, bool NT>
struct Int4Enc {
  static constexpr bool kTrack = false;
  static constexpr bool kPipeline = false;  // memory-bound: the plain trips measure faster
  static constexpr bool kNT = NT;
  // the GEMM that follows reads the INT4 codes: keep them in the cache even
  // when the tensor itself is streamed
  static constexpr bool kNTStore = false;
  const Int4Args* a;
  const Int4Params* p;
  __device__ U8 load(int64_t e0) const { return load8<BF16, NT>(a->x, e0); }
  __device__ uint32_t word(const U8& v, uint64_t, int) const { return p->zero ? 0u : int4_word(v, *p); }
};

template <bool BF16, bool NT>
__global__ __launch_bounds__(kThreads) void int4_encode_tile_kernel(Int4Args a, int lg, int lt) {
  __shared__ __attribute__((aligned(16))) uint32_t lds[(1 << kInt4TileLg) + 32 * kTilePad];
  const Int4Params p = int4_block_params(a);
  uint32_t unused = 0;
  encode_tiles<1>(Int4Enc<BF16, NT>{&a, &p}, a.rows, a.cols, lg, lt, a.codes, a.codes_t, 0, lds, unused);
}

// Small tensors (up to kInt4SmallN elements, such as a convolution's weight):
// one launch instead of two.  Each of a few workgroups takes the maximum of
// the whole tensor itself (it is small and stays in L2 after the first
// read), with eight 8-element groups in flight per thread, and then encodes
// its share of the tiles or groups.
constexpr int64_t kInt4SmallN = 1 << 16;
constexpr int kInt4SmallBlocks = 16;

template <bool BF16, int MODE>
__global__ __launch_bounds__(kThreads) void int4_small_kernel(Int4Args a, int lg, int lt) {
  __shared__ uint32_t scratch[kThreads / kWave];
  __shared__ __attribute__((aligned(16))) uint32_t lds[(1 << kInt4TileLg) + 32 * kTilePad];
  uint32_t m = 0;
  if (a.clip <= 0.0f) {
    constexpr int U = 8;
    const int64_t ngroups = a.n >> 3;
    int64_t g = threadIdx.x;
    for (; g + (U - 1) * kThreads < ngroups; g += U * kThreads) {
      U8 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = load8<BF16>(a.x, (g + u * kThreads) * 8);
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < 8; ++e) m = max(m, max_key<MODE>(v[u].v[e]));
    }
    for (; g < ngroups; g += kThreads) {
      const U8 v = load8<BF16>(a.x, g * 8);
#pragma unroll
      for (int e = 0; e < 8; ++e) m = max(m, max_key<MODE>(v.v[e]));
    }
    if (threadIdx.x == 0 && (a.n & 7)) {
      const U8 v = load8_tail<BF16>(a.x, ngroups * 8, a.n);  // missing elements read +0 (key 0)
#pragma unroll
      for (int e = 0; e < 8; ++e) m = max(m, max_key<MODE>(v.v[e]));
    }
    m = block_max_u32(m, scratch);
  }
  const Int4Params p = int4_params(a, m);
  if (a.codes_t) {
    uint32_t unused = 0;
    encode_tiles<1>(Int4Enc<BF16, false>{&a, &p}, a.rows, a.cols, lg, lt, a.codes, a.codes_t, 0, lds, unused);
    return;
  }
  const int64_t ngroups = (a.n + 7) >> 3;
  for (int64_t g = (int64_t)blockIdx.x * kThreads + threadIdx.x; g < ngroups; g += (int64_t)gridDim.x * kThreads) {
    const bool full = (g * 8 + 8) <= a.n;
    const U8 v = full ? load8<BF16>(a.x, g * 8) : load8_tail<BF16>(a.x, g * 8, a.n);
    const uint32_t word = p.zero ? 0u : int4_word(v, p);
    if (full)
      store_word<false>(a.codes + g * 4, word);
    else
      store_bytes(a.codes + g * 4, word, (int)((a.n - g * 8 + 1) >> 1));
  }
}

// ------------------------------- launchers ---------------------------------

// Every encode block folds the partials it is given before it starts, so
// while they are given directly their count is kept proportional to the
// tensor (at least 16 groups of 8 elements per max-pass thread); large
// tensors get up to kMaxPartials blocks (8 groups per thread) and one fold.
static int max_pass_blocks(int64_t n) {
  const int64_t groups = (n + 7) >> 3;
  int64_t b = (groups + kThreads * 16 - 1) / (kThreads * 16);
  if (b > kDirectPartials) b = (groups + kThreads * 8 - 1) / (kThreads * 8);
  if (b < 1) b = 1;
  if (b > kMaxPartials) b = kMaxPartials;
  return (int)b;
}

// partials, their fold and the status word
size_t quant_workspace_bytes(int64_t /*n*/) { return (kStatusWord + 1) * sizeof(uint32_t); }

size_t quant_status_offset() { return kStatusWord * sizeof(uint32_t); }

static int encode_blocks_flat(int64_t n) {
  const int64_t groups = (n + 7) >> 3;
  int64_t b = (groups + kThreads - 1) / kThreads;
  if (b < 1) b = 1;
  if (b > kMaxEncodeBlocks) b = kMaxEncodeBlocks;
  return (int)b;
}

// Transposing tile shape: log2 of the column groups per tile (lg) and of the
// code words per tile (lt).  Tiles shrink from 2^max_lt words until there are at
// least three per compute unit (six for narrow matrices) or a tile is 1024
// words (or 8 rows) small.
struct TileShape {
  int lg, lt, blocks;
};

static int64_t tile_count(int64_t rows, int64_t cols, int lg, int lt) {
  const int64_t tr = 1LL << (lt - lg), tg = 1LL << lg;
  return ((rows + tr - 1) / tr) * (((cols >> 3) + tg - 1) / tg);
}

static TileShape tile_shape(int64_t rows, int64_t cols, int max_lt) {
  // Narrow matrices (at most 8 column groups, e.g. a convolution's 64
  // channels) have tall tiles whose count rarely divides the 256 compute units
  // evenly: there, twice as many smaller tiles go to at most 1024 persistent
  // workgroups (four per CU), which evens out the per-CU load (LUQ on the
  // 200704 x 64 conv gradient: 26.9 -> 25.1 us).  Wide matrices (the MLP
  // tensors) measured slower that way and keep one tile per workgroup.
  const int64_t cgs = cols >> 3;
  const bool narrow = cgs <= 8;
  const int64_t want = narrow ? 1536 : 768;
  TileShape t;
  t.lg = 0;
  while (t.lg < 5 && (1LL << t.lg) < cgs) ++t.lg;
  t.lt = max_lt;
  while (t.lt > 10 && t.lt - 1 - t.lg >= 3 && tile_count(rows, cols, t.lg, t.lt) < want) --t.lt;
  int64_t b = tile_count(rows, cols, t.lg, t.lt);
  if (b < 1) b = 1;
  if (b > kMaxEncodeBlocks) b = kMaxEncodeBlocks;
  if (narrow && b > 1024) b = 1024;
  t.blocks = (int)b;
  return t;
}

// Max pass.  Tensors that fit in the last-level cache are read with ordinary
// loads so that the encode pass can find them there; larger ones are streamed
// with non-temporal loads, except for their last kKeepBytes.

template <bool BF16, int MODE>
static void launch_max_pass(const void* x, int64_t n, int nblocks, uint32_t* partial, hipStream_t st,
                            int64_t stream_bytes = kCacheBytes, int64_t keep_bytes = kKeepBytes) {
  if (n * (BF16 ? 2 : 4) > stream_bytes)
    hipLaunchKernelGGL((max_partial_kernel<BF16, MODE, true>), dim3(nblocks), dim3(kThreads), 0, st, x, n,
                       partial, keep_bytes);
  else
    hipLaunchKernelGGL((max_partial_kernel<BF16, MODE, false>), dim3(nblocks), dim3(kThreads), 0, st, x, n,
                       partial, keep_bytes);
  if (nblocks > kDirectPartials)
    hipLaunchKernelGGL(fold_partials_kernel, dim3(1), dim3(1024), 0, st, partial, nblocks, partial + kMaxPartials);
}

// What the encode blocks fold: the partials themselves, or the one folded word.
static const uint32_t* encode_partials(const uint32_t* partial, int nblocks, int* nparts) {
  *nparts = nblocks > kDirectPartials ? 1 : nblocks;
  return nblocks > kDirectPartials ? partial + kMaxPartials : partial;
}

// Encode pass.  Its read is the tensor's second; it is non-temporal exactly
// when the max pass's was (tensors too large to stay in the last-level cache),
// and so are its code stores then.
static bool stream_reads(int64_t n, bool bf16) { return n * (bf16 ? 2 : 4) > kCacheBytes; }

// ns: 1 or 2 sample planes, or kSmpSum (two samples stored as int8 sums).
template <bool BF16, bool NT, bool HS>
static int luq_encode_launch(const LuqArgs& a, int ns, hipStream_t st) {
  if (a.codes_t) {
    const TileShape t = tile_shape(a.rows, a.cols, kLuqTileLg);
    if (ns == 1)
      hipLaunchKernelGGL((luq_encode_tile_kernel<BF16, NT, 1, HS>), dim3(t.blocks), dim3(kThreads), 0, st, a, t.lg,
                         t.lt);
    else if (ns == 2)
      hipLaunchKernelGGL((luq_encode_tile_kernel<BF16, NT, 2, HS>), dim3(t.blocks), dim3(kThreads), 0, st, a, t.lg,
                         t.lt);
    else
      hipLaunchKernelGGL((luq_encode_tile_kernel<BF16, NT, 2, HS, true>), dim3(t.blocks), dim3(kThreads), 0, st, a,
                         t.lg, t.lt);
    return t.blocks;
  }
  const int nb = encode_blocks_flat(a.n);
  if (ns == 1)
    hipLaunchKernelGGL((luq_encode_flat_kernel<BF16, NT, 1, HS>), dim3(nb), dim3(kThreads), 0, st, a);
  else if (ns == 2)
    hipLaunchKernelGGL((luq_encode_flat_kernel<BF16, NT, 2, HS>), dim3(nb), dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL((luq_encode_flat_kernel<BF16, NT, 2, HS, true>), dim3(nb), dim3(kThreads), 0, st, a);
  return nb;
}

template <bool BF16>
static hipError_t luq_launch_t(LuqArgs a, int ns, int nmax, hipStream_t st) {
  uint32_t* ws = const_cast<uint32_t*>(a.partial);
  // a bf16 gradient too large to stay cached beside a training step's other
  // data, but not streamed (kInt4StreamBytes .. kCacheBytes): the max pass
  // reads all of it non-temporally.  Read through the cache, it would evict
  // (and wait for the write-back of) the output the previous kernel left
  // there; the encode, bound by its ALU work, reads it again from memory.
  const int64_t bytes = a.n * (BF16 ? 2 : 4);
  if (BF16 && bytes > kInt4StreamBytes && bytes <= kCacheBytes)
    launch_max_pass<BF16, 0>(a.g, a.n, nmax, ws, st, 0, 0);
  else
    launch_max_pass<BF16, 0>(a.g, a.n, nmax, ws, st);
  a.partial = encode_partials(ws, nmax, &a.nparts);
  if (stream_reads(a.n, BF16))
    luq_encode_launch<BF16, true, false>(a, ns, st);
  else
    luq_encode_launch<BF16, false, false>(a, ns, st);
  return hipGetLastError();
}

hipError_t launch_luq_quantize(const void* g, int bf16, int64_t rows, int64_t cols, int R, int pw2,
                               uint64_t seed, uint32_t counter, int ns, uint8_t* codes,
                               uint8_t* codes_t, float* alpha, float* maxabs, void* ws,
                               hipStream_t st) {
  const int64_t n = rows * cols;
  uint32_t* status = ws ? static_cast<uint32_t*>(ws) + kStatusWord : nullptr;
  if (n == 0) {
    hipLaunchKernelGGL(write_two_floats_kernel, dim3(1), dim3(1), 0, st, alpha, 0.0f, maxabs, 0.0f, status);
    return hipGetLastError();
  }
  LuqArgs a;
  a.g = g;
  a.rows = rows;
  a.cols = cols;
  a.n = n;
  a.R = R;
  a.pw2 = pw2 != 0;
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
  a.state = nullptr;
  a.part_out = nullptr;
  a.status = status;
  return bf16 ? luq_launch_t<true>(a, ns, a.nparts, st) : luq_launch_t<false>(a, ns, a.nparts, st);
}

// ---------------------------- allocation-free LUQ ----------------------------
//
// For callers that cannot allocate device memory: the workspace of
// luq_quantize_grad (partial maxima, their fold, the status word) lives in
// this file-scope device array instead, one copy per GPU, held until the
// process ends.  In host code `scratch` names a host-side stand-in, not the
// device array: its device address is looked up once per device with
// hipGetSymbolAddress and only that address is used.  Calls on one GPU share
// the array, so calls that overlap in time on one GPU race; nothing in it
// needs to start at zero (every word a call reads, the same call wrote).
constexpr size_t kScratchWords = kStatusWord + 1;
static __device__ __align__(256) uint32_t scratch[kScratchWords];

constexpr int kMaxScratchDevices = 64;
static std::atomic<uint32_t*> g_scratch_ptr[kMaxScratchDevices];

size_t noalloc_scratch_bytes() { return sizeof(uint32_t) * kScratchWords; }

// The device address of `scratch` on the current device (looked up on the
// first call on that device); null with the HIP error in *err on failure.
static uint32_t* scratch_on_current_device(hipError_t* err) {
  int dev = 0;
  *err = hipGetDevice(&dev);
  if (*err != hipSuccess) return nullptr;
  if (dev < 0 || dev >= kMaxScratchDevices) {
    *err = hipErrorInvalidDevice;
    return nullptr;
  }
  uint32_t* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    void* addr = nullptr;
    *err = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
    if (*err != hipSuccess || !addr) {
      if (*err == hipSuccess) *err = hipErrorInvalidSymbol;
      return nullptr;
    }
    p = static_cast<uint32_t*>(addr);
    g_scratch_ptr[dev].store(p, std::memory_order_release);  // racing threads store the same address
  }
  return p;
}

hipError_t launch_luq_quantize_noalloc(const void* g, int bf16, int64_t rows, int64_t cols, int R, int pw2,
                                       uint64_t seed, uint32_t counter, int ns, uint8_t* codes, uint8_t* codes_t,
                                       float* alpha, float* maxabs, hipStream_t st) {
  if (quant_workspace_bytes(rows * cols) > noalloc_scratch_bytes()) return hipErrorInvalidValue;
  hipError_t err = hipSuccess;
  uint32_t* ws = scratch_on_current_device(&err);
  if (!ws) return err;
  return launch_luq_quantize(g, bf16, rows, cols, R, pw2, seed, counter, ns, codes, codes_t, alpha, maxabs, ws, st);
}

hipError_t launch_luq_quantize_hindsight(const void* g, int bf16, int64_t rows, int64_t cols, int R, int pw2,
                                         uint64_t seed, uint32_t counter, int ns, float eta, uint8_t* codes,
                                         uint8_t* codes_t, float* state, float* alpha, float* maxabs, void* ws,
                                         hipStream_t st) {
  const int64_t n = rows * cols;
  LuqArgs a;
  a.g = g;
  a.rows = rows;
  a.cols = cols;
  a.n = n;
  a.R = R;
  a.pw2 = pw2 != 0;
  a.k0 = (uint32_t)seed;
  a.k1 = (uint32_t)(seed >> 32);
  a.counter = counter;
  a.partial = nullptr;
  a.nparts = 0;
  a.codes = codes;
  a.codes_t = codes_t;
  a.plane = (int64_t)plane_bytes(n);
  a.alpha_out = alpha;
  a.max_out = maxabs;
  a.state = state;
  a.part_out = static_cast<uint32_t*>(ws);
  a.status = nullptr;  // written by the fold
  int nblocks = 0;
  if (n > 0) {
    const bool nt = stream_reads(n, bf16 != 0);
    nblocks = bf16 ? (nt ? luq_encode_launch<true, true, true>(a, ns, st) : luq_encode_launch<true, false, true>(a, ns, st))
                   : (nt ? luq_encode_launch<false, true, true>(a, ns, st)
                         : luq_encode_launch<false, false, true>(a, ns, st));
  }
  hipLaunchKernelGGL(hindsight_fold_kernel, dim3(1), dim3(1024), 0, st, a.part_out, nblocks, state,
                     1.0f - eta, eta, R, pw2 != 0, alpha, maxabs,
                     ws ? static_cast<uint32_t*>(ws) + kStatusWord : nullptr);  // c1 = fl32(1 - eta) (host float arithmetic)
  return hipGetLastError();
}

template <bool BF16>
static hipError_t int4_launch_t(Int4Args a, hipStream_t st) {
  if (a.n <= kInt4SmallN) {
    const TileShape t = tile_shape(a.rows, a.cols, kInt4TileLg);
    int blocks = a.codes_t ? t.blocks : (int)((((a.n + 7) >> 3) + kThreads - 1) / kThreads);
    if (blocks > kInt4SmallBlocks) blocks = kInt4SmallBlocks;
    if (a.is_signed)
      hipLaunchKernelGGL((int4_small_kernel<BF16, 0>), dim3(blocks), dim3(kThreads), 0, st, a, t.lg, t.lt);
    else
      hipLaunchKernelGGL((int4_small_kernel<BF16, 1>), dim3(blocks), dim3(kThreads), 0, st, a, t.lg, t.lt);
    return hipGetLastError();
  }
  if (a.clip <= 0.0f) {
    if (a.is_signed)
      launch_max_pass<BF16, 0>(a.x, a.n, a.nparts, const_cast<uint32_t*>(a.partial), st, kInt4StreamBytes, 0);
    else
      launch_max_pass<BF16, 1>(a.x, a.n, a.nparts, const_cast<uint32_t*>(a.partial), st, kInt4StreamBytes, 0);
    a.partial = encode_partials(a.partial, a.nparts, &a.nparts);
  }
  const bool nt = a.n * (BF16 ? 2 : 4) > kInt4StreamBytes;
  if (a.codes_t) {
    const TileShape t = tile_shape(a.rows, a.cols, kInt4TileLg);
    if (nt)
      hipLaunchKernelGGL((int4_encode_tile_kernel<BF16, true>), dim3(t.blocks), dim3(kThreads), 0, st, a, t.lg, t.lt);
    else
      hipLaunchKernelGGL((int4_encode_tile_kernel<BF16, false>), dim3(t.blocks), dim3(kThreads), 0, st, a, t.lg, t.lt);
  } else if (nt) {
    hipLaunchKernelGGL((int4_encode_flat_kernel<BF16, true>), dim3(encode_blocks_flat(a.n)), dim3(kThreads), 0, st, a);
  } else {
    hipLaunchKernelGGL((int4_encode_flat_kernel<BF16, false>), dim3(encode_blocks_flat(a.n)), dim3(kThreads), 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_int4_quantize(const void* x, int bf16, int64_t rows, int64_t cols, int is_signed,
                                float clip, uint8_t* codes, uint8_t* codes_t, float* scale,
                                void* ws, hipStream_t st) {
  const int64_t n = rows * cols;
  uint32_t* status = ws ? static_cast<uint32_t*>(ws) + kStatusWord : nullptr;
  if (n == 0) {
    hipLaunchKernelGGL(write_two_floats_kernel, dim3(1), dim3(1), 0, st, scale, 0.0f,
                       (float*)nullptr, 0.0f, status);
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
  a.status = status;
  return bf16 ? int4_launch_t<true>(a, st) : int4_launch_t<false>(a, st);
}

}  // namespace luq

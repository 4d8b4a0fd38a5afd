// Device helpers shared by the libluq kernels (gfx950 / CDNA4, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace luq {

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon et al., SC'11).  Ten rounds; each round takes the
// full 64-bit products of the two multipliers with words 0 and 2 (one
// v_mad_u64_u32 each) and mixes in the key, which is bumped by the Weyl
// constants after every round.  The key is wave-uniform, so its schedule
// stays in scalar registers.
// ---------------------------------------------------------------------------
struct U4 {
  uint32_t x, y, z, w;
};

// a ^ b ^ k in one VALU instruction (k wave-uniform): gfx950's three-input
// bitwise op with the odd-parity truth table 0x96.  The compiler does not
// form it on its own here.
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t k) {
  uint32_t r;
  asm("v_bitop3_b32 %0, %1, %2, %3 bitop3:0x96" : "=v"(r) : "v"(a), "v"(b), "s"(k));
  return r;
}

__device__ __forceinline__ U4 philox4x32_10(U4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c.x;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c.z;
    const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    c = U4{xor3(hi1, c.y, k0), lo1, xor3(hi0, c.w, k1), lo0};
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

// ---------------------------------------------------------------------------
// Loads of 8 consecutive elements as float32 bit patterns (exact for bf16:
// a bfloat16 is the upper half of the float32 with the same value).
// ---------------------------------------------------------------------------
struct U8 {
  uint32_t v[8];
};

typedef uint32_t v4u32 __attribute__((ext_vector_type(4)));

// One code word at p (4-byte aligned); NT marks the store non-temporal (the
// codes of a tensor too large for the last-level cache).
template <bool NT>
__device__ __forceinline__ void store_word(uint8_t* p, uint32_t v) {
  if constexpr (NT) __builtin_nontemporal_store(v, reinterpret_cast<uint32_t*>(p));
  else *reinterpret_cast<uint32_t*>(p) = v;
}

// 16 bytes at p; NT marks the load non-temporal (streaming data read once).
template <bool NT>
__device__ __forceinline__ v4u32 load16(const void* p) {
  if constexpr (NT) return __builtin_nontemporal_load(static_cast<const v4u32*>(p));
  return *static_cast<const v4u32*>(p);
}

template <bool BF16, bool NT = false>
__device__ __forceinline__ U8 load8(const void* base, int64_t elem) {
  U8 r;
  if constexpr (BF16) {
    const v4u32 q = load16<NT>(static_cast<const uint16_t*>(base) + elem);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      r.v[2 * i] = q[i] << 16;
      r.v[2 * i + 1] = q[i] & 0xFFFF0000u;
    }
  } else {
    const float* p = static_cast<const float*>(base) + elem;
    const v4u32 a = load16<NT>(p), b = load16<NT>(p + 4);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      r.v[i] = a[i];
      r.v[4 + i] = b[i];
    }
  }
  return r;
}

// Bounded variant for a ragged tail: elements at or beyond n read as +0.
template <bool BF16>
__device__ __forceinline__ U8 load8_tail(const void* base, int64_t elem, int64_t n) {
  U8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    uint32_t b = 0;
    if (elem + i < n) {
      if constexpr (BF16)
        b = (uint32_t)(static_cast<const uint16_t*>(base)[elem + i]) << 16;
      else
        b = static_cast<const uint32_t*>(base)[elem + i];
    }
    r.v[i] = b;
  }
  return r;
}

// ---------------------------------------------------------------------------
// Reductions of unsigned keys (float32 bit patterns of non-negative values,
// whose unsigned order is the float order; non-finite values sort above
// every finite one).
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, off, kWave));
  return v;
}

// Max over a block of `threads` threads (a multiple of 64, at most 1024).
// Every thread gets the result.  `scratch` holds at least threads/64 words.
__device__ __forceinline__ uint32_t block_max_u32(uint32_t v, uint32_t* scratch) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int nwaves = blockDim.x / kWave;
  v = wave_max_u32(v);
  __syncthreads();  // scratch may still be read by a previous call
  if (lane == 0) scratch[wave] = v;
  __syncthreads();
  uint32_t m = 0;
  for (int i = 0; i < nwaves; ++i) m = max(m, scratch[i]);
  return m;
}

// Max of the per-block partial keys written by a max pass.  Eight loads per
// thread are in flight at once: indices past the end are clamped to the last
// partial, which leaves the maximum unchanged and keeps every load in bounds
// (a conditional load would make each one wait for the previous).
__device__ __forceinline__ uint32_t reduce_partials(const uint32_t* partial, int nparts,
                                                    uint32_t* scratch) {
  uint32_t m = 0;
  const int step = blockDim.x;
  for (int i0 = threadIdx.x; i0 < nparts; i0 += 8 * step) {
    uint32_t v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = partial[min(i0 + k * step, nparts - 1)];
#pragma unroll
    for (int k = 0; k < 8; ++k) m = max(m, v[k]);
  }
  return block_max_u32(m, scratch);
}

// ---------------------------------------------------------------------------
// 8x8 transpose of 4-bit fields: on entry r[i] holds row i (nibble j at bits
// 4j); on exit r[j] holds column j (nibble i at bits 4i).  Three rounds of
// field swaps between row pairs at distance 1, 2 and 4 (4-, 8-, 16-bit).
// ---------------------------------------------------------------------------
__device__ __forceinline__ void swap_fields(uint32_t& a, uint32_t& b, int s, uint32_t mask) {
  const uint32_t t = ((a >> s) ^ b) & mask;
  b ^= t;
  a ^= t << s;
}

__device__ __forceinline__ void transpose8x8_nibbles(uint32_t (&r)[8]) {
  swap_fields(r[0], r[1], 4, 0x0F0F0F0Fu);
  swap_fields(r[2], r[3], 4, 0x0F0F0F0Fu);
  swap_fields(r[4], r[5], 4, 0x0F0F0F0Fu);
  swap_fields(r[6], r[7], 4, 0x0F0F0F0Fu);
  swap_fields(r[0], r[2], 8, 0x00FF00FFu);
  swap_fields(r[1], r[3], 8, 0x00FF00FFu);
  swap_fields(r[4], r[6], 8, 0x00FF00FFu);
  swap_fields(r[5], r[7], 8, 0x00FF00FFu);
  swap_fields(r[0], r[4], 16, 0x0000FFFFu);
  swap_fields(r[1], r[5], 16, 0x0000FFFFu);
  swap_fields(r[2], r[6], 16, 0x0000FFFFu);
  swap_fields(r[3], r[7], 16, 0x0000FFFFu);
}

// ---------------------------------------------------------------------------
// SMP operand as bytes (Section 5.1: the average of two samples taken with
// one alpha is alpha/2 times the sum of their decoded values).
// ---------------------------------------------------------------------------

// The 8 nibbles of x, one per byte in element order: lo = elements 0..3,
// hi = elements 4..7.
__device__ __forceinline__ void spread_nibbles(uint32_t x, uint32_t& lo, uint32_t& hi) {
  // byte 2i of the selection from x, byte 2i+1 from x >> 4 (whose byte i
  // starts with the high nibble of x's byte i)
  const uint32_t y = x >> 4;
  lo = __builtin_amdgcn_perm(y, x, 0x05010400u) & 0x0F0F0F0Fu;
  hi = __builtin_amdgcn_perm(y, x, 0x07030602u) & 0x0F0F0F0Fu;
}

// Sum of the decoded values of two LUQ codes per byte (one nibble per byte):
// magnitudes 2^(e-1) from a byte LUT, added (<= 64 for fields <= 6, so no
// carries), then negated where either code carries a sign (both samples of
// an element have its sign; zero codes have none).
__device__ __forceinline__ uint32_t smp_sum4(uint32_t n0, uint32_t n1) {
  const uint32_t t_lo = 0x04020100u, t_hi = 0x40201008u;  // 0, 1, 2, 4, 8, 16, 32, 64
  const uint32_t m = __builtin_amdgcn_perm(t_hi, t_lo, n0 & 0x07070707u) +
                     __builtin_amdgcn_perm(t_hi, t_lo, n1 & 0x07070707u);
  const uint32_t sg = ((n0 | n1) >> 3) & 0x01010101u;
  return (m ^ ((sg << 8) - sg)) + sg;  // (m ^ 0xFF) + 1 in the negative bytes
}

// int8 sums of the 8 elements of two sample code words, in element order.
__device__ __forceinline__ void smp_sum_bytes(uint32_t c0, uint32_t c1, uint32_t& lo, uint32_t& hi) {
  uint32_t l0, h0, l1, h1;
  spread_nibbles(c0, l0, h0);
  spread_nibbles(c1, l1, h1);
  lo = smp_sum4(l0, l1);
  hi = smp_sum4(h0, h1);
}

// 4x4 transpose of bytes: r[i] holds row i (byte j = column j); c[j] gets
// column j (byte i = row i).
__device__ __forceinline__ void transpose4x4_bytes(const uint32_t (&r)[4], uint32_t (&c)[4]) {
  const uint32_t t0 = __builtin_amdgcn_perm(r[1], r[0], 0x05010400u);  // r0c0 r1c0 r0c1 r1c1
  const uint32_t t1 = __builtin_amdgcn_perm(r[1], r[0], 0x07030602u);  // r0c2 r1c2 r0c3 r1c3
  const uint32_t t2 = __builtin_amdgcn_perm(r[3], r[2], 0x05010400u);
  const uint32_t t3 = __builtin_amdgcn_perm(r[3], r[2], 0x07030602u);
  c[0] = __builtin_amdgcn_perm(t2, t0, 0x05040100u);
  c[1] = __builtin_amdgcn_perm(t2, t0, 0x07060302u);
  c[2] = __builtin_amdgcn_perm(t3, t1, 0x05040100u);
  c[3] = __builtin_amdgcn_perm(t3, t1, 0x07060302u);
}

typedef uint32_t v2u32 __attribute__((ext_vector_type(2)));

// 8 bytes (lo, hi) at p (8-byte aligned).
template <bool NT>
__device__ __forceinline__ void store_word2(uint8_t* p, uint32_t lo, uint32_t hi) {
  const v2u32 v = {lo, hi};
  if constexpr (NT) __builtin_nontemporal_store(v, reinterpret_cast<v2u32*>(p));
  else *reinterpret_cast<v2u32*>(p) = v;
}

// Stores the first `nbytes` (0..4) bytes of w at p (ragged tails).
__device__ __forceinline__ void store_bytes(uint8_t* p, uint32_t w, int nbytes) {
  for (int i = 0; i < nbytes; ++i) p[i] = (uint8_t)(w >> (8 * i));
}

}  // namespace luq

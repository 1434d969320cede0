// Device-side helpers shared by the libhswa kernels (gfx950 / CDNA4, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hswa_launch.h"

namespace hswa {

constexpr int kWave = 64;

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x4 __attribute__((__vector_size__(4 * sizeof(float))));
typedef float f32x16 __attribute__((__vector_size__(16 * sizeof(float))));
typedef uint32_t u32x4 __attribute__((__vector_size__(4 * sizeof(uint32_t))));
typedef uint32_t u32x2 __attribute__((__vector_size__(2 * sizeof(uint32_t))));

// 16x16 output, 32-deep bf16 matrix multiply-accumulate (v_mfma_f32_16x16x32_bf16).
// Lane l supplies row (l % 16) of A and column (l % 16) of B, each as 8
// consecutive reduction elements of block l / 16; it receives C rows
// 4 * (l / 16) + i, i = 0..3, of column l % 16.
__device__ __forceinline__ f32x4 mfma16x16x32(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ u32x4 ldg128(const void *p) {
  return *reinterpret_cast<const u32x4 *>(p);
}

__device__ __forceinline__ void stg128(void *p, u32x4 v) { *reinterpret_cast<u32x4 *>(p) = v; }

// 16-byte load through the global address space, for a source pointer chosen
// at run time between buffers (which would otherwise become a flat load, one
// that also counts against the LDS wait counter).
typedef __attribute__((address_space(1))) const u32x4 global_u32x4;
__device__ __forceinline__ u32x4 ldg128_global(const void *p) { return *(global_u32x4 *)p; }

// Bits i (0 .. 7) of the keys k0 + i inside [lo, hi].
__device__ __forceinline__ uint32_t key_range_bits(int k0, int lo, int hi) {
  const int a = min(max(lo - k0, 0), 8);
  const int z = min(max(hi - k0 + 1, 0), 8);
  return ((1u << z) - 1u) & ~((1u << a) - 1u);
}

// Element offset in the K pool of (page, KV head g, in-page key offset o, dim d).
// In a block of B = 2^vb_shift keys, key k sits in half (k >> 2) & 1 at row
// ((k >> 3) << 2) | (k & 3); dim d in slab d >> 5, 16-byte piece (d >> 3) & 3.
// A slab is [4 pieces][B/2 rows][8 dims], so for B = 32 the bf16-MFMA A operand
// of 16 keys (lane = row + 16 * piece) x 32 dims is lane-linear.
__device__ __forceinline__ int64_t k_offset(const PoolView &pv, int64_t page, int hkv, int g, int o, int d) {
  const int kb = pv.vb_shift;
  const int k = o & ((1 << kb) - 1);
  const int half = (k >> 2) & 1, row = ((k >> 3) << 2) | (k & 3);
  const int slab = (half << 2) | (d >> 5);
  return (((page * hkv + g) << pv.pg_shift) << kHeadDimShift) + ((int64_t)(o >> kb) << (kb + kHeadDimShift)) +
         ((((slab << 2) | ((d >> 3) & 3)) << (kb - 1)) + row) * 8 + (d & 7);
}

// Element offset in the V pool of (page, KV head g, in-page key offset o, dim d).
__device__ __forceinline__ int64_t v_offset(const PoolView &pv, int64_t page, int hkv, int g, int o, int d) {
  const int vb = pv.vb_shift;
  return (((page * hkv + g) << pv.pg_shift) << kHeadDimShift) + ((int64_t)(o >> vb) << (vb + kHeadDimShift)) +
         ((int64_t)d << vb) + (o & ((1 << vb) - 1));
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Round two floats to bf16 (nearest, ties to even) and pack them (lo first);
// one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

__device__ __forceinline__ uint16_t to_bf16_bits(float x) {
  __bf16 a = (__bf16)x;
  return __builtin_bit_cast(uint16_t, a);
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t bits16) {
  return __builtin_bit_cast(float, bits16 << 16);
}

// Keep the bf16 elements of an 8-element vector whose bit is set in `keep8`
// (bit i = element i); zero the others. Used so that masked keys contribute
// exact zeros even when their cache slots hold NaN or garbage.
__device__ __forceinline__ u32x4 keep_bf16x8(u32x4 v, uint32_t keep8) {
  u32x4 r;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    uint32_t m = ((keep8 >> (2 * j)) & 1u ? 0x0000FFFFu : 0u) | ((keep8 >> (2 * j + 1)) & 1u ? 0xFFFF0000u : 0u);
    r[j] = v[j] & m;
  }
  return r;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// acc + lo + hi of two packed bf16 values (v_dot2_f32_bf16 against ones).
__device__ __forceinline__ float dot2_bf16_ones(uint32_t packed, float acc) {
  const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, packed), one, acc, false);
}

// Maximum without the NaN-quieting canonicalisation that fmaxf implies (scores
// here are finite or -inf, never NaN).
__device__ __forceinline__ float max2(float a, float b) {
  float r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ __forceinline__ float max3(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}
__device__ __forceinline__ float max8(const float *x) {
  return max3(max3(x[0], x[1], x[2]), max3(x[3], x[4], x[5]), max2(x[6], x[7]));
}

// Lane exchanges across 16-lane rows with the gfx950 permlane swaps (VALU, no
// LDS round trip): the pair returned holds x[l] and x[l ^ 16] (or x[l ^ 32]).
__device__ __forceinline__ float max_xor16(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return max2(__builtin_bit_cast(float, (uint32_t)r[0]), __builtin_bit_cast(float, (uint32_t)r[1]));
}
__device__ __forceinline__ float max_xor32(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return max2(__builtin_bit_cast(float, (uint32_t)r[0]), __builtin_bit_cast(float, (uint32_t)r[1]));
}
__device__ __forceinline__ float sum_xor16(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return __builtin_bit_cast(float, (uint32_t)r[0]) + __builtin_bit_cast(float, (uint32_t)r[1]);
}
__device__ __forceinline__ float sum_xor32(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __builtin_bit_cast(float, (uint32_t)r[0]) + __builtin_bit_cast(float, (uint32_t)r[1]);
}

constexpr float kLog2e = 1.4426950408889634f;

// Writes one output row from the MFMA accumulator layout: lane r + 16 q holds
// dims 16 dt + 4 q .. +3 of row r as two bf16 pairs w[dt] (dt = 0..7). Lanes l
// and l ^ 16 (same row) swap halves so that each holds 8 consecutive dims (dt
// even in the lanes with q even, odd in the others); one 16-byte store then
// writes a 64-byte run of each of the wave's 16 rows. The stores are
// nontemporal: an output is written once and not read back. Every lane of the
// wave must take part (the swaps are cross-lane); a lane with `write` false
// (its partner has the same row, hence the same flag) stores nothing.
__device__ __forceinline__ void store_out_row(uint16_t *orow, const u32x2 (&w)[8], int q, bool write) {
  u32x4 v[4];
#pragma unroll
  for (int pp = 0; pp < 4; ++pp) {
    const auto s0 = __builtin_amdgcn_permlane16_swap(w[2 * pp][0], w[2 * pp + 1][0], false, false);
    const auto s1 = __builtin_amdgcn_permlane16_swap(w[2 * pp][1], w[2 * pp + 1][1], false, false);
    v[pp] = u32x4{(uint32_t)s0[0], (uint32_t)s1[0], (uint32_t)s0[1], (uint32_t)s1[1]};
  }
  if (!write) return;
#pragma unroll
  for (int pp = 0; pp < 4; ++pp)
    __builtin_nontemporal_store(v[pp], reinterpret_cast<u32x4 *>(orow + 32 * pp + 16 * (q & 1) + 8 * (q >> 1)));
}

// Launch a kernel taking one parameter struct and return the status of exactly
// this launch (hipGetLastError would also report errors left behind by earlier,
// unrelated runtime calls of the caller).
template <typename Params>
inline hipError_t launch_kernel(void (*kernel)(Params), dim3 grid, dim3 block, hipStream_t stream,
                                const Params &p) {
  void *args[] = {const_cast<Params *>(&p)};
  return hipLaunchKernel(reinterpret_cast<const void *>(kernel), grid, block, args, 0, stream);
}

}  // namespace hswa

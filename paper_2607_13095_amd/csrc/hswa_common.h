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

// Round two floats to bf16 (nearest, ties to even) and pack them (lo first).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  __bf16 a = (__bf16)lo, b = (__bf16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
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

__device__ __forceinline__ float wave_max_xor(float v, int mask) {
  return fmaxf(v, __shfl_xor(v, mask, kWave));
}

__device__ __forceinline__ float wave_sum_xor(float v, int mask) { return v + __shfl_xor(v, mask, kWave); }

constexpr float kLog2e = 1.4426950408889634f;

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

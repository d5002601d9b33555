// Device-side types and helpers shared by the SpecQuant HIP kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sq {

typedef _Float16 half_t;
typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float float4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

__device__ __forceinline__ float f16_bits_to_f32(uint16_t b) {
  return (float)__builtin_bit_cast(half_t, b);
}

__device__ __forceinline__ uint16_t f32_to_f16_bits(float v) {
  return __builtin_bit_cast(uint16_t, (half_t)v);
}

// Sum across the 64 lanes of a wavefront; every lane receives the total.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

// Output conversion for y[m][n] in either fp16 or fp32.
template <bool F16Out>
__device__ __forceinline__ void store_out(void* y, int64_t idx, float v) {
  if constexpr (F16Out)
    reinterpret_cast<uint16_t*>(y)[idx] = f32_to_f16_bits(v);
  else
    reinterpret_cast<float*>(y)[idx] = v;
}

}  // namespace sq

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

template <int Ctrl>
__device__ __forceinline__ float dpp_add(float v) {
  return v + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), Ctrl, 0xF, 0xF,
                                                                   false));
}

// Sums of V = 4T values across the 64 lanes of a wavefront, transposed: the
// lane halves are folded with v_permlane32_swap, the row pairs with
// v_permlane16_swap, and the 16-lane rows with DPP, 2.5 operations per value.
// Afterwards every lane of row j of w[t] holds the total of value
// 4t + (0, 2, 1, 3)[j].
template <int T>
__device__ __forceinline__ void wave_sums(const float (&v)[4 * T], float (&w)[T]) {
#pragma unroll
  for (int t = 0; t < T; ++t) {
    float u[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const auto p = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(int, v[4 * t + 2 * h]),
                                                      __builtin_bit_cast(int, v[4 * t + 2 * h + 1]), false, false);
      const int p0 = p[0], p1 = p[1];  // bit-cast scalar copies: vector element lvalues are misread
      u[h] = __builtin_bit_cast(float, p0) + __builtin_bit_cast(float, p1);
    }
    const auto q = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(int, u[0]), __builtin_bit_cast(int, u[1]),
                                                    false, false);
    const int q0 = q[0], q1 = q[1];
    float x = __builtin_bit_cast(float, q0) + __builtin_bit_cast(float, q1);
    x = dpp_add<0xB1>(x);   // quad_perm [1,0,3,2]
    x = dpp_add<0x4E>(x);   // quad_perm [2,3,0,1]
    x = dpp_add<0x141>(x);  // row_half_mirror
    x = dpp_add<0x140>(x);  // row_mirror: every lane holds its row's total
    w[t] = x;
  }
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

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

// RMS normalisation shared by the residual-add kernel and the projections
// that normalise their own input rows, so that both give the same bits.
// A row of k fp32 values is summed in squares by 256 threads: thread t takes
// the float4 cells t, t + 256, ... in order, each as (a^2 + b^2) + (c^2 + d^2)
// (no fused multiply-add); the threads' sums meet by wave_sum and then as
// (w0 + w1) + (w2 + w3) over the four wavefronts.
__device__ __forceinline__ float rms_cell_sq(float4_t v) {
#pragma clang fp contract(off)
  return (v[0] * v[0] + v[1] * v[1]) + (v[2] * v[2] + v[3] * v[3]);
}

// 1 / sqrt(mean + eps) of a row from its four wavefront sums, in fp64,
// rounded once to fp32.
__device__ __forceinline__ float rms_inverse(const float* wsum4, int k, float eps) {
  const float total = (wsum4[0] + wsum4[1]) + (wsum4[2] + wsum4[3]);
  return (float)(1.0 / sqrt((double)total / (double)k + (double)eps));
}

// One normalised value: f16(h * r * w), the products in fp32 left to right.
__device__ __forceinline__ half_t rms_scale(float h, float r, half_t w) {
#pragma clang fp contract(off)
  return (half_t)(h * r * (float)w);
}

// The sums of squares of the M staged rows of a projection that normalises
// its own input (row m is hrow0 + m * stride), on the threads of each group of
// 256 (group gr takes rows gr, gr + groups, ...; RPT rows per thread at most,
// rows of at most 4096 values).  load() issues the loads, finish() sums them
// in the order of the residual-add kernel and writes each wavefront's sum of
// row m to wsum[4 m + wavefront % 4].
template <int RPT>
struct RmsRows {
  float4_t v[RPT][4];
  __device__ __forceinline__ void load(const float* __restrict__ hrow0, int64_t stride, int M, int k) {
    const int t = threadIdx.x & 255, gr = threadIdx.x >> 8, ngr = blockDim.x >> 8, n4 = k >> 2;
#pragma unroll
    for (int j = 0; j < RPT; ++j) {
      const int m = gr + j * ngr;
      const float4_t* hr = reinterpret_cast<const float4_t*>(hrow0 + (int64_t)(m < M ? m : 0) * stride);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int c = t + 256 * i;
        v[j][i] = c < n4 ? hr[c] : float4_t{0.f, 0.f, 0.f, 0.f};
      }
    }
  }
  __device__ __forceinline__ void finish(int M, int k, float* wsum) const {
    const int t = threadIdx.x & 255, gr = threadIdx.x >> 8, ngr = blockDim.x >> 8, n4 = k >> 2;
#pragma unroll
    for (int j = 0; j < RPT; ++j) {
      const int m = gr + j * ngr;
      if (m >= M) continue;  // uniform across the wavefront
      float ss = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (t + 256 * i < n4) ss += rms_cell_sq(v[j][i]);
      ss = wave_sum(ss);
      if ((t & 63) == 0) wsum[4 * m + (t >> 6)] = ss;
    }
  }
};

// Eight normalised activations f16(h * r * w) of one 16-byte cell, from the
// eight fp32 values h0 | h1 and the eight fp16 norm weights wc.
__device__ __forceinline__ u32x4 rms_cell(float4_t h0, float4_t h1, u32x4 wc, float r) {
  const half8_t w8 = __builtin_bit_cast(half8_t, wc);
  half8_t o;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    o[e] = rms_scale(h0[e], r, w8[e]);
    o[4 + e] = rms_scale(h1[e], r, w8[4 + e]);
  }
  return __builtin_bit_cast(u32x4, o);
}

// The SiLU-gated product f16(g / (1 + e^-g) * u) of a gate and an up value,
// shared by the SiLU kernel and the gate|up projection that applies it to its
// own outputs (the same bits).
__device__ __forceinline__ uint16_t silu_gate_bits(float g, float u) {
  return f32_to_f16_bits(g / (1.f + expf(-g)) * u);
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

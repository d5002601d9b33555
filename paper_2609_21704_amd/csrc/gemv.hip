// Dequant-fused draft GEMVs (SpecQuant SS III-D.2: the draft parent Q4 or Q8
// produces the speculative tokens; every draft step streams the whole
// quantized stack once at m = 1 .. 8 activation rows).
//
// The kernels are HBM-bound: each weight byte is read exactly once, with
// 16-byte loads that are contiguous across the lanes of a wavefront.  The
// activations of the workgroup's K range are staged once in LDS; each lane
// reads its x chunk from LDS once per chunk position and reuses it for the
// four rows its wavefront streams together.
//
// INT4 (W4A16).  A 16-byte load holds 32 consecutive 4-bit codes of one row,
// i.e. a quarter of one 128-element group.  Each 32-bit word (codes of k..k+7)
// is turned into four half2 values without a conversion instruction: a nibble
// masked into mantissa bits 0-3 (or 4-7) of the binary16 constant 1024 (or
// 64) is the exact value 1024 + q (or 64 + q); one shift by 8 serves the
// upper nibble pairs.  Subtracting the packed constant c + z in fp16 is exact
// and leaves q - z in [-15, 15], so v_dot2_f32_f16 forms exact products
// (q - z) * x and the fp32 accumulation error is bounded by sum |(q - z) x|;
// the group scale multiplies the chunk sum once.  Per word: one shift, four
// and-or, four packed subtracts, four dot2 -- 1.6 VALU operations per weight
// at m = 1.
//
// FP8 (W8A16).  A 16-byte load holds 16 E4M3 codes; v_cvt_scalef32_pk_f16_fp8
// converts two codes to two exact binary16 values, v_dot2_f32_f16 accumulates,
// and the per-row fp32 scale is applied once after the reduction.
#include "sq_device.hpp"
#include "sq_internal.hpp"

namespace sq {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kRows = 4;                    // rows streamed together by one wavefront
constexpr size_t kLdsBudget = 64 * 1024;    // bytes of LDS one workgroup may use

// ----------------------------------------------------------------- INT4 ----
// LDS layout for a K slice of nchunk 32-element chunks (consecutive chunks,
// which consecutive lanes read, are consecutive 16-byte cells):
//   xs [M][4 words][nchunk][8 halves], halves of word w in the order
//      x[8w+0], x[8w+4], x[8w+1], x[8w+5], x[8w+2], x[8w+6], x[8w+3], x[8w+7]
// matching the nibble pairs (0,4), (1,5), (2,6), (3,7) of a code word.
template <int M>
__device__ __forceinline__ void stage_x_w4(const uint16_t* __restrict__ x, int64_t k, int64_t k0, int nchunk,
                                           half_t* xs) {
  for (int idx = threadIdx.x; idx < nchunk * M * 4; idx += kThreads) {
    const int c = idx / (M * 4), rem = idx % (M * 4), m = rem >> 2, wd = rem & 3;
    const u32x4 raw = *reinterpret_cast<const u32x4*>(x + (int64_t)m * k + k0 + 32 * c + 8 * wd);
    half_t e[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) e[i] = __builtin_bit_cast(half_t, (uint16_t)(raw[i >> 1] >> (16 * (i & 1))));
    const half8_t p = {e[0], e[4], e[1], e[5], e[2], e[6], e[3], e[7]};
    *reinterpret_cast<half8_t*>(xs + (((size_t)m * 4 + wd) * nchunk + c) * 8) = p;
  }
}

template <int M, bool F16Out>
__global__ __launch_bounds__(kThreads) void gemv_w4_kernel(const uint16_t* __restrict__ x, int64_t k, int64_t kslice,
                                                           const uint8_t* __restrict__ codes,
                                                           const uint16_t* __restrict__ scales,
                                                           const uint16_t* __restrict__ zeros, int64_t n,
                                                           void* __restrict__ y, float* __restrict__ partial) {
  extern __shared__ __align__(16) char smem[];
  const int split = blockIdx.y;
  const int64_t k0 = (int64_t)split * kslice;
  const int64_t kl = (k - k0) < kslice ? (k - k0) : kslice;
  const int nchunk = (int)(kl / 32);
  half_t* xs = reinterpret_cast<half_t*>(smem);
  stage_x_w4<M>(x, k, k0, nchunk, xs);
  __syncthreads();

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t groups = k / 128;
  const int64_t nquads = (n + kRows - 1) / kRows;
  for (int64_t quad = (int64_t)blockIdx.x * kWaves + wave; quad < nquads; quad += (int64_t)gridDim.x * kWaves) {
    const int64_t r0 = quad * kRows;
    float acc[kRows][M];
#pragma unroll
    for (int r = 0; r < kRows; ++r)
#pragma unroll
      for (int m = 0; m < M; ++m) acc[r][m] = 0.f;

    for (int c = lane; c < nchunk; c += kWave) {
      const int64_t kc = k0 + 32 * (int64_t)c;
      const int64_t g = kc >> 7;
      u32x4 wq[kRows];
      uint32_t zb[kRows];
      float s[kRows];
#pragma unroll
      for (int r = 0; r < kRows; ++r) {
        const int64_t row = (r0 + r) < n ? (r0 + r) : (n - 1);
        wq[r] = *reinterpret_cast<const u32x4*>(codes + row * (k >> 1) + (kc >> 1));
        s[r] = f16_bits_to_f32(scales[row * groups + g]);
        zb[r] = zeros[row * groups + g];
      }
      // (q - z) as exact half2 values for the 4 words of each row.  The masks
      // and magic constants live in VGPRs so that each mask-and-insert is a
      // single v_and_or_b32 (a VOP3 encoding cannot carry two literals).
      uint32_t mlo = 0x000F000Fu, mhi = 0x00F000F0u, k1024 = 0x64006400u, k64 = 0x54005400u;
      asm("" : "+v"(mlo), "+v"(mhi), "+v"(k1024), "+v"(k64));
      half2_t dq[kRows][16];
#pragma unroll
      for (int r = 0; r < kRows; ++r) {
        const half2_t z2 = __builtin_bit_cast(half2_t, zb[r] | (zb[r] << 16));
        const half2_t c1024 = z2 + half2_t{(half_t)1024.0f, (half_t)1024.0f};
        const half2_t c64 = z2 + half2_t{(half_t)64.0f, (half_t)64.0f};
#pragma unroll
        for (int wd = 0; wd < 4; ++wd) {
          const uint32_t q = wq[r][wd];
          const uint32_t q8 = q >> 8;
          dq[r][4 * wd + 0] = __builtin_bit_cast(half2_t, (q & mlo) | k1024) - c1024;   // q0, q4
          dq[r][4 * wd + 1] = __builtin_bit_cast(half2_t, (q & mhi) | k64) - c64;       // q1, q5
          dq[r][4 * wd + 2] = __builtin_bit_cast(half2_t, (q8 & mlo) | k1024) - c1024;  // q2, q6
          dq[r][4 * wd + 3] = __builtin_bit_cast(half2_t, (q8 & mhi) | k64) - c64;      // q3, q7
        }
      }
#pragma unroll
      for (int m = 0; m < M; ++m) {
        half2_t xv[16];
#pragma unroll
        for (int wd = 0; wd < 4; ++wd) {
          const half2_t* xp = reinterpret_cast<const half2_t*>(xs + (((size_t)m * 4 + wd) * nchunk + c) * 8);
#pragma unroll
          for (int i = 0; i < 4; ++i) xv[4 * wd + i] = xp[i];
        }
#pragma unroll
        for (int r = 0; r < kRows; ++r) {
          float a = 0.f;
#pragma unroll
          for (int i = 0; i < 16; ++i) a = __builtin_amdgcn_fdot2(dq[r][i], xv[i], a, false);
          acc[r][m] += s[r] * a;
        }
      }
    }
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
#pragma unroll
      for (int m = 0; m < M; ++m) {
        const float v = wave_sum(acc[r][m]);
        if (lane == 0 && r0 + r < n) {
          if (partial)
            partial[((int64_t)split * M + m) * n + r0 + r] = v;
          else
            store_out<F16Out>(y, (int64_t)m * n + r0 + r, v);
        }
      }
    }
  }
}

// ------------------------------------------------------------------ FP8 ----
// LDS layout: xs [M][2 halves of the chunk][nchunk][8 halves], natural order.
template <int M, bool F16Out>
__global__ __launch_bounds__(kThreads) void gemv_w8_kernel(const uint16_t* __restrict__ x, int64_t k, int64_t kslice,
                                                           const uint8_t* __restrict__ codes,
                                                           const float* __restrict__ scales, int64_t n,
                                                           void* __restrict__ y, float* __restrict__ partial) {
  extern __shared__ __align__(16) char smem[];
  const int split = blockIdx.y;
  const int64_t k0 = (int64_t)split * kslice;
  const int64_t kl = (k - k0) < kslice ? (k - k0) : kslice;
  const int nchunk = (int)(kl / 16);
  half_t* xs = reinterpret_cast<half_t*>(smem);
  for (int idx = threadIdx.x; idx < nchunk * M * 2; idx += kThreads) {
    const int c = idx / (2 * M), rem = idx % (2 * M), m = rem >> 1, h = rem & 1;
    *reinterpret_cast<u32x4*>(xs + (((size_t)m * 2 + h) * nchunk + c) * 8) =
        *reinterpret_cast<const u32x4*>(x + (int64_t)m * k + k0 + 16 * c + 8 * h);
  }
  __syncthreads();

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t nquads = (n + kRows - 1) / kRows;
  for (int64_t quad = (int64_t)blockIdx.x * kWaves + wave; quad < nquads; quad += (int64_t)gridDim.x * kWaves) {
    const int64_t r0 = quad * kRows;
    float acc[kRows][M];
#pragma unroll
    for (int r = 0; r < kRows; ++r)
#pragma unroll
      for (int m = 0; m < M; ++m) acc[r][m] = 0.f;

    for (int c = lane; c < nchunk; c += kWave) {
      const int64_t kc = k0 + 16 * (int64_t)c;
      half2_t wv[kRows][8];
#pragma unroll
      for (int r = 0; r < kRows; ++r) {
        const int64_t row = (r0 + r) < n ? (r0 + r) : (n - 1);
        const u32x4 q = *reinterpret_cast<const u32x4*>(codes + row * k + kc);
#pragma unroll
        for (int wd = 0; wd < 4; ++wd) {
          wv[r][2 * wd + 0] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(q[wd], 1.0f, false);
          wv[r][2 * wd + 1] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(q[wd], 1.0f, true);
        }
      }
#pragma unroll
      for (int m = 0; m < M; ++m) {
        half2_t xv[8];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const half2_t* xp = reinterpret_cast<const half2_t*>(xs + (((size_t)m * 2 + h) * nchunk + c) * 8);
#pragma unroll
          for (int i = 0; i < 4; ++i) xv[4 * h + i] = xp[i];
        }
#pragma unroll
        for (int r = 0; r < kRows; ++r) {
          float a = acc[r][m];
#pragma unroll
          for (int i = 0; i < 8; ++i) a = __builtin_amdgcn_fdot2(wv[r][i], xv[i], a, false);
          acc[r][m] = a;
        }
      }
    }
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      const int64_t row = (r0 + r) < n ? (r0 + r) : (n - 1);
      const float sc = scales[row];
#pragma unroll
      for (int m = 0; m < M; ++m) {
        const float v = wave_sum(acc[r][m]);
        if (lane == 0 && r0 + r < n) {
          if (partial)
            partial[((int64_t)split * M + m) * n + r0 + r] = v * sc;
          else
            store_out<F16Out>(y, (int64_t)m * n + r0 + r, v * sc);
        }
      }
    }
  }
}

template <bool F16Out>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ partial, int splits, int64_t mn,
                                                            void* __restrict__ y) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < mn; i += (int64_t)gridDim.x * 256) {
    float v = 0.f;
    for (int s = 0; s < splits; ++s) v += partial[(int64_t)s * mn + i];
    store_out<F16Out>(y, i, v);
  }
}

// ------------------------------------------------------------ launching ----
struct Plan {
  int splits;
  int64_t kslice;
  unsigned grid_x;
  size_t lds;
};

// Split K when the activations of a full row do not fit the LDS budget, or
// when there are too few row quads to give every CU work.
Plan make_plan(int64_t n, int64_t k, int64_t kgrain, size_t lds_per_grain, int64_t target_blocks) {
  Plan p;
  const int64_t kmax = (int64_t)(kLdsBudget / lds_per_grain) * kgrain;
  const int64_t nquads = (n + kRows - 1) / kRows;
  const int64_t blocks_x = (nquads + kWaves - 1) / kWaves;
  const int64_t splits_min = (k + kmax - 1) / kmax;
  int64_t splits = splits_min;
  if (blocks_x * splits < target_blocks) {
    const int64_t want = (target_blocks + blocks_x - 1) / blocks_x;
    const int64_t most = k / (4 * kgrain) > 1 ? k / (4 * kgrain) : 1;  // keep >= 4 grains per split
    const int64_t extra = want < most ? want : most;
    splits = extra > splits_min ? extra : splits_min;
  }
  int64_t kslice = (k + splits - 1) / splits;
  kslice = (kslice + kgrain - 1) / kgrain * kgrain;
  p.splits = (int)((k + kslice - 1) / kslice);
  p.kslice = kslice;
  p.grid_x = (unsigned)(blocks_x < 65535 ? blocks_x : 65535);
  p.lds = (size_t)(kslice / kgrain) * lds_per_grain;
  return p;
}

template <int M>
hipError_t gemv_w4_m(const uint16_t* x, int64_t k, const uint8_t* codes, const uint16_t* scales,
                     const uint16_t* zeros, int64_t n, void* y, bool f16_out, hipStream_t stream) {
  // per 128 k: 4 chunks x M x 64 B of permuted x
  const size_t lds_per_grain = (size_t)4 * M * 64;
  const Plan p = make_plan(n, k, 128, lds_per_grain, 512);
  float* partial = nullptr;
  if (p.splits > 1) {
    partial = static_cast<float*>(workspace((size_t)p.splits * M * n * sizeof(float)));
    if (!partial) return hipErrorOutOfMemory;
  }
  const dim3 grid(p.grid_x, p.splits);
  if (f16_out)
    hipLaunchKernelGGL((gemv_w4_kernel<M, true>), grid, dim3(kThreads), p.lds, stream, x, k, p.kslice, codes, scales,
                       zeros, n, y, partial);
  else
    hipLaunchKernelGGL((gemv_w4_kernel<M, false>), grid, dim3(kThreads), p.lds, stream, x, k, p.kslice, codes,
                       scales, zeros, n, y, partial);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || p.splits == 1) return err;
  return launch_splitk_reduce(partial, p.splits, (int64_t)M * n, y, f16_out, stream);
}

template <int M>
hipError_t gemv_w8_m(const uint16_t* x, int64_t k, const uint8_t* codes, const float* scales, int64_t n, void* y,
                     bool f16_out, hipStream_t stream) {
  // per 16 k: one chunk x M x 32 B of x
  const size_t lds_per_grain = (size_t)M * 32;
  const Plan p = make_plan(n, k, 16, lds_per_grain, 512);
  float* partial = nullptr;
  if (p.splits > 1) {
    partial = static_cast<float*>(workspace((size_t)p.splits * M * n * sizeof(float)));
    if (!partial) return hipErrorOutOfMemory;
  }
  const dim3 grid(p.grid_x, p.splits);
  if (f16_out)
    hipLaunchKernelGGL((gemv_w8_kernel<M, true>), grid, dim3(kThreads), p.lds, stream, x, k, p.kslice, codes, scales,
                       n, y, partial);
  else
    hipLaunchKernelGGL((gemv_w8_kernel<M, false>), grid, dim3(kThreads), p.lds, stream, x, k, p.kslice, codes,
                       scales, n, y, partial);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || p.splits == 1) return err;
  return launch_splitk_reduce(partial, p.splits, (int64_t)M * n, y, f16_out, stream);
}

}  // namespace

hipError_t launch_splitk_reduce(const float* partial, int splits, int64_t mn, void* y, bool f16_out,
                                hipStream_t stream) {
  int64_t blocks = (mn + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (f16_out)
    hipLaunchKernelGGL(splitk_reduce_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, stream, partial, splits, mn,
                       y);
  else
    hipLaunchKernelGGL(splitk_reduce_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, stream, partial, splits, mn,
                       y);
  return hipGetLastError();
}

hipError_t launch_gemv_w4(const uint16_t* x, int m, int64_t k, const uint8_t* codes, const uint16_t* scales,
                          const uint16_t* zeros, int64_t n, void* y, bool f16_out, hipStream_t stream) {
  switch (m) {
    case 1: return gemv_w4_m<1>(x, k, codes, scales, zeros, n, y, f16_out, stream);
    case 2: return gemv_w4_m<2>(x, k, codes, scales, zeros, n, y, f16_out, stream);
    case 3: return gemv_w4_m<3>(x, k, codes, scales, zeros, n, y, f16_out, stream);
    case 4: return gemv_w4_m<4>(x, k, codes, scales, zeros, n, y, f16_out, stream);
    case 5: return gemv_w4_m<5>(x, k, codes, scales, zeros, n, y, f16_out, stream);
    case 6: return gemv_w4_m<6>(x, k, codes, scales, zeros, n, y, f16_out, stream);
    case 7: return gemv_w4_m<7>(x, k, codes, scales, zeros, n, y, f16_out, stream);
    case 8: return gemv_w4_m<8>(x, k, codes, scales, zeros, n, y, f16_out, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemv_w8(const uint16_t* x, int m, int64_t k, const uint8_t* codes, const float* scales, int64_t n,
                          void* y, bool f16_out, hipStream_t stream) {
  switch (m) {
    case 1: return gemv_w8_m<1>(x, k, codes, scales, n, y, f16_out, stream);
    case 2: return gemv_w8_m<2>(x, k, codes, scales, n, y, f16_out, stream);
    case 3: return gemv_w8_m<3>(x, k, codes, scales, n, y, f16_out, stream);
    case 4: return gemv_w8_m<4>(x, k, codes, scales, n, y, f16_out, stream);
    case 5: return gemv_w8_m<5>(x, k, codes, scales, n, y, f16_out, stream);
    case 6: return gemv_w8_m<6>(x, k, codes, scales, n, y, f16_out, stream);
    case 7: return gemv_w8_m<7>(x, k, codes, scales, n, y, f16_out, stream);
    case 8: return gemv_w8_m<8>(x, k, codes, scales, n, y, f16_out, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace sq

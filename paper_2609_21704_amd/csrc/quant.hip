// Offline derivation of the quantized draft parents from the FP16 parent
// (SpecQuant SS III-A.1: Q4 = f(W16, 4); SS III-A.2: Q8 = f(W16, 8)).
//
// Both quantizers do their arithmetic in fp64 with IEEE division and
// round-to-nearest-even, without contraction, so the produced bytes are a
// deterministic function of the FP16 input.  Both are HBM-bound streaming
// kernels: 2 B read per weight, 17/32 B (INT4 g128) or 1 B (FP8) written.
#include "sq_device.hpp"
#include "sq_internal.hpp"

#pragma clang fp contract(off)

namespace sq {
namespace {

__device__ __forceinline__ double f16_bits_to_f64(uint32_t h) {
  return (double)__builtin_bit_cast(half_t, (uint16_t)h);
}

// Smallest binary16 value >= s for a finite s > 0 that is a normal double.
// The binary16 grid near s has spacing 2^(e-10) (e = floor(log2 s) >= -14) or
// 2^-24 (subnormal range); scaling by that spacing is exact, so ceil() picks
// the next grid point exactly.
__device__ __forceinline__ double f16_ceil(double s) {
  const uint64_t bits = (uint64_t)__double_as_longlong(s);
  const int e = (int)((bits >> 52) & 0x7FF) - 1023;
  const int sp = (e < -14) ? -24 : e - 10;
  return ldexp(ceil(ldexp(s, -sp)), sp);
}

// One group's quantization, by its 16 consecutive lanes (sub = 0 .. 15).
__device__ __forceinline__ void quantize_int4_group(const uint16_t* __restrict__ w, int64_t ngroups, int64_t gi,
                                                    int sub, uint8_t* __restrict__ codes,
                                                    uint16_t* __restrict__ scales, uint16_t* __restrict__ zeros,
                                                    int32_t* flag) {
  const bool active = gi < ngroups;
  u32x4 raw = {0u, 0u, 0u, 0u};
  if (active) raw = *reinterpret_cast<const u32x4*>(w + gi * 128 + sub * 8);

  double v[8];
  bool bad = false;
  double lo = 0.0, hi = 0.0;  // the range always contains zero
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t h = (raw[i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
    bad |= (h & 0x7C00u) == 0x7C00u;
    v[i] = f16_bits_to_f64(h);
    lo = v[i] < lo ? v[i] : lo;
    hi = v[i] > hi ? v[i] : hi;
  }
  // the 16 threads of a group are consecutive lanes of one wavefront
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1) {
    const double olo = __shfl_xor(lo, off, 16);
    const double ohi = __shfl_xor(hi, off, 16);
    lo = olo < lo ? olo : lo;
    hi = ohi > hi ? ohi : hi;
    bad |= __shfl_xor((int)bad, off, 16) != 0;
  }
  if (!active) return;  // whole 16-lane groups only: no shuffle follows

  uint32_t packed = 0;
  uint16_t sbits, zbits;
  if (bad) {
    sbits = 0x7E00;  // NaN scale marks the group
    zbits = 0;
    if (sub == 0 && flag) atomicOr(flag, 1);
  } else if (hi == lo) {
    sbits = 0x3C00;  // 1.0
    zbits = 0;
  } else {
    const double s16 = f16_ceil((hi - lo) / 15.0);
    double z = rint(-lo / s16);
    z = z > 0.0 ? (z > 15.0 ? 15.0 : z) : 0.0;  // also maps -0.0 (lo == 0) to +0.0
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      double c = rint(v[i] / s16) + z;
      c = c < 0.0 ? 0.0 : (c > 15.0 ? 15.0 : c);
      packed |= (uint32_t)c << (4 * i);  // element i -> byte i/2, nibble i%2
    }
    // s16 and z are exactly representable in binary16
    sbits = f32_to_f16_bits((float)s16);
    zbits = f32_to_f16_bits((float)z);
  }
  reinterpret_cast<uint32_t*>(codes + gi * 64)[sub] = packed;
  if (sub == 0) {
    scales[gi] = sbits;
    zeros[gi] = zbits;
  }
}

// INT4 g128: 16 threads per group of 128 elements, 8 elements (16 B) each;
// a workgroup handles 16 consecutive groups per pass of its grid-stride loop.
// Groups are contiguous in memory because k % 128 == 0, so group gi starts at
// element 128 * gi and its 64 code bytes at byte 64 * gi.
__global__ __launch_bounds__(256) void quantize_int4_kernel(const uint16_t* __restrict__ w, int64_t ngroups,
                                                            uint8_t* __restrict__ codes,
                                                            uint16_t* __restrict__ scales,
                                                            uint16_t* __restrict__ zeros, int32_t* flag) {
  for (int64_t gbase = (int64_t)blockIdx.x * 16; gbase < ngroups; gbase += (int64_t)gridDim.x * 16)
    quantize_int4_group(w, ngroups, gbase + (threadIdx.x >> 4), threadIdx.x & 15, codes, scales, zeros, flag);
}

// OCP E4M3 encode of a finite double: round to nearest, ties to even,
// saturating to +-448, sign of zero kept.  Normal results round the 52-bit
// fraction to 3 bits with integer arithmetic; the subnormal grid (multiples of
// 2^-9 below 2^-6) uses rint on an exactly scaled value.
__device__ __forceinline__ uint32_t e4m3_encode(double v) {
  const uint64_t bits = (uint64_t)__double_as_longlong(v);
  const uint32_t sign = (uint32_t)(bits >> 63) << 7;
  const uint64_t mag = bits & 0x7FFFFFFFFFFFFFFFull;
  const double a = __longlong_as_double((long long)mag);
  uint32_t code;
  if (a > 448.0) {
    code = 0x7E;
  } else if (a < 0.015625) {
    code = (uint32_t)rint(a * 512.0);  // 8 here is the smallest normal, 0x08
  } else {
    const int e = (int)(mag >> 52) - 1023;  // -6 .. 8
    const uint64_t frac = mag & ((1ull << 52) - 1);
    uint64_t r = frac >> 49;
    const uint64_t rem = frac & ((1ull << 49) - 1);
    const uint64_t halfway = 1ull << 48;
    if (rem > halfway || (rem == halfway && (r & 1))) r += 1;  // a carry bumps the exponent
    code = ((uint32_t)(e + 7) << 3) + (uint32_t)r;
  }
  if (code > 0x7E) code = 0x7E;
  return sign | code;
}

// FP8: one workgroup per row (grid-stride), two passes over the row: the
// fp16 magnitude maximum (bit patterns of finite fp16 magnitudes are ordered),
// then the encode.  k % 16 == 0, so every 16-B load and 8-B store is aligned.
__global__ __launch_bounds__(256) void quantize_fp8_kernel(const uint16_t* __restrict__ w, int64_t n, int64_t k,
                                                           uint8_t* __restrict__ codes, float* __restrict__ scales,
                                                           int32_t* flag) {
  __shared__ uint32_t red[4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int64_t row = blockIdx.x; row < n; row += gridDim.x) {
    const uint16_t* src = w + row * k;
    uint32_t amax = 0;
    for (int64_t c = (int64_t)threadIdx.x * 8; c < k; c += 256 * 8) {
      const u32x4 raw = *reinterpret_cast<const u32x4*>(src + c);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint32_t h = (raw[i >> 1] >> (16 * (i & 1))) & 0x7FFFu;
        amax = h > amax ? h : amax;  // non-finite magnitudes (>= 0x7C00) dominate
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const uint32_t o = __shfl_xor(amax, off, 64);
      amax = o > amax ? o : amax;
    }
    if (lane == 0) red[wave] = amax;
    __syncthreads();
    amax = red[0];
#pragma unroll
    for (int i = 1; i < 4; ++i) amax = red[i] > amax ? red[i] : amax;
    __syncthreads();  // red[] is reused by the next row

    uint8_t* dst = codes + row * k;
    if (amax >= 0x7C00u) {  // NaN or Inf somewhere in the row
      for (int64_t c = (int64_t)threadIdx.x * 8; c < k; c += 256 * 8)
        *reinterpret_cast<uint64_t*>(dst + c) = 0;
      if (threadIdx.x == 0) {
        scales[row] = __builtin_nanf("");
        if (flag) atomicOr(flag, 1);
      }
      continue;
    }
    const double am = f16_bits_to_f64(amax);
    const float s = (amax == 0) ? 1.0f : (float)(am / 448.0);
    const double sd = (double)s;
    if (threadIdx.x == 0) scales[row] = s;
    for (int64_t c = (int64_t)threadIdx.x * 8; c < k; c += 256 * 8) {
      const u32x4 raw = *reinterpret_cast<const u32x4*>(src + c);
      uint64_t out = 0;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint32_t h = (raw[i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
        out |= (uint64_t)e4m3_encode(f16_bits_to_f64(h) / sd) << (8 * i);
      }
      *reinterpret_cast<uint64_t*>(dst + c) = out;
    }
  }
}

}  // namespace

hipError_t launch_quantize_int4(const uint16_t* w, int64_t n, int64_t k, uint8_t* codes, uint16_t* scales,
                                uint16_t* zeros, int32_t* flag, hipStream_t stream) {
  const int64_t ngroups = n * (k / 128);
  const int64_t need = (ngroups + 15) / 16;
  const int64_t blocks = need < 65536 * 16 ? need : 65536 * 16;
  hipLaunchKernelGGL(quantize_int4_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, w, ngroups, codes, scales,
                     zeros, flag);
  return hipGetLastError();
}

hipError_t launch_quantize_fp8(const uint16_t* w, int64_t n, int64_t k, uint8_t* codes, float* scales,
                               int32_t* flag, hipStream_t stream) {
  const int64_t blocks = n < 65536 * 16 ? n : 65536 * 16;
  hipLaunchKernelGGL(quantize_fp8_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, w, n, k, codes, scales,
                     flag);
  return hipGetLastError();
}

}  // namespace sq

// Streaming-read probe: a diagnostic beside the method, not a step of it.
// It reads a buffer once with 16-byte loads in grid-stride order (each load
// instruction of a wavefront covers 1 KiB of consecutive bytes) and does
// nothing else, so the duration of a launch is what a plain read of that many
// bytes costs on the device: the measured ceiling the HBM-bound kernels are
// compared against.  Every word read enters an XOR per workgroup, which is
// written out so that no load can be dropped.  Shape (measured over 8.8 MB ..
// 4 GiB reads): 2048 workgroups of 256 threads, one load in flight per lane;
// four loads in flight per lane were up to 14 % slower, and 1024 workgroups
// up to 9 %.
#include "sq_device.hpp"
#include "sq_internal.hpp"

namespace sq {
namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeUnroll = 1;

__global__ __launch_bounds__(kProbeThreads) void stream_read_kernel(const u32x4* __restrict__ src, int64_t cells,
                                                                     uint32_t* __restrict__ sink) {
  const int64_t stride = (int64_t)gridDim.x * kProbeThreads;
  uint32_t acc = 0;
  for (int64_t i = (int64_t)blockIdx.x * kProbeThreads + threadIdx.x; i < cells; i += kProbeUnroll * stride) {
    u32x4 v[kProbeUnroll];
#pragma unroll
    for (int j = 0; j < kProbeUnroll; ++j) {
      const int64_t t = i + j * stride;
      v[j] = t < cells ? src[t] : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int j = 0; j < kProbeUnroll; ++j) acc ^= v[j][0] ^ v[j][1] ^ v[j][2] ^ v[j][3];
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, o, 64);
  __shared__ uint32_t part[kProbeThreads / 64];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t w = 0;
#pragma unroll
    for (int i = 0; i < kProbeThreads / 64; ++i) w ^= part[i];
    sink[blockIdx.x] = w;
  }
}

}  // namespace

hipError_t launch_stream_read(const void* src, int64_t bytes, uint32_t* sink, int blocks, hipStream_t stream) {
  hipLaunchKernelGGL(stream_read_kernel, dim3((unsigned)blocks), dim3(kProbeThreads), 0, stream,
                     static_cast<const u32x4*>(src), bytes / 16, sink);
  return hipGetLastError();
}

}  // namespace sq

// Parent verification GEMM with the FP16 parent (SpecQuant SS III-D.3: the
// parent Q16 = W16 checks all drafted positions of a block in one pass).
//
// y[m][n] = sum_c x[m][c] * W[n][c] with m = b * (kd + 1) rows (5 to 36 at the
// configurations of interest).  The weight stream dominates (2 bytes per
// weight, read once); at m = 36 the contraction exceeds what the vector ALUs
// can sustain at HBM speed, so it runs on the matrix cores:
// v_mfma_f32_16x16x32_f16, with the m rows padded to 16-row tiles.
//
// Operand mapping (16x16x32, wave64): lane l holds A[l%16][8(l/16) .. +8) and
// B[8(l/16) .. +8)[l%16]; the result lane l holds D[4(l/16) + r][l%16].  A is
// the activation tile (rows m), B the weight tile (B[c][j] = W[n0 + j][c]).
// A lane loads 64 contiguous bytes of one weight row per 128-wide k step, so
// four lanes cover 256 contiguous bytes of a row; MFMA t (t = 0..3) consumes
// the lane's k offsets 32(l/16) + 8t .. +8, and the A fragment is read with
// the same k permutation, which leaves the sum unchanged.
//
// A workgroup owns 16 weight rows; its four wavefronts take interleaved 128-wide
// k steps of the workgroup's K slice (two steps in flight per iteration) and
// are summed through LDS in wavefront order.  Small-n matrices are also split
// along K across workgroups, with a deterministic second pass.
#include "sq_device.hpp"
#include "sq_internal.hpp"

namespace sq {
namespace {

constexpr int kThreads = 256;
constexpr int kStep = 128;              // k elements per wavefront step
constexpr int kUnroll = 2;              // steps in flight per wavefront

__device__ __forceinline__ half8_t load_h8(const uint16_t* p) {
  return __builtin_bit_cast(half8_t, *reinterpret_cast<const u32x4*>(p));
}

template <int MT, bool F16Out>
__global__ __launch_bounds__(kThreads) void gemm_f16_kernel(const uint16_t* __restrict__ x, int m_rows, int64_t k,
                                                            const uint16_t* __restrict__ w, int64_t n, int64_t kslice,
                                                            void* __restrict__ y, float* __restrict__ partial) {
  __shared__ float red[4][MT * 256];
  const int split = blockIdx.y;
  const int64_t k0 = (int64_t)split * kslice;
  const int64_t kl = (k - k0) < kslice ? (k - k0) : kslice;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int li = lane & 15, lk = lane >> 4;
  const int64_t n0 = (int64_t)blockIdx.x * 16;
  const int64_t row = (n0 + li) < n ? (n0 + li) : (n - 1);
  const uint16_t* wrow = w + row * k + k0;

  float4_t acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt] = float4_t{0.f, 0.f, 0.f, 0.f};
  const half8_t zero8 = {};

  for (int64_t kk = (int64_t)wave * kStep; kk < kl; kk += 4 * kStep * kUnroll) {
    half8_t b[kUnroll][4];
    half8_t a[kUnroll][MT][4];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int64_t kidx = kk + (int64_t)u * 4 * kStep + 32 * lk + 8 * t;
        b[u][t] = kidx < kl ? load_h8(wrow + kidx) : zero8;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const int mr = mt * 16 + li;
          a[u][mt][t] = (mr < m_rows && kidx < kl) ? load_h8(x + (int64_t)mr * k + k0 + kidx) : zero8;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
          acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[u][mt][t], b[u][t], acc[mt], 0, 0, 0);
  }

#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) red[wave][(mt * 4 + r) * 64 + lane] = acc[mt][r];
  __syncthreads();
  for (int idx = threadIdx.x; idx < MT * 256; idx += kThreads) {
    const float v = ((red[0][idx] + red[1][idx]) + red[2][idx]) + red[3][idx];
    const int mt = idx >> 8, r = (idx >> 6) & 3, l = idx & 63;
    const int mr = mt * 16 + 4 * (l >> 4) + r;
    const int64_t col = n0 + (l & 15);
    if (mr < m_rows && col < n) {
      if (partial)
        partial[((int64_t)split * m_rows + mr) * n + col] = v;
      else
        store_out<F16Out>(y, (int64_t)mr * n + col, v);
    }
  }
}

template <int MT>
hipError_t gemm_mt(const uint16_t* x, int m, int64_t k, const uint16_t* w, int64_t n, void* y, bool f16_out,
                   hipStream_t stream) {
  const int64_t blocks_x = (n + 15) / 16;
  const int64_t target = 512;
  int64_t splits = 1;
  if (blocks_x < target) {
    const int64_t want = (target + blocks_x - 1) / blocks_x;
    const int64_t most = k / (4 * kStep * kUnroll) > 1 ? k / (4 * kStep * kUnroll) : 1;
    splits = want < most ? want : most;
  }
  int64_t kslice = (k + splits - 1) / splits;
  kslice = (kslice + kStep - 1) / kStep * kStep;
  splits = (k + kslice - 1) / kslice;
  float* partial = nullptr;
  if (splits > 1) {
    partial = static_cast<float*>(workspace((size_t)splits * m * n * sizeof(float)));
    if (!partial) return hipErrorOutOfMemory;
  }
  if (blocks_x > 0x7FFFFFFF) return hipErrorInvalidValue;
  const dim3 grid((unsigned)blocks_x, (unsigned)splits);
  if (f16_out)
    hipLaunchKernelGGL((gemm_f16_kernel<MT, true>), grid, dim3(kThreads), 0, stream, x, m, k, w, n, kslice, y,
                       partial);
  else
    hipLaunchKernelGGL((gemm_f16_kernel<MT, false>), grid, dim3(kThreads), 0, stream, x, m, k, w, n, kslice, y,
                       partial);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || splits == 1) return err;
  return launch_splitk_reduce(partial, (int)splits, (int64_t)m * n, y, f16_out, stream);
}

}  // namespace

hipError_t launch_gemm_f16(const uint16_t* x, int m, int64_t k, const uint16_t* w, int64_t n, void* y, bool f16_out,
                           hipStream_t stream) {
  if (m <= 16) return gemm_mt<1>(x, m, k, w, n, y, f16_out, stream);
  if (m <= 32) return gemm_mt<2>(x, m, k, w, n, y, f16_out, stream);
  if (m <= 48) return gemm_mt<3>(x, m, k, w, n, y, f16_out, stream);
  if (m <= 64) return gemm_mt<4>(x, m, k, w, n, y, f16_out, stream);
  return hipErrorInvalidValue;
}

}  // namespace sq

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
// The grid is persistent: a workgroup walks 16-row tiles; its four wavefronts
// split each tile's K into interleaved 128-wide steps and fetch the next
// item's operands while the matrix cores work on the current one.  The four
// partial tiles are summed through LDS in wavefront order.
#include "sq_device.hpp"
#include "sq_internal.hpp"

namespace sq {
namespace {

constexpr int kThreads = 256;
constexpr int kStep = 128;  // k elements per wavefront step

__device__ __forceinline__ half8_t load_h8(const uint16_t* p) {
  return __builtin_bit_cast(half8_t, *reinterpret_cast<const u32x4*>(p));
}

template <int MT, int U>
struct Item {
  half8_t b[U][4];       // weight fragments
  half8_t a[U][MT][4];   // activation fragments
};

// Operands of item j of a tile for this wavefront: steps (j U + u) * 4 + wave.
template <int MT, int U>
__device__ __forceinline__ void load_item(Item<MT, U>& it, const uint16_t* __restrict__ x, int m_rows, int64_t k,
                                          const uint16_t* __restrict__ w, int64_t n, int64_t tile, int j, int wave,
                                          int li, int lk) {
  const int64_t row = (tile * 16 + li) < n ? (tile * 16 + li) : (n - 1);
  const uint16_t* wrow = w + row * k;
  const half8_t zero8 = {};
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t step = ((int64_t)j * U + u) * 4 + wave;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int64_t kidx = step * kStep + 32 * lk + 8 * t;
      const bool ok = kidx < k;
      it.b[u][t] = ok ? load_h8(wrow + kidx) : zero8;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int mr = mt * 16 + li;
        it.a[u][mt][t] = (ok && mr < m_rows) ? load_h8(x + (int64_t)mr * k + kidx) : zero8;
      }
    }
  }
}

template <int MT, int U, bool F16Out>
__global__ __launch_bounds__(kThreads) void gemm_f16_kernel(const uint16_t* __restrict__ x, int m_rows, int64_t k,
                                                            const uint16_t* __restrict__ w, int64_t n,
                                                            void* __restrict__ y) {
  __shared__ float red[4][MT * 256];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int li = lane & 15, lk = lane >> 4;
  const int64_t ntile = (n + 15) / 16;
  const int64_t nsteps = (k + kStep - 1) / kStep;
  const int nitem = (int)((nsteps + 4 * U - 1) / (4 * U));  // the same for every wavefront
  int64_t tile = blockIdx.x;
  int j = 0;
  if (tile >= ntile) return;  // uniform across the workgroup

  Item<MT, U> cur;
  load_item<MT, U>(cur, x, m_rows, k, w, n, tile, 0, wave, li, lk);
  float4_t acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt] = float4_t{0.f, 0.f, 0.f, 0.f};

  while (true) {
    int64_t tile_n = tile;
    int j_n = j + 1;
    if (j_n == nitem) {
      j_n = 0;
      tile_n = tile + gridDim.x;
    }
    Item<MT, U> nxt;
    if (tile_n < ntile) load_item<MT, U>(nxt, x, m_rows, k, w, n, tile_n, j_n, wave, li, lk);

#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
          acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(cur.a[u][mt][t], cur.b[u][t], acc[mt], 0, 0, 0);

    if (j == nitem - 1) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
        for (int r = 0; r < 4; ++r) red[wave][(mt * 4 + r) * 64 + lane] = acc[mt][r];
        acc[mt] = float4_t{0.f, 0.f, 0.f, 0.f};
      }
      __syncthreads();
      const int64_t n0 = tile * 16;
      for (int idx = threadIdx.x; idx < MT * 256; idx += kThreads) {
        const float v = ((red[0][idx] + red[1][idx]) + red[2][idx]) + red[3][idx];
        const int mt = idx >> 8, r = (idx >> 6) & 3, l = idx & 63;
        const int mr = mt * 16 + 4 * (l >> 4) + r;
        const int64_t col = n0 + (l & 15);
        if (mr < m_rows && col < n) store_out<F16Out>(y, (int64_t)mr * n + col, v);
      }
      __syncthreads();
    }
    if (tile_n >= ntile) break;
    tile = tile_n;
    j = j_n;
    cur = nxt;
  }
}

template <int MT, int U>
hipError_t gemm_mt(const uint16_t* x, int m, int64_t k, const uint16_t* w, int64_t n, void* y, bool f16_out,
                   hipStream_t stream) {
  const int64_t ntile = (n + 15) / 16;
  const int64_t cap = (int64_t)cu_count() * 4;
  const dim3 grid((unsigned)(ntile < cap ? ntile : cap));
  if (f16_out)
    hipLaunchKernelGGL((gemm_f16_kernel<MT, U, true>), grid, dim3(kThreads), 0, stream, x, m, k, w, n, y);
  else
    hipLaunchKernelGGL((gemm_f16_kernel<MT, U, false>), grid, dim3(kThreads), 0, stream, x, m, k, w, n, y);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_f16(const uint16_t* x, int m, int64_t k, const uint16_t* w, int64_t n, void* y, bool f16_out,
                           hipStream_t stream) {
  if (m <= 16) return gemm_mt<1, 2>(x, m, k, w, n, y, f16_out, stream);
  if (m <= 32) return gemm_mt<2, 1>(x, m, k, w, n, y, f16_out, stream);
  if (m <= 48) return gemm_mt<3, 1>(x, m, k, w, n, y, f16_out, stream);
  if (m <= 64) return gemm_mt<4, 1>(x, m, k, w, n, y, f16_out, stream);
  return hipErrorInvalidValue;
}

}  // namespace sq

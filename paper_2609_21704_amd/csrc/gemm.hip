// Parent verification GEMM with the FP16 parent (SpecQuant SS III-D.3: the
// parent Q16 = W16 checks all drafted positions of a block in one pass).
// Two kernels here: gemm_rows_kernel (m <= 8, row blocks on the vector ALUs,
// described at the kernel) and gemm_f16_kernel (the tiled matrix-core GEMM
// below); the large matrices stream through linear_kernel (m <= 16 from
// 28 MiB of weights, m = 17..64 from 4 MiB).
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

// Verification over row blocks for small m (m <= 8): at 5 flops per weight
// byte the contraction is far below the matrix cores' ridge, and v_dot2
// keeps up with HBM (m / 2 instructions per weight), so the weight rows
// stream through the vector ALUs in the split of the INT4 row-block GEMV.  A
// workgroup of NWV wavefronts (16 per CU in all) owns a contiguous block of
// rows, whose weights are one contiguous range of 32-byte pieces (16 weights
// of one row); each wavefront walks a run of whole steps of 64 pieces, the
// odd steps going to the oldest wavefronts.  A row holds at least 32 pieces,
// so a step meets at most NA rows; each lane adds its piece into the sum of
// its row, and when the walk leaves a row the wavefront reduces that row's m
// sums into LDS slots [wavefront][m][row], added in wavefront order after
// one barrier.  The activations sit in LDS as [m][half][piece] cells of 8
// halves, so the 64 lanes of one read take consecutive cells.  When the
// activations of a whole row do not fit, KS = 2 workgroups share each row
// block, one per half of K (blockIdx.y); the two partial sums of a value meet
// in a 64-bit slot by atomic exchange (the value travels inside the atomic, so
// no fence is needed): the second to arrive adds slice 0's + slice 1's in that
// order, stores the result and empties the slot for the next launch.
// Output modes: y fp32, y fp16, or y fp32 added to.
enum : int { kOutF32 = 0, kOutF16 = 1, kOutAcc = 2 };

template <int M, int NA, int NWV, int XB, int D, int KS, bool NRM>
__global__ __launch_bounds__(1024) void gemm_rows_kernel(const uint16_t* __restrict__ x, int64_t k,
                                                        const uint16_t* __restrict__ w, int64_t rows_q,
                                                        int rows_rem, int64_t n, void* __restrict__ y,
                                                        int out_mode, unsigned long long* __restrict__ slots,
                                                        NormSrc nr) {
  // The arguments the first loads need come first: the library is built with
  // the first 14 argument dwords preloaded into scalar registers at dispatch.
  asm volatile("" ::"s"(x), "s"(k), "s"(w), "s"(rows_q), "s"(rows_rem), "s"(n));
  extern __shared__ __align__(16) char smem[];
  constexpr int nwave = NWV, nthr = 64 * NWV;
  const int b = blockIdx.x;
  const int64_t r0 = (int64_t)b * rows_q + (b < rows_rem ? b : rows_rem);
  const int nrows = (int)rows_q + (b < rows_rem ? 1 : 0);
  const int slice = KS > 1 ? (int)blockIdx.y : 0;
  const int64_t kl = k / KS, k0 = slice * kl;  // this workgroup's part of K
  const int ppr = (int)(kl >> 4);  // pieces per row
  const int P = nrows * ppr;       // pieces of the block (< 2^27, or 2^24 when KS > 1, by the host's check)
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // runs of whole steps: sb each, one more for the sx oldest wavefronts
  const int T = (P + 63) >> 6;
  const int sb = T / nwave, sx = T - sb * nwave;  // nwave: a power of two
  const int ps0 = 64 * (wave * sb + (wave < sx ? wave : sx));
  const int ps = ps0 < P ? ps0 : P, pe0 = ps0 + 64 * (sb + (wave < sx ? 1 : 0)), pe = pe0 < P ? pe0 : P;
  const int nsteps = (pe - ps + 63) >> 6;
  half_t* xs = reinterpret_cast<half_t*>(smem);
  // NRM: the rows' wavefront sums of squares [M][4] after the activations, then the row sums
  float* wsum = reinterpret_cast<float*>(smem + (size_t)M * 2 * ppr * 16);
  float* red = reinterpret_cast<float*>(smem + (size_t)M * 2 * ppr * 16 + (NRM ? 128 : 0));  // [nwave][M][nrows]
  const uint16_t* bw = w + r0 * k + k0;
  const float rppr = 1.0f / (float)ppr;

  // piece p of the block: weights 16 p .. 16 p + 15 of the block's range (rows
  // are contiguous; with K slices, row p / ppr at piece p % ppr of the slice);
  // a lane past the run reads the run's last piece again and adds nothing.
  // Unconditional, so the compiler waits only for the oldest.
  struct Piece {
    u32x4 c[2];
  };
  auto load = [&](int s) -> Piece {
    Piece f;
    int p = ps + 64 * s + lane;
    p = p < pe ? p : pe - 1;
    p = p > 0 ? p : 0;  // a run without pieces reads piece 0
    int64_t off = (int64_t)p * 16;
    if constexpr (KS > 1) {  // the float quotient is within one of p / ppr (p < 2^24)
      int ri = (int)((float)p * rppr);
      int ch = p - ri * ppr;
      if (ch < 0) {
        --ri;
        ch += ppr;
      } else if (ch >= ppr) {
        ++ri;
        ch -= ppr;
      }
      off = (int64_t)ri * k + ch * 16;
    }
    const u32x4* cp = reinterpret_cast<const u32x4*>(bw + off);
    f.c[0] = cp[0];
    f.c[1] = cp[1];
    return f;
  };

  // activations first (XB cells per thread cover all of x), then the first step;
  // NRM: the rows' sums of squares first, then the cells' h and norm weights
  const int xtotal = M * 2 * ppr;
  RmsRows<2> rr;  // NRM: M <= 8 rows over the four groups of 256 threads
  if constexpr (NRM) rr.load(nr.h + (int64_t)(nr.group - 1) * k, (int64_t)nr.group * k, M, (int)k);
  u32x4 xv[XB];
  float4_t xh[NRM ? XB : 1][2];
  u32x4 xw[NRM ? XB : 1];
#pragma unroll
  for (int i = 0; i < XB; ++i) {
    int idx = i * nthr + (int)threadIdx.x;
    idx = idx < xtotal ? idx : xtotal - 1;
    int m = 0, c = idx;  // c: 8-element cell of row m
#pragma unroll
    for (int mm = 1; mm < M; ++mm)
      if (c >= 2 * ppr) {
        c -= 2 * ppr;
        m = mm;
      }
    if constexpr (NRM) {
      const float* hr = nr.h + ((int64_t)m * nr.group + nr.group - 1) * k + k0 + 8 * c;
      xh[i][0] = *reinterpret_cast<const float4_t*>(hr);
      xh[i][1] = *reinterpret_cast<const float4_t*>(hr + 4);
      xw[i] = *reinterpret_cast<const u32x4*>(nr.w + k0 + 8 * c);
    } else {
      xv[i] = *reinterpret_cast<const u32x4*>(x + (int64_t)m * k + k0 + 8 * c);
    }
  }
  Piece ring[D];
#pragma unroll
  for (int j = 0; j < D; ++j) ring[j] = load(j);
  if constexpr (NRM) {
    rr.finish(M, (int)k, wsum);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    float r[M];
#pragma unroll
    for (int m = 0; m < M; ++m) r[m] = rms_inverse(wsum + 4 * m, (int)k, nr.eps);
#pragma unroll
    for (int i = 0; i < XB; ++i) {
      int idx = i * nthr + (int)threadIdx.x;
      idx = idx < xtotal ? idx : xtotal - 1;
      int m = 0, c = idx;
#pragma unroll
      for (int mm = 1; mm < M; ++mm)
        if (c >= 2 * ppr) {
          c -= 2 * ppr;
          m = mm;
        }
      float rm = r[0];
#pragma unroll
      for (int mm = 1; mm < M; ++mm) rm = m == mm ? r[mm] : rm;
      xv[i] = rms_cell(xh[i][0], xh[i][1], xw[i], rm);
    }
  }
#pragma unroll
  for (int i = 0; i < XB; ++i) {
    const int idx = i * nthr + (int)threadIdx.x;
    if (idx < xtotal) {
      int m = 0, c = idx;
#pragma unroll
      for (int mm = 1; mm < M; ++mm)
        if (c >= 2 * ppr) {
          c -= 2 * ppr;
          m = mm;
        }
      *reinterpret_cast<u32x4*>(xs + (((size_t)m * 2 + (c & 1)) * ppr + (c >> 1)) * 8) = xv[i];
    }
  }
  for (int i = (int)threadIdx.x; i < nwave * M * nrows; i += nthr) red[i] = 0.f;
  // an accumulated output: this thread's first value read now, its latency under the walk
  float yold = 0.f;
  if (out_mode == kOutAcc && (int)threadIdx.x < M * nrows) {
    int m = 0, row = (int)threadIdx.x;
#pragma unroll
    for (int mm = 1; mm < M; ++mm)
      if (row >= nrows) {
        row -= nrows;
        m = mm;
      }
    yold = reinterpret_cast<const float*>(y)[(int64_t)m * n + r0 + row];
  }
  // LDS writes done, then the barrier: no wait for the weight loads in flight
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();

  // the walk: step base piece `cb`, its row `crow` and offset `coff` in that row
  int cb = ps;
  int crow = (int)((double)ps / (double)ppr);  // exact: both below 2^27
  crow -= crow * ppr > ps ? 1 : 0;
  crow += (crow + 1) * ppr <= ps ? 1 : 0;
  int coff = ps - crow * ppr;
  int cur = crow;  // acc[i] holds row cur + i
  float acc[NA][M];
#pragma unroll
  for (int i = 0; i < NA; ++i)
#pragma unroll
    for (int m = 0; m < M; ++m) acc[i][m] = 0.f;

  auto flush = [&](const float (&a)[M], int row) {
    constexpr int TT = (M + 3) / 4;
    float v[4 * TT];
#pragma unroll
    for (int i = 0; i < 4 * TT; ++i) v[i] = i < M ? a[i] : 0.f;
    float ws[TT];
    wave_sums<TT>(v, ws);
    // lane 16 j holds value 4 t + (0, 2, 1, 3)[j] of ws[t]
    const int j = lane >> 4;
    const int which = j == 0 ? 0 : (j == 1 ? 2 : (j == 2 ? 1 : 3));
    if ((lane & 15) == 0) {
#pragma unroll
      for (int t = 0; t < TT; ++t) {
        const int m = 4 * t + which;
        if (m < M) red[(wave * M + m) * nrows + row] = ws[t];
      }
    }
  };

  for (int s0 = 0; s0 < nsteps; s0 += D) {
#pragma unroll
   for (int jr = 0; jr < D; ++jr) {
    const int s = s0 + jr;
    if (s < nsteps) {
    const Piece& f = ring[jr];
    while (cur < crow) {  // the walk left row cur
      flush(acc[0], cur);
#pragma unroll
      for (int i = 0; i + 1 < NA; ++i)
#pragma unroll
        for (int m = 0; m < M; ++m) acc[i][m] = acc[i + 1][m];
#pragma unroll
      for (int m = 0; m < M; ++m) acc[NA - 1][m] = 0.f;
      ++cur;
    }
    // the lane's row is crow + rel
    int chunk = coff + lane, rel = 0;
    if (chunk >= ppr) {
      chunk -= ppr;
      rel = 1;
    }
    if (NA > 2 && chunk >= ppr) {
      chunk -= ppr;
      rel = 2;
    }
    const bool ok = cb + lane < pe;
    float a[M];
#pragma unroll
    for (int m = 0; m < M; ++m) a[m] = 0.f;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
      for (int m = 0; m < M; ++m) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(xs + (((size_t)m * 2 + h) * ppr + chunk) * 8);
        float t = a[m];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t we = f.c[h][e], xe = v[e];  // scalar copies
          t = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, we), __builtin_bit_cast(half2_t, xe), t, false);
        }
        a[m] = t;
      }
    }
#pragma unroll
    for (int m = 0; m < M; ++m) {
      const float v = ok ? a[m] : 0.f;
#pragma unroll
      for (int i = 0; i < NA; ++i) acc[i][m] += rel == i ? v : 0.f;
    }
    cb += 64;
    coff += 64;
    while (coff >= ppr) {
      coff -= ppr;
      ++crow;
    }
    }
    ring[jr] = load(s + D);
   }
  }
  if (nsteps > 0) {
#pragma unroll
    for (int i = 0; i < NA; ++i)
      if (cur + i < nrows) flush(acc[i], cur + i);
  }
  __syncthreads();
  for (int t = (int)threadIdx.x; t < M * nrows; t += nthr) {
    float v = 0.f;
    for (int q = 0; q < nwave; ++q) v += red[q * M * nrows + t];  // consecutive threads, consecutive words
    int m = 0, row = t;
#pragma unroll
    for (int mm = 1; mm < M; ++mm)
      if (row >= nrows) {
        row -= nrows;
        m = mm;
      }
    const int64_t o = (int64_t)m * n + r0 + row;
    if constexpr (KS > 1) {  // meet the other slice's partial sum of this value
      const unsigned long long oth = atomicExch(slots + o, (1ull << 32) | __builtin_bit_cast(uint32_t, v));
      if (oth == 0ull) continue;  // the other slice finishes this value
      const float ov = __builtin_bit_cast(float, (uint32_t)(oth & 0xFFFFFFFFull));
      v = slice == 0 ? v + ov : ov + v;
      atomicExch(slots + o, 0ull);  // empty for the next launch
    }
    if (out_mode == kOutF16)
      reinterpret_cast<uint16_t*>(y)[o] = f32_to_f16_bits(v);
    else if (out_mode == kOutAcc)
      reinterpret_cast<float*>(y)[o] = (t == (int)threadIdx.x ? yold : reinterpret_cast<const float*>(y)[o]) + v;
    else
      reinterpret_cast<float*>(y)[o] = v;
  }
}

template <int V>
struct RowsIntC {
  static constexpr int value = V;
};

constexpr size_t kRowsLds = 150 * 1024;
// steps of loads in flight per wavefront: one for whole rows (measured on 7B
// q|k|v at m = 5: depth 1 / 2 / 3 at 9.5 / 10.0 / 11.1 us), two with K slices,
// whose wavefronts walk several steps (7B down at m = 5: 29.9 -> 28.1 us)
template <int KS>
constexpr int verify_rows_depth() { return KS > 1 ? 2 : 1; }

template <int M>
hipError_t gemm_rows_m(const uint16_t* x, int64_t k, const uint16_t* w, int64_t n, void* y, int out_mode,
                       const NormSrc* nrm, hipStream_t stream) {
  if (k < 512 || k % 16 != 0) return hipErrorNotSupported;  // whole 16-weight pieces per row
  if (nrm && k > 4096) return hipErrorNotSupported;          // normalised rows of at most 4096 values
  const NormSrc nr = nrm ? *nrm : NormSrc{nullptr, nullptr, 0.f, 1};
  constexpr int nwave = 16, nthr = 64 * nwave;
  // one K slice where the activations and row slots fit, else two (k % 32 == 0),
  // with half as many row blocks so that the workgroups still fill the CUs once
  auto fits = [&](int ks, int64_t& blocks, size_t& lds) {
    const int64_t wg = cu_count() / ks;
    blocks = n < wg ? n : wg;
    const int64_t rows_max = (n + blocks - 1) / blocks;
    const int64_t ppr = k / ks / 16;
    const int64_t xcells = (int64_t)M * 2 * ppr;
    lds = (size_t)xcells * 16 + (nrm ? 128 : 0) + (size_t)nwave * M * rows_max * sizeof(float);
    const int64_t pmax = ks > 1 ? (int64_t(1) << 24) : (int64_t(1) << 27);
    return k % (16 * ks) == 0 && ppr >= 32 && lds <= kRowsLds && rows_max * ppr < pmax && xcells <= 8 * nthr;
  };
  int64_t blocks = 0;
  size_t lds = 0;
  int ks = 1;
  if (!fits(1, blocks, lds)) {
    ks = 2;
    if (!fits(2, blocks, lds)) return hipErrorNotSupported;
  }
  const int64_t ppr = k / ks / 16, xcells = (int64_t)M * 2 * ppr;
  // normalised rows: one K slice, at most four cells per thread
  if (nrm && (ks != 1 || xcells > 4 * nthr)) return hipErrorNotSupported;
  unsigned long long* slots = nullptr;
  if (ks > 1) {  // one 64-bit meeting slot per output value
    int32_t* c = nullptr;
    const hipError_t e = zeroed_counters(2 * (size_t)M * n, stream, &c);
    if (e != hipSuccess) return e;
    slots = reinterpret_cast<unsigned long long*>(c);
  }
  const int64_t q = n / blocks;
  const int rem = (int)(n % blocks);
  // at least half the LDS of a CU, so that no CU holds two of these workgroups
  // while another holds none (the registers of the small-m kernels would allow two)
  const size_t lds_launch = lds > 81 * 1024 ? lds : 81 * 1024;
  auto go = [&](auto na_tag, auto xb_tag, auto ks_tag) {
    constexpr int NA = decltype(na_tag)::value, XB = decltype(xb_tag)::value, KS = decltype(ks_tag)::value;
    if constexpr (KS == 1 && XB <= 4) {
      if (nrm) {
        hipLaunchKernelGGL((gemm_rows_kernel<M, NA, nwave, XB, verify_rows_depth<KS>(), KS, true>),
                           dim3((unsigned)blocks, (unsigned)KS), dim3(nthr), lds_launch, stream, x, k, w, q, rem,
                           n, y, out_mode, slots, nr);
        return;
      }
    }
    hipLaunchKernelGGL((gemm_rows_kernel<M, NA, nwave, XB, verify_rows_depth<KS>(), KS, false>),
                       dim3((unsigned)blocks, (unsigned)KS), dim3(nthr), lds_launch, stream, x, k, w, q, rem, n, y,
                       out_mode, slots, nr);
  };
  using C1 = RowsIntC<1>;
  using C2 = RowsIntC<2>;
  using C3 = RowsIntC<3>;
  using C4 = RowsIntC<4>;
  using C8 = RowsIntC<8>;
  // rows (or slices of rows) of 32 .. 63 pieces: a step meets up to three rows;
  // the fewest activation cells per thread that cover the activations
  const bool three = ppr < 64;
  auto pick = [&](auto na_tag, auto ks_tag) {
    if (xcells <= 2 * nthr)
      go(na_tag, C2{}, ks_tag);
    else if (xcells <= 3 * nthr)
      go(na_tag, C3{}, ks_tag);
    else if (xcells <= 4 * nthr)
      go(na_tag, C4{}, ks_tag);
    else
      go(na_tag, C8{}, ks_tag);
  };
  if (ks > 1)
    three ? pick(C3{}, C2{}) : pick(C2{}, C2{});
  else
    three ? pick(C3{}, C1{}) : pick(C2{}, C1{});
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_rows_f16(const uint16_t* x, int m, int64_t k, const uint16_t* w, int64_t n, void* y,
                                bool f16_out, hipStream_t stream, const NormSrc* nrm, bool accum) {
  const int mode = accum ? kOutAcc : (f16_out ? kOutF16 : kOutF32);
  switch (m) {
    case 1: return gemm_rows_m<1>(x, k, w, n, y, mode, nrm, stream);
    case 2: return gemm_rows_m<2>(x, k, w, n, y, mode, nrm, stream);
    case 3: return gemm_rows_m<3>(x, k, w, n, y, mode, nrm, stream);
    case 4: return gemm_rows_m<4>(x, k, w, n, y, mode, nrm, stream);
    case 5: return gemm_rows_m<5>(x, k, w, n, y, mode, nrm, stream);
    case 6: return gemm_rows_m<6>(x, k, w, n, y, mode, nrm, stream);
    case 7: return gemm_rows_m<7>(x, k, w, n, y, mode, nrm, stream);
    case 8: return gemm_rows_m<8>(x, k, w, n, y, mode, nrm, stream);
    default: return hipErrorNotSupported;
  }
}

hipError_t launch_gemm_f16(const uint16_t* x, int m, int64_t k, const uint16_t* w, int64_t n, void* y, bool f16_out,
                           hipStream_t stream) {
  if (m <= 16) return gemm_mt<1, 2>(x, m, k, w, n, y, f16_out, stream);
  if (m <= 32) return gemm_mt<2, 1>(x, m, k, w, n, y, f16_out, stream);
  if (m <= 48) return gemm_mt<3, 1>(x, m, k, w, n, y, f16_out, stream);
  if (m <= 64) return gemm_mt<4, 1>(x, m, k, w, n, y, f16_out, stream);
  return hipErrorInvalidValue;
}

}  // namespace sq

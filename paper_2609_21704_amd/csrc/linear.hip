// Weight-streaming linear layers on the matrix cores: the draft projections
// with the INT4 or FP8 parent (SpecQuant SS III-D.2) and the verification
// pass with the FP16 parent (SS III-D.3),
//   y[m][n] = sum_c x[m][c] * W'[n][c],   1 <= m <= 64,
// with W' the dequantized weight (INT4: (q - z) * s per 128-element group;
// FP8: decode(c) * s per row; FP16: W itself).
//
// Every weight byte is read once, as 16-byte loads.  A tile is 16 weight rows;
// lane l of a wavefront holds row l % 16 and lane quarter j = l / 16 holds the
// j-th quarter of each 16-byte-per-lane slab, which is the B operand layout of
// v_mfma_f32_16x16x32_f16 (lane l: B[8 j .. 8 j + 8)[l % 16]).  The
// activations are the A operand, read from LDS in the same k order, and the
// output tile D[m][n] accumulates in fp32 on the matrix cores; the m rows
// are padded to MT 16-row tiles, each a matrix-core product with the same
// (dequantized) weight fragment.
//   INT4: a 16-byte slab is one 128-element group of 16 rows (quarter j holds
//     codes 32 j .. 32 j + 32); each 32-bit code word becomes 8 halves without
//     a conversion instruction (a nibble masked into the mantissa of the
//     binary16 constant 1024 (or 64) is 1024 + q (or 64 + q), one shift by 8
//     serves the upper nibble pairs) and one packed subtraction of c + z gives
//     the exact q - z, so the matrix core forms exact products; the four words
//     of a group accumulate into a group tile that is scaled once by s.
//   FP8: v_cvt_scalef32_pk_f16_fp8 gives exact halves; the row scale is
//     applied to the row total.
//   FP16: the weights are the B operand as loaded.
//
// Work split: a unit is one tile x kU slabs along k (4 KB); a task is a tile's
// units, cut into chunks of a fixed number of units.  The chunks are split
// into equal contiguous ranges, one per workgroup of 8 wavefronts, one
// workgroup per CU (8 wavefronts per CU keep fewer bytes in flight than 16 and
// stream faster: 7B gate|up 54.0 -> 52.5 us at m = 5).  Inside a workgroup the
// wavefronts take chunks from a counter in LDS, so that wavefronts the memory
// system serves faster take more (their progress differs by tens of percent
// when the shares are fixed); a wavefront fetches its next unit while it
// computes the current one, and stores each chunk's partial sum in that
// chunk's LDS slot.  After the workgroup's barrier each task's chunks are
// added in chunk order, so results do not depend on which wavefront ran
// which chunk.  Every workgroup owns at least one task's chunks, so a task
// spans at most two workgroups: their two partial sums meet in a 64-bit slot
// by atomic exchange (the value travels inside the atomic, so no fence is
// needed); the second to arrive adds lower + upper in that order, stores the
// result and empties the slot for the next launch.  The activations of a K
// slice are staged in LDS once per workgroup; when they do not fit, K is cut
// into slices.  Two slices meet per output value in a 64-bit slot the same
// way (slice 0's partial is the left operand); the partial outputs of more
// slices are added in slice order by a second kernel.
//
// Direct mode (m > 16, when the chunks' partial sums would not fit in LDS:
// m x 16 floats per chunk): a chunk is a whole task, so a workgroup owns whole
// tasks, a wavefront finishes each task it takes and writes its values at
// once (or this K slice's partial outputs, added by the second kernel), and
// the activations get all of the LDS.
#include <type_traits>
#include "sq_device.hpp"
#include "sq_internal.hpp"

namespace sq {
namespace {

enum : int { kW4 = 0, kW8 = 1, kF16 = 2 };
constexpr int kU = 4;  // 16-byte slabs per lane per unit

// k values one 16-byte slab covers across the four lane quarters, and the
// MFMA k-windows (8 k per lane) in one lane's 16 bytes
template <int KIND>
constexpr int k_per_slab() { return KIND == kW4 ? 128 : (KIND == kW8 ? 64 : 32); }
template <int KIND>
constexpr int words_per_slab() { return KIND == kW4 ? 4 : (KIND == kW8 ? 2 : 1); }
template <int KIND>
constexpr int weight_bits() { return KIND == kW4 ? 4 : (KIND == kW8 ? 8 : 16); }


template <int KIND>
struct Unit {
  u32x4 c[kU];
  uint32_t s[1];  // INT4: scale and zero bits of the lane quarter's group (exchanged at use)
  uint32_t z[1];
};

struct Geo {
  int64_t n, k, k0, kl;  // rows, row length, slice start and length
  int S;                 // units per task in this slice
  int xs_stride;         // LDS activation row stride in 16-byte cells
  int64_t row_bytes;
  int groups;            // INT4 groups per full row
};

// Codes of unit (tile t, block b) for this lane: slab u covers k from
// (b kU + u) * k_per_slab within the slice; lane quarter j holds its j-th
// quarter.  Rows past n read row n - 1 again and are never stored; slabs past
// the slice read the slice's first slab and are zeroed before use.
template <int KIND>
__device__ __forceinline__ Unit<KIND> load_unit(const uint8_t* __restrict__ w, const uint16_t* __restrict__ scales,
                                                const uint16_t* __restrict__ zeros, const Geo& g, int64_t t, int b,
                                                int lane) {
  Unit<KIND> f;
  constexpr int KS = k_per_slab<KIND>();
  const int j = lane >> 4;
  const int64_t row0 = t * 16;
  const int64_t last = g.n - 1 - row0;
  const int rl = (lane & 15) < last ? (lane & 15) : (int)last;
  const uint8_t* rb = w + (row0 + rl) * g.row_bytes + ((g.k0 * weight_bits<KIND>()) >> 3);
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const int64_t kq = (int64_t)(b * kU + u) * KS + j * (KS / 4);  // first k of the lane's 16 bytes
    const int64_t off = kq < g.kl ? ((kq * weight_bits<KIND>()) >> 3) : 0;
    f.c[u] = *reinterpret_cast<const u32x4*>(rb + off);
    if constexpr (KIND == kW4) {
      // the scale / zero of group (b kU + j) of the lane's row, for slab j
      int64_t gi = (g.k0 >> 7) + (int64_t)b * kU + j;
      const int64_t gmax = (g.k0 + g.kl) / 128 - 1;
      gi = gi < gmax ? gi : gmax;
      if (u == 0) {
        const int64_t idx = (row0 + rl) * g.groups + gi;
        f.s[0] = scales[idx];
        f.z[0] = zeros[idx];
      }
    }
  }
  return f;
}

// Every lane receives the values v of the four lanes of its column
// (l % 16 + 16 q, q = 0..3): two permlane32 and one permlane16 swap.
__device__ __forceinline__ void quarters(uint32_t v, uint32_t (&out)[4]) {
  const auto p = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  const uint32_t even = p[0], odd = p[1];  // scalar copies: vector element lvalues are misread
  const auto e = __builtin_amdgcn_permlane32_swap(even, even, false, false);
  const auto o = __builtin_amdgcn_permlane32_swap(odd, odd, false, false);
  out[0] = e[0];
  out[2] = e[1];
  out[1] = o[0];
  out[3] = o[1];
}

// floor(a / b) for 0 <= a < 2^52 and 1 <= b < 2^52.  The correctly rounded
// double quotient is within one of it, and one step corrects that; integer
// division would expand to a long software sequence.
__device__ __forceinline__ int64_t div_floor(int64_t a, int64_t b) {
  int64_t q = (int64_t)((double)a / (double)b);
  if (q * b > a)
    --q;
  else if ((q + 1) * b <= a)
    ++q;
  return q;
}

// q = a / b, r = a % b for 0 <= a < 2^24 and 16 <= b, with rb = 1 / b: the
// float estimate is off by at most one.
__device__ __forceinline__ void divmod_cells(int a, int b, float rb, int& q, int& r) {
  q = (int)((float)a * rb);
  r = a - q * b;
  if (r < 0) {
    --q;
    r += b;
  } else if (r >= b) {
    ++q;
    r -= b;
  }
}

// Activations of a K slice in LDS: row m at cells [m * stride, + kl_cells);
// a cell holds 8 consecutive k (INT4: in the order 0,4,1,5,2,6,3,7 -- the
// nibble pairs of a code word); k past the slice is zero.  A thread's cells
// are the flat indices base + i * blockDim.x + threadIdx.x over [M][kl_cells];
// their (row, cell) pairs advance by a fixed step, without a division per
// cell.  The loads of a batch (eight cells per thread) are unconditional (a
// cell past the end reads the last cell, a k past the slice reads the last
// k of the slice; neither is used) and are issued before the weight prefetch,
// so that they do not queue behind it in HBM; the stores follow.
template <int KIND>
struct XStage {
  static constexpr int B = 8;
  u32x4 v[B];
  int row[B], cell[B];

  __device__ __forceinline__ void load(const uint16_t* __restrict__ x, int M, int64_t k, const Geo& g, int kl_cells,
                                       int base) {
    const int total = M * kl_cells, nthreads = (int)blockDim.x;
    const float rb = 1.0f / (float)kl_cells;
    int m, c, dm, dc;
    divmod_cells(base + (int)threadIdx.x, kl_cells, rb, m, c);
    divmod_cells(nthreads, kl_cells, rb, dm, dc);
#pragma unroll
    for (int i = 0; i < B; ++i) {
      const bool in = base + i * nthreads + (int)threadIdx.x < total;
      row[i] = in ? m : -1;
      cell[i] = c;
      const int64_t kk = (int64_t)c * 8;
      const int64_t kc = kk < g.kl ? kk : g.kl - 8;
      const int mr = in ? m : M - 1;
      v[i] = *reinterpret_cast<const u32x4*>(x + (int64_t)mr * k + g.k0 + kc);
      c += dc;
      m += dm;
      if (c >= kl_cells) {
        c -= kl_cells;
        ++m;
      }
    }
  }

  __device__ __forceinline__ void store(const Geo& g, half_t* xs) const {
#pragma unroll
    for (int i = 0; i < B; ++i) {
      if (row[i] < 0) continue;
      const u32x4 raw = (int64_t)cell[i] * 8 < g.kl ? v[i] : u32x4{0u, 0u, 0u, 0u};
      u32x4 out = raw;
      if constexpr (KIND == kW4) {
        // halves (x0,x1),(x2,x3),(x4,x5),(x6,x7) -> (x0,x4),(x1,x5),(x2,x6),(x3,x7)
        out[0] = __builtin_amdgcn_perm(raw[2], raw[0], 0x05040100u);
        out[1] = __builtin_amdgcn_perm(raw[2], raw[0], 0x07060302u);
        out[2] = __builtin_amdgcn_perm(raw[3], raw[1], 0x05040100u);
        out[3] = __builtin_amdgcn_perm(raw[3], raw[1], 0x07060302u);
      }
      *reinterpret_cast<u32x4*>(xs + ((size_t)row[i] * g.xs_stride + cell[i]) * 8) = out;
    }
  }
};

__device__ __forceinline__ half8_t as_h8(u32x4 v) { return __builtin_bit_cast(half8_t, v); }

// (several activation tiles hold more registers; a CU runs one workgroup of 8
// wavefronts, two per SIMD)
template <int KIND, int NW, int MT>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(MT == 1 ? 4 : 2)))
void linear_kernel(const uint16_t* __restrict__ x, int M, int64_t k, int64_t kslice, const uint8_t* __restrict__ w,
                   const uint16_t* __restrict__ scales16, const uint16_t* __restrict__ zeros16,
                   const float* __restrict__ scales32, int64_t n, void* __restrict__ y, int f16_out,
                   float* __restrict__ split_out, int64_t nwg_max, int chunk_units, unsigned long long* xchg,
                   unsigned long long* slice_xchg, int direct) {
  extern __shared__ __align__(16) char smem[];
  __shared__ int next_chunk;
  constexpr int KS = k_per_slab<KIND>();
  constexpr int UK = kU * KS;  // k per unit
  const int split = blockIdx.y;
  Geo g;
  g.n = n;
  g.k = k;
  g.k0 = (int64_t)split * kslice;
  g.kl = (k - g.k0) < kslice ? (k - g.k0) : kslice;
  g.S = (int)((g.kl + UK - 1) / UK);
  const int kl_cells = (int)((int64_t)g.S * UK / 8);
  g.xs_stride = kl_cells | 1;  // odd: rows of the A fragments fall in different banks
  g.row_bytes = (k * weight_bits<KIND>()) >> 3;
  g.groups = (int)(k >> 7);
  const int64_t ntask = (n + 15) / 16;
  const int C = chunk_units < g.S ? chunk_units : g.S;
  const int J = (g.S + C - 1) / C;  // chunks per task: units [j C, min(j C + C, S))
  const int64_t FC = ntask * J;
  const int64_t nwg = ntask < nwg_max ? ntask : nwg_max;  // every workgroup owns at least one task's chunks
  const int64_t wg = blockIdx.x;
  if (wg >= nwg) return;  // uniform across the workgroup

  half_t* xs = reinterpret_cast<half_t*>(smem);
  // the chunks' partial sums [nch][M][16], after the activations in LDS
  float* pl = reinterpret_cast<float*>(smem + ((size_t)M * g.xs_stride * 16 + 15) / 16 * 16);

  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 15, q = lane >> 4;

  // activations first, then the first unit of this wavefront's first chunk
  // (chunk wv; the others come from the counter), so that x is not queued
  // behind the weight stream
  if (threadIdx.x == 0) next_chunk = NW;
  XStage<KIND> xst;
  xst.load(x, M, k, g, kl_cells, 0);
  // equal contiguous chunk ranges: workgroup wg owns chunks [c0, c1)
  const int64_t c0 = div_floor(wg * FC, nwg), c1 = div_floor((wg + 1) * FC, nwg);
  const int nch = (int)(c1 - c0);
  // local chunk cl: task t, units [b, b_end) of it
  auto chunk_at = [&](int cl, int64_t& t, int& b, int& b_end) {
    const int64_t c = c0 + cl;
    t = div_floor(c, J);
    b = (int)(c - t * J) * C;
    b_end = b + C < g.S ? b + C : g.S;
  };
  int cl = wv;
  int64_t t = 0;
  int b = 0, b_end = 0;
  Unit<KIND> fa, fb;
  if (cl < nch) {
    chunk_at(cl, t, b, b_end);
    fa = load_unit<KIND>(w, scales16, zeros16, g, t, b, lane);
  }
  xst.store(g, xs);
  const int xbatch = XStage<KIND>::B * (int)blockDim.x;
  for (int base = xbatch; base < M * kl_cells; base += xbatch) {  // activations beyond the first batch
    xst.load(x, M, k, g, kl_cells, base);
    xst.store(g, xs);
  }
  __syncthreads();

  // the finished value (m, row): row scale (FP8), then y or this slice's partial output
  auto store_y = [&](int64_t row, int m, float val) {
    if constexpr (KIND == kW8) val *= scales32[row];
    if (split_out)
      split_out[((int64_t)split * M + m) * n + row] = val;
    else if (f16_out)
      reinterpret_cast<uint16_t*>(y)[(int64_t)m * n + row] = f32_to_f16_bits(val);
    else
      reinterpret_cast<float*>(y)[(int64_t)m * n + row] = val;
  };

  if (cl < nch) {
    // a valid activation row for the padding rows of each A tile (their outputs are dropped)
    int arow[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) arow[mt] = mt * 16 + col < M ? mt * 16 + col : 0;
    float4_t acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = float4_t{0.f, 0.f, 0.f, 0.f};
    bool more = true;

    // masks and magic numbers in VGPRs, so each mask-and-insert is one v_and_or_b32
    uint32_t mlo = 0x000F000Fu, mhi = 0x00F000F0u, k1024 = 0x64006400u, k64 = 0x54005400u;
    asm("" : "+v"(mlo), "+v"(mhi), "+v"(k1024), "+v"(k64));

    auto step = [&](const Unit<KIND>& cur, Unit<KIND>& nxt) {
      // the next unit: the chunk's next, else the first of the next chunk from
      // the counter, else (none left) this one again, so that the load stays
      // unconditional
      int64_t t_n = t;
      int b_n = b + 1, be_n = b_end, cl_n = cl;
      bool more_n = true;
      if (b_n == b_end) {
        int got = 0;
        if (lane == 0) got = atomicAdd(&next_chunk, 1);
        cl_n = __builtin_amdgcn_readfirstlane(got);
        more_n = cl_n < nch;
        if (more_n)
          chunk_at(cl_n, t_n, b_n, be_n);
        else
          b_n = b;
      }
      nxt = load_unit<KIND>(w, scales16, zeros16, g, t_n, b_n, lane);
      __builtin_amdgcn_sched_barrier(0);  // issue the loads before the compute below
      uint32_t sc[4], zc[4];
      if constexpr (KIND == kW4) {
        quarters(cur.s[0], sc);
        quarters(cur.z[0], zc);
      }
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int64_t kslab = (int64_t)(b * kU + u) * KS;  // first k of slab u in the slice
        const bool valid = kslab + q * (KS / 4) < g.kl;
        const u32x4 c = valid ? cur.c[u] : u32x4{0u, 0u, 0u, 0u};
        const int cell0 = (int)(kslab / 8) + q * (KS / 32);
        if constexpr (KIND == kW4) {
          const half2_t z2 = __builtin_bit_cast(half2_t, zc[u] | (zc[u] << 16));
          const half2_t c1024 = z2 + half2_t{(half_t)1024.0f, (half_t)1024.0f};
          const half2_t c64 = z2 + half2_t{(half_t)64.0f, (half_t)64.0f};
          // every activation tile meets the same dequantized fragment
          float4_t gacc[MT];
#pragma unroll
          for (int wd = 0; wd < 4; ++wd) {
            const uint32_t qw = c[wd];
            const uint32_t q8 = qw >> 8;
            const half2_t d0 = __builtin_bit_cast(half2_t, (qw & mlo) | k1024) - c1024;  // q0 - z, q4 - z
            const half2_t d1 = __builtin_bit_cast(half2_t, (qw & mhi) | k64) - c64;      // q1 - z, q5 - z
            const half2_t d2 = __builtin_bit_cast(half2_t, (q8 & mlo) | k1024) - c1024;  // q2 - z, q6 - z
            const half2_t d3 = __builtin_bit_cast(half2_t, (q8 & mhi) | k64) - c64;      // q3 - z, q7 - z
            const half8_t bw = half8_t{d0[0], d0[1], d1[0], d1[1], d2[0], d2[1], d3[0], d3[1]};
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
              const half8_t a =
                  as_h8(*reinterpret_cast<const u32x4*>(xs + ((size_t)arow[mt] * g.xs_stride + cell0 + wd) * 8));
              gacc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bw, wd == 0 ? float4_t{0.f, 0.f, 0.f, 0.f} : gacc[mt],
                                                                0, 0, 0);
            }
          }
          const float s = valid ? f16_bits_to_f32((uint16_t)sc[u]) : 0.f;
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) acc[mt] += s * gacc[mt];
        } else if constexpr (KIND == kW8) {
#pragma unroll
          for (int wd = 0; wd < 2; ++wd) {
            const uint32_t w0 = c[2 * wd], w1 = c[2 * wd + 1];
            const half2_t h0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w0, 1.0f, false);
            const half2_t h1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w0, 1.0f, true);
            const half2_t h2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w1, 1.0f, false);
            const half2_t h3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w1, 1.0f, true);
            const half8_t bw = half8_t{h0[0], h0[1], h1[0], h1[1], h2[0], h2[1], h3[0], h3[1]};
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
              const half8_t a =
                  as_h8(*reinterpret_cast<const u32x4*>(xs + ((size_t)arow[mt] * g.xs_stride + cell0 + wd) * 8));
              acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bw, acc[mt], 0, 0, 0);
            }
          }
        } else {
          const half8_t bw = as_h8(c);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            const half8_t a =
                as_h8(*reinterpret_cast<const u32x4*>(xs + ((size_t)arow[mt] * g.xs_stride + cell0) * 8));
            acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bw, acc[mt], 0, 0, 0);
          }
        }
      }
      if (b + 1 == b_end) {  // the chunk's last unit
        if (MT > 1 && direct) {
          // the chunk is a whole task of this workgroup: its values are finished
          // here (meeting the other K slice's in a 64-bit slot when there are two)
          const int64_t row = t * 16 + col;
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int m = mt * 16 + 4 * q + r;
              if (m >= M || row >= n) continue;
              float val = acc[mt][r];
              if (slice_xchg) {
                unsigned long long* sl = slice_xchg + (size_t)m * n + row;
                const unsigned long long oth = atomicExch(sl, (1ull << 32) | __builtin_bit_cast(uint32_t, val));
                if (oth == 0ull) continue;  // the other slice finishes this value
                const float o = __builtin_bit_cast(float, (uint32_t)(oth & 0xFFFFFFFFull));
                val = split == 0 ? val + o : o + val;
                atomicExch(sl, 0ull);  // empty for the next launch
              }
              store_y(row, m, val);
            }
        } else {  // its partial sum goes to the chunk's slot
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int m = mt * 16 + 4 * q + r;
              if (m < M) pl[((size_t)cl * M + m) * 16 + col] = acc[mt][r];
            }
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[mt] = float4_t{0.f, 0.f, 0.f, 0.f};
      }
      t = t_n;
      b = b_n;
      b_end = be_n;
      cl = cl_n;
      more = more_n;
    };

    while (true) {
      step(fa, fb);
      if (!more) break;
      step(fb, fa);
      if (!more) break;
    }
  }
  __syncthreads();


  // Every task with chunks here: its chunks' partial sums are added in chunk
  // order (wavefront wv takes tasks wv, wv + NW, ...).  A task whose chunks
  // all lie here is finished; one shared with a neighbouring workgroup meets
  // the other half in a 64-bit slot.  With two K slices each finished value
  // then meets the other slice's the same way (slice 0's partial is the left
  // operand).  The loops stay rolled: this tail runs once per launch, and
  // unrolled it would be fetched into the instruction cache cold.
  // Lane quarter q takes output rows m = q + 4 j.
  constexpr int MQ = 4 * MT;
  const int64_t t_lo = div_floor(c0, J), t_hi = div_floor(c1 - 1, J);
#pragma unroll 1
  for (int64_t tt = t_lo + wv; !(MT > 1 && direct) && tt <= t_hi; tt += NW) {
    const int64_t ca = tt * J > c0 ? tt * J : c0, cb = (tt + 1) * J < c1 ? (tt + 1) * J : c1;
    const int64_t row = tt * 16 + col;
    int mm[MQ];
    float val[MQ];
    bool ok[MQ];
#pragma unroll
    for (int j = 0; j < MQ; ++j) {
      mm[j] = q + 4 * j;
      ok[j] = mm[j] < M;
      val[j] = 0.f;
    }
#pragma unroll 1
    for (int64_t c = ca; c < cb; ++c) {
      const float* pc = pl + (size_t)(c - c0) * M * 16 + col;
#pragma unroll
      for (int j = 0; j < MQ; ++j)
        if (ok[j]) val[j] += pc[mm[j] * 16];
    }
    unsigned long long oth[MQ];
    if (ca != tt * J || cb != (tt + 1) * J) {  // shared with a neighbouring workgroup (uniform in the wavefront)
      const bool upper = tt * J < c0;          // this workgroup holds the task's later chunks
      unsigned long long* ws = xchg + ((size_t)split * nwg_max + (upper ? wg - 1 : wg)) * M * 16 + col;
#pragma unroll
      for (int j = 0; j < MQ; ++j) {
        oth[j] = 0ull;
        if (ok[j]) oth[j] = atomicExch(ws + mm[j] * 16, (1ull << 32) | __builtin_bit_cast(uint32_t, val[j]));
      }
#pragma unroll
      for (int j = 0; j < MQ; ++j) {
        if (!ok[j]) continue;
        if (oth[j] == 0ull) {  // the other workgroup finishes this value
          ok[j] = false;
          continue;
        }
        const float o = __builtin_bit_cast(float, (uint32_t)(oth[j] & 0xFFFFFFFFull));
        val[j] = upper ? o + val[j] : val[j] + o;
        atomicExch(ws + mm[j] * 16, 0ull);  // empty for the next launch
      }
    }
#pragma unroll
    for (int j = 0; j < MQ; ++j) ok[j] = ok[j] && row < n;
    if (slice_xchg) {
#pragma unroll
      for (int j = 0; j < MQ; ++j) {
        oth[j] = 0ull;
        if (ok[j])
          oth[j] = atomicExch(slice_xchg + (size_t)mm[j] * n + row, (1ull << 32) | __builtin_bit_cast(uint32_t, val[j]));
      }
#pragma unroll
      for (int j = 0; j < MQ; ++j) {
        if (!ok[j]) continue;
        if (oth[j] == 0ull) {  // the other slice finishes this value
          ok[j] = false;
          continue;
        }
        const float o = __builtin_bit_cast(float, (uint32_t)(oth[j] & 0xFFFFFFFFull));
        val[j] = split == 0 ? val[j] + o : o + val[j];
        atomicExch(slice_xchg + (size_t)mm[j] * n + row, 0ull);  // empty for the next launch
      }
    }
#pragma unroll
    for (int j = 0; j < MQ; ++j)
      if (ok[j]) store_y(row, mm[j], val[j]);
  }
}

template <bool F16Out>
__global__ __launch_bounds__(256) void slice_reduce_kernel(const float* __restrict__ partial, int splits,
                                                           int64_t mn, void* __restrict__ y) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < mn; i += (int64_t)gridDim.x * 256) {
    float v = 0.f;
    for (int s = 0; s < splits; ++s) v += partial[(int64_t)s * mn + i];
    store_out<F16Out>(y, i, v);
  }
}

constexpr int64_t kChunkMinUnits = 4;  // units per chunk, at least (measured: 4 beats 1 and 2)
constexpr size_t kLdsTotal = 150 * 1024;   // one workgroup per CU
constexpr size_t kPieceBudget = 32 * 1024; // chunk partial sums

template <int KIND, int NW, int MT>
hipError_t linear_launch(const uint16_t* x, int m, int64_t k, const uint8_t* w, const uint16_t* scales16,
                         const uint16_t* zeros16, const float* scales32, int64_t n, void* y, bool f16_out,
                         bool direct, hipStream_t stream) {
  constexpr int64_t UK = (int64_t)kU * k_per_slab<KIND>();
  // K slices of whole units whose activations fit (2 bytes per k and row, plus a pad cell per row);
  // the direct mode keeps no chunk partial sums in LDS
  int64_t kmax = (int64_t)((kLdsTotal - (direct ? 0 : kPieceBudget)) / ((size_t)m * 2)) - 8;
  kmax = kmax / UK * UK;
  if (kmax < UK) return hipErrorNotSupported;  // the caller takes another kernel
  const int splits = (int)((k + kmax - 1) / kmax);
  int64_t kslice = (k + splits - 1) / splits;
  kslice = (kslice + UK - 1) / UK * UK;
  const int64_t kfirst = kslice < k ? kslice : k;
  const int64_t S = (kfirst + UK - 1) / UK;
  const int64_t cells = (S * UK / 8) | 1;
  const int64_t ntask = (n + 15) / 16;
  // one workgroup per CU, shared by the slices; each owns at least one task's chunks
  int64_t nwg_max = ntask;
  const int64_t cap = (int64_t)cu_count() / splits;
  if (nwg_max > cap) nwg_max = cap;
  if (nwg_max < 1) nwg_max = 1;
  // the smallest chunk whose partial sums ([chunks per workgroup][m][16] floats) fit the budget;
  // direct: one chunk per task, no partial sums
  int64_t C = direct ? S : kChunkMinUnits, nch_max = 0;
  for (;; ++C) {
    const int64_t J = (S + C - 1) / C;
    nch_max = (ntask * J + nwg_max - 1) / nwg_max;
    if (direct || (size_t)nch_max * m * 16 * sizeof(float) <= kPieceBudget || C >= S) break;
  }
  if (!direct && (size_t)nch_max * m * 16 * sizeof(float) > kPieceBudget) return hipErrorNotSupported;
  // the kernel's chunk arithmetic is exact below 2^52 (workgroup index x chunks per slice)
  if ((double)(nwg_max + 1) * (double)(ntask * S) >= 4503599627370496.0) return hipErrorNotSupported;
  const size_t lds = ((size_t)m * cells * 16 + 15) / 16 * 16 + (direct ? 0 : (size_t)nch_max * m * 16 * sizeof(float));

  // two K slices meet per output value in a 64-bit slot; more are summed by a second kernel
  const bool slice_meet = splits == 2 && !direct;
  const size_t split_bytes =
      splits > 1 && !slice_meet ? ((size_t)splits * m * n * sizeof(float) + 255) / 256 * 256 : 0;
  float* split_out = nullptr;
  if (split_bytes > 0) {
    void* ws = nullptr;
    const hipError_t e = workspace(split_bytes, stream, &ws);
    if (e != hipSuccess) return e;
    split_out = static_cast<float*>(ws);
  }
  // 64-bit meeting slots: workgroup boundaries of every slice, then one per output value
  const size_t wg_slots = (size_t)splits * nwg_max * m * 16;
  const size_t value_slots = slice_meet ? (size_t)m * n : 0;
  int32_t* slots = nullptr;
  const hipError_t ce = zeroed_counters(2 * (wg_slots + value_slots), stream, &slots);
  if (ce != hipSuccess) return ce;
  unsigned long long* xchg = reinterpret_cast<unsigned long long*>(slots);
  // more than half the LDS, so that a CU holds one workgroup
  const size_t lds_launch = lds < 81 * 1024 ? 81 * 1024 : lds;
  hipLaunchKernelGGL((linear_kernel<KIND, NW, MT>), dim3((unsigned)nwg_max, (unsigned)splits), dim3(NW * 64),
                     lds_launch, stream, x, m, k, kslice, w, scales16, zeros16, scales32, n, y, (int)f16_out,
                     split_out, nwg_max, (int)C, xchg, slice_meet ? xchg + wg_slots : nullptr, (int)direct);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || splits == 1 || slice_meet) return err;
  int64_t blocks = ((int64_t)m * n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (f16_out)
    hipLaunchKernelGGL(slice_reduce_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, stream, split_out, splits,
                       (int64_t)m * n, y);
  else
    hipLaunchKernelGGL(slice_reduce_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, stream, split_out, splits,
                       (int64_t)m * n, y);
  return hipGetLastError();
}

template <int KIND>
hipError_t linear_dispatch(const uint16_t* x, int m, int64_t k, const uint8_t* w, const uint16_t* scales16,
                           const uint16_t* zeros16, const float* scales32, int64_t n, void* y, bool f16_out,
                           hipStream_t stream) {
  if (m < 1 || m > 64) return hipErrorInvalidValue;
  // chunks of a task spread over the wavefronts where their partial sums fit
  // in LDS, else whole tasks per wavefront (direct; its epilogue needs MT > 1)
  auto go = [&](auto mt_tag) {
    constexpr int MT = decltype(mt_tag)::value;
    hipError_t e = linear_launch<KIND, 8, MT>(x, m, k, w, scales16, zeros16, scales32, n, y, f16_out, false, stream);
    if (e == hipErrorNotSupported && MT > 1)
      e = linear_launch<KIND, 8, MT>(x, m, k, w, scales16, zeros16, scales32, n, y, f16_out, true, stream);
    return e;
  };
  if (m > 48) return go(std::integral_constant<int, 4>{});
  if (m > 32) return go(std::integral_constant<int, 3>{});
  if (m > 16) return go(std::integral_constant<int, 2>{});
  const hipError_t e = go(std::integral_constant<int, 1>{});
  // the quantized copies have no other kernel above m = 8: two tiles, the second one padding
  if (e == hipErrorNotSupported && KIND != kF16 && m > 8) return go(std::integral_constant<int, 2>{});
  return e;
}

}  // namespace

hipError_t launch_linear_w4(const uint16_t* x, int m, int64_t k, const uint8_t* codes, const uint16_t* scales,
                            const uint16_t* zeros, int64_t n, void* y, bool f16_out, hipStream_t stream) {
  return linear_dispatch<kW4>(x, m, k, codes, scales, zeros, nullptr, n, y, f16_out, stream);
}

hipError_t launch_linear_w8(const uint16_t* x, int m, int64_t k, const uint8_t* codes, const float* scales,
                            int64_t n, void* y, bool f16_out, hipStream_t stream) {
  return linear_dispatch<kW8>(x, m, k, codes, nullptr, nullptr, scales, n, y, f16_out, stream);
}

hipError_t launch_linear_f16(const uint16_t* x, int m, int64_t k, const uint16_t* w, int64_t n, void* y,
                             bool f16_out, hipStream_t stream) {
  return linear_dispatch<kF16>(x, m, k, reinterpret_cast<const uint8_t*>(w), nullptr, nullptr, nullptr, n, y, f16_out,
                               stream);
}

}  // namespace sq

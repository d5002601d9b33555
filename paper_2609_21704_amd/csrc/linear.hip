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
// output tile D[m][n] accumulates in fp32 on the matrix cores; m is padded to
// 16-row tiles (MT of them).
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
// units.  The units are split into equal contiguous ranges, one per
// workgroup, and each workgroup's range into equal contiguous ranges, one per
// wavefront (stream-K); a wavefront fetches its next unit while it computes
// the current one.  A task split between wavefronts is summed in wavefront
// order after the workgroup's barrier (the pieces go through a global scratch
// buffer, so that LDS holds only activations).  Every workgroup owns at least
// one task's units, so a task spans at most two workgroups: their two
// partial sums meet in a 64-bit slot by atomic exchange (the value travels
// inside the atomic, so no fence is needed); the second to arrive adds
// lower + upper in that order, stores the result and empties the slot for the
// next launch.  Results do not depend on timing.  The activations of a K
// slice are staged in LDS once per workgroup; when they do not fit, K is cut
// into slices whose partial outputs a second kernel adds in slice order.
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

template <bool B>
struct BoolC {
  static constexpr bool value = B;
};

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

// Activations of a K slice in LDS: row m at cells [m * stride, + kl_pad / 8);
// a cell holds 8 consecutive k (INT4: in the order 0,4,1,5,2,6,3,7 -- the
// nibble pairs of a code word); k past the slice is zero.
template <int KIND>
__device__ __forceinline__ u32x4 x_cell(const uint16_t* __restrict__ x, int64_t k, const Geo& g, int m, int c) {
  const int64_t kk = (int64_t)c * 8;
  const u32x4 raw = kk < g.kl ? *reinterpret_cast<const u32x4*>(x + (int64_t)m * k + g.k0 + kk)
                              : u32x4{0u, 0u, 0u, 0u};
  u32x4 out = raw;
  if constexpr (KIND == kW4) {
    // halves (x0,x1),(x2,x3),(x4,x5),(x6,x7) -> (x0,x4),(x1,x5),(x2,x6),(x3,x7)
    out[0] = __builtin_amdgcn_perm(raw[2], raw[0], 0x05040100u);
    out[1] = __builtin_amdgcn_perm(raw[2], raw[0], 0x07060302u);
    out[2] = __builtin_amdgcn_perm(raw[3], raw[1], 0x05040100u);
    out[3] = __builtin_amdgcn_perm(raw[3], raw[1], 0x07060302u);
  }
  return out;
}

// Activations of a K slice in LDS: row m at cells [m * stride, + kl_cells);
// a cell holds 8 consecutive k (INT4: in the order 0,4,1,5,2,6,3,7 -- the
// nibble pairs of a code word); k past the slice is zero.  The loads of a
// batch (eight cells per thread) are issued before the weight prefetch, so
// that they do not queue behind it in HBM; the stores follow.
template <int KIND>
struct XStage {
  static constexpr int B = 8;
  u32x4 v[B];

  __device__ __forceinline__ void load(const uint16_t* __restrict__ x, int M, int64_t k, const Geo& g, int kl_cells,
                                       int base) {
    const int total = M * kl_cells, nthreads = (int)blockDim.x;
#pragma unroll
    for (int i = 0; i < B; ++i) {
      int idx = base + i * nthreads + (int)threadIdx.x;
      idx = idx < total ? idx : total - 1;
      v[i] = x_cell<KIND>(x, k, g, idx / kl_cells, idx % kl_cells);
    }
  }

  __device__ __forceinline__ void store(int M, const Geo& g, int kl_cells, int base, half_t* xs) const {
    const int total = M * kl_cells, nthreads = (int)blockDim.x;
#pragma unroll
    for (int i = 0; i < B; ++i) {
      const int idx = base + i * nthreads + (int)threadIdx.x;
      if (idx < total)
        *reinterpret_cast<u32x4*>(xs + ((size_t)(idx / kl_cells) * g.xs_stride + idx % kl_cells) * 8) = v[i];
    }
  }
};

__device__ __forceinline__ int64_t part_begin(int64_t i, int64_t total, int64_t parts) { return i * total / parts; }
__device__ __forceinline__ int64_t part_owner(int64_t j, int64_t total, int64_t parts) {
  return ((j + 1) * parts - 1) / total;
}

__device__ __forceinline__ half8_t as_h8(u32x4 v) { return __builtin_bit_cast(half8_t, v); }

template <int KIND, int MT, int NW>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(4)))
void linear_kernel(const uint16_t* __restrict__ x, int M, int64_t k, int64_t kslice, const uint8_t* __restrict__ w,
                   const uint16_t* __restrict__ scales16, const uint16_t* __restrict__ zeros16,
                   const float* __restrict__ scales32, int64_t n, void* __restrict__ y, int f16_out,
                   float* __restrict__ split_out, int64_t nwg_max, float* pieces, unsigned long long* xchg) {
  extern __shared__ __align__(16) char smem[];
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
  const int64_t F = ntask * g.S;
  int64_t nwg = F / g.S;
  nwg = nwg < 1 ? 1 : (nwg > nwg_max ? nwg_max : nwg);
  const int64_t wg = blockIdx.x;
  if (wg >= nwg) return;  // uniform across the workgroup
  const int64_t u0 = part_begin(wg, F, nwg), u1 = part_begin(wg + 1, F, nwg), U = u1 - u0;

  half_t* xs = reinterpret_cast<half_t*>(smem);
  // this workgroup's pieces [NW][2][M][16]: after the activations in LDS when
  // m <= 16, else in the global scratch buffer
  float* pl = MT == 1 ? reinterpret_cast<float*>(smem + ((size_t)M * g.xs_stride * 16 + 15) / 16 * 16)
                      : pieces + ((size_t)split * nwg_max + wg) * NW * 2 * M * 16;

  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t f_beg = u0 + part_begin(wv, U, NW), f_end = u0 + part_begin(wv + 1, U, NW);
  const int64_t t_first = f_beg / g.S;
  const int col = lane & 15, q = lane >> 4;

  // activations first, then the first unit, so that x is not queued behind
  // the weight stream
  XStage<KIND> xst;
  xst.load(x, M, k, g, kl_cells, 0);
  Unit<KIND> fa, fb;
  if (f_beg < f_end) fa = load_unit<KIND>(w, scales16, zeros16, g, t_first, (int)(f_beg - t_first * g.S), lane);
  xst.store(M, g, kl_cells, 0, xs);
  const int xbatch = XStage<KIND>::B * (int)blockDim.x;
  for (int base = xbatch; base < M * kl_cells; base += xbatch) {  // activations beyond the first batch
    xst.load(x, M, k, g, kl_cells, base);
    xst.store(M, g, kl_cells, base, xs);
  }
  __syncthreads();

  // a valid activation row for the padding rows of the A tiles (their outputs are dropped)
  int arow[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) arow[mt] = (16 * mt + col) < M ? (16 * mt + col) : 0;

  // output value (m, row) of this lane's accumulator element (mt, r)
  auto emit = [&](int64_t row, int m, float val) {
    if constexpr (KIND == kW8) val *= scales32[row];
    if (split_out)
      split_out[((int64_t)split * M + m) * n + row] = val;
    else if (f16_out)
      reinterpret_cast<uint16_t*>(y)[(int64_t)m * n + row] = f32_to_f16_bits(val);
    else
      reinterpret_cast<float*>(y)[(int64_t)m * n + row] = val;
  };

  if (f_beg < f_end) {
    int64_t t = t_first;
    int b = (int)(f_beg - t * g.S);
    int piece_b0 = b;
    float4_t acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = float4_t{0.f, 0.f, 0.f, 0.f};

    // masks and magic numbers in VGPRs, so each mask-and-insert is one v_and_or_b32
    uint32_t mlo = 0x000F000Fu, mhi = 0x00F000F0u, k1024 = 0x64006400u, k64 = 0x54005400u;
    asm("" : "+v"(mlo), "+v"(mhi), "+v"(k1024), "+v"(k64));

    auto finish_piece = [&](bool whole) {
      const int64_t row = t * 16 + col;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = 16 * mt + 4 * q + r;
          if (m < M) {
            if (whole) {
              if (row < n) emit(row, m, acc[mt][r]);
            } else {
              pl[(((size_t)wv * 2 + (t == t_first ? 0 : 1)) * M + m) * 16 + col] = acc[mt][r];
            }
          }
        }
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[mt] = float4_t{0.f, 0.f, 0.f, 0.f};
    };

    auto step = [&](auto prefetch, const Unit<KIND>& cur, Unit<KIND>& nxt) {
      constexpr bool Prefetch = decltype(prefetch)::value;
      int64_t t_n = t;
      int b_n = b + 1;
      if (b_n == g.S) {
        b_n = 0;
        ++t_n;
      }
      if constexpr (Prefetch) {
        nxt = load_unit<KIND>(w, scales16, zeros16, g, t_n, b_n, lane);
        __builtin_amdgcn_sched_barrier(0);  // issue the loads before the compute below
      }
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
              const half8_t a = as_h8(*reinterpret_cast<const u32x4*>(
                  xs + ((size_t)arow[mt] * g.xs_stride + cell0 + wd) * 8));
              gacc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bw, wd == 0 ? float4_t{0.f, 0.f, 0.f, 0.f}
                                                                               : gacc[mt], 0, 0, 0);
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
              const half8_t a = as_h8(*reinterpret_cast<const u32x4*>(
                  xs + ((size_t)arow[mt] * g.xs_stride + cell0 + wd) * 8));
              acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bw, acc[mt], 0, 0, 0);
            }
          }
        } else {
          const half8_t bw = as_h8(c);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            const half8_t a = as_h8(*reinterpret_cast<const u32x4*>(
                xs + ((size_t)arow[mt] * g.xs_stride + cell0) * 8));
            acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bw, acc[mt], 0, 0, 0);
          }
        }
      }
      if (b == g.S - 1 || !Prefetch) {  // the end of this wavefront's piece of task t
        finish_piece(piece_b0 == 0 && b == g.S - 1);
        piece_b0 = 0;
      }
      t = t_n;
      b = b_n;
    };

    // units f_beg .. f_end - 1; every unit but the last prefetches its successor
    int64_t left = f_end - f_beg;
    for (; left > 2; left -= 2) {
      step(BoolC<true>{}, fa, fb);
      step(BoolC<true>{}, fb, fa);
    }
    if (left == 2) {
      step(BoolC<true>{}, fa, fb);
      step(BoolC<false>{}, fb, fa);
    } else {
      step(BoolC<false>{}, fa, fb);
    }
  }
  __syncthreads();
  if (f_beg >= f_end) return;

  // Tasks split between wavefronts or workgroups: the wavefront holding a
  // task's last unit inside this workgroup sums its pieces in wavefront
  // order, then stores the total or meets the other workgroup.
  const int64_t t_last = (f_end - 1) / g.S;
  for (int64_t t = t_first; t <= t_last; t += (t_last > t_first ? t_last - t_first : 1)) {
    const int64_t w_start = t * g.S > u0 ? t * g.S : u0;
    const int64_t w_stop = (t + 1) * g.S < u1 ? (t + 1) * g.S : u1;
    const bool in_wg = t * g.S >= u0 && (t + 1) * g.S <= u1;
    const bool in_wave = w_start >= f_beg && w_stop <= f_end;
    const bool mine = w_stop - 1 >= f_beg && w_stop - 1 < f_end;
    if (!(in_wave && in_wg) && mine) {
      const int wv_lo = (int)part_owner(w_start - u0, U, NW);
      const int64_t row = t * 16 + col;
      // the pieces' slots, one per wavefront (-1: that wavefront holds no piece of t)
      int slot[NW];
#pragma unroll
      for (int u = 0; u < NW; ++u) {
        const int64_t ub = part_begin(u, U, NW);
        const bool has = u >= wv_lo && u <= wv && ub != part_begin(u + 1, U, NW);
        slot[u] = has ? ((u0 + ub) / g.S == t ? 0 : 1) : -1;
      }
      for (int m = q; m < M; m += 4) {  // each lane quarter takes every fourth output row
        // fixed trip count: every load is in flight at once; the sum runs in wavefront order
        float v[NW];
#pragma unroll
        for (int u = 0; u < NW; ++u) v[u] = slot[u] >= 0 ? pl[(((size_t)u * 2 + slot[u]) * M + m) * 16 + col] : 0.f;
        float tot = 0.f;
#pragma unroll
        for (int u = 0; u < NW; ++u)
          if (slot[u] >= 0) tot += v[u];
        if (!in_wg) {
          const bool upper = t * g.S < u0;  // this workgroup holds the task's later units
          const int64_t bnd = upper ? wg - 1 : wg;
          unsigned long long* slot = xchg + (((size_t)split * nwg_max + bnd) * M + m) * 16 + col;
          const unsigned long long me = (1ull << 32) | __builtin_bit_cast(uint32_t, tot);
          const unsigned long long other = atomicExch(slot, me);
          if (other == 0ull) continue;  // the other workgroup finishes this value
          const float o = __builtin_bit_cast(float, (uint32_t)(other & 0xFFFFFFFFull));
          tot = upper ? o + tot : tot + o;
          atomicExch(slot, 0ull);  // empty for the next launch
        }
        if (row < n) emit(row, m, tot);
      }
    }
    if (t_last == t_first) break;
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

template <int KIND, int MT, int NW>
hipError_t linear_launch(const uint16_t* x, int m, int64_t k, const uint8_t* w, const uint16_t* scales16,
                         const uint16_t* zeros16, const float* scales32, int64_t n, void* y, bool f16_out,
                         hipStream_t stream) {
  constexpr int64_t UK = (int64_t)kU * k_per_slab<KIND>();
  // LDS: one workgroup per CU; the pieces of split tasks sit there too when m <= 16
  const size_t lds_pieces = MT == 1 ? (size_t)NW * 2 * m * 16 * sizeof(float) : 0;
  const size_t x_lds_max = (size_t)150 * 1024 - lds_pieces;
  // K slices of whole units whose activations fit (2 bytes per k and row, plus a pad cell per row)
  int64_t kmax = (int64_t)(x_lds_max / ((size_t)m * 2)) - 8;
  kmax = kmax / UK * UK;
  if (kmax < UK) return hipErrorInvalidValue;
  const int splits = (int)((k + kmax - 1) / kmax);
  int64_t kslice = (k + splits - 1) / splits;
  kslice = (kslice + UK - 1) / UK * UK;
  const int64_t kfirst = kslice < k ? kslice : k;
  const int64_t S = (kfirst + UK - 1) / UK;
  const int64_t cells = (S * UK / 8) | 1;
  const size_t lds = ((size_t)m * cells * 16 + 15) / 16 * 16 + lds_pieces;
  const int64_t ntask = (n + 15) / 16;
  // one workgroup per CU, shared by the slices; each owns at least one task
  int64_t nwg_max = ntask;
  const int64_t cap = (int64_t)cu_count() * (16 / NW) / splits;
  if (nwg_max > cap) nwg_max = cap;
  if (nwg_max < 1) nwg_max = 1;

  const size_t split_bytes = splits > 1 ? ((size_t)splits * m * n * sizeof(float) + 255) / 256 * 256 : 0;
  const size_t piece_bytes = MT == 1 ? 0 : (size_t)splits * nwg_max * NW * 2 * m * 16 * sizeof(float);
  char* ws = nullptr;
  if (split_bytes + piece_bytes > 0) {
    ws = static_cast<char*>(workspace(split_bytes + piece_bytes));
    if (!ws) return hipErrorOutOfMemory;
  }
  int32_t* slots = zeroed_counters((size_t)2 * splits * nwg_max * m * 16);  // 64-bit meeting slots
  if (!slots) return hipErrorOutOfMemory;
  float* split_out = splits > 1 ? reinterpret_cast<float*>(ws) : nullptr;
  float* pieces = reinterpret_cast<float*>(ws + split_bytes);
  hipLaunchKernelGGL((linear_kernel<KIND, MT, NW>), dim3((unsigned)nwg_max, (unsigned)splits), dim3(NW * 64), lds,
                     stream, x, m, k, kslice, w, scales16, zeros16, scales32, n, y, (int)f16_out, split_out, nwg_max,
                     pieces, reinterpret_cast<unsigned long long*>(slots));
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || splits == 1) return err;
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
  if (m <= 16) return linear_launch<KIND, 1, 16>(x, m, k, w, scales16, zeros16, scales32, n, y, f16_out, stream);
  if constexpr (KIND == kF16) {
    if (m <= 32) return linear_launch<KIND, 2, 16>(x, m, k, w, scales16, zeros16, scales32, n, y, f16_out, stream);
    if (m <= 48) return linear_launch<KIND, 3, 16>(x, m, k, w, scales16, zeros16, scales32, n, y, f16_out, stream);
    if (m <= 64) return linear_launch<KIND, 4, 16>(x, m, k, w, scales16, zeros16, scales32, n, y, f16_out, stream);
  }
  return hipErrorInvalidValue;
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

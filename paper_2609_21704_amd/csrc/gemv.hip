// Dequant-fused draft GEMVs (SpecQuant SS III-D.2: the draft parent Q4 or Q8
// produces the speculative tokens; every draft step streams the whole
// quantized stack once at m = 1 .. 8 activation rows).
//
// The kernels are HBM-bound: each weight byte is read once, with 16-byte
// loads, 32 contiguous bytes per lane per row.  Two work splits, chosen per
// launch by measured crossover (gemv_m):
//   gemv_kernel (tasks of rows): a task is a block of up to four rows; one
//     step of a task is 64 lanes x 32 bytes of each of its rows.  A team of
//     nw wavefronts (nw = 4 from four steps per task, 2 from two, else 1)
//     works on one task at a time, its wavefronts splitting the task's steps;
//     a workgroup holds T teams and stages the activations of its K range in
//     LDS once for all of them.  The grid is persistent, about 16 wavefronts
//     per CU: teams walk tasks with a stride of the total team count,
//     fetching their next step while computing the current one.  Row sums are
//     reduced across a wavefront with DPP and across a team's wavefronts
//     through LDS, in a fixed order; teams of several wavefronts advance
//     through their tasks in step with the workgroup's barriers (a team
//     without a task left runs an unstored copy of its last).  Where a task
//     is one step (INT4, m = 1, K within 64 chunks) the activations of a
//     lane's chunk stay in its registers for every task.  Its tasks of
//     two or four rows share each activation read: it takes the matrices with
//     many rows (gate|up, the LM head).
//   gemv_rows_kernel (row blocks, INT4, m <= 2): each CU's workgroups own a
//     contiguous block of rows, walked by their wavefronts in runs of whole
//     64-piece steps; it takes the launches where a task would be one row or
//     would leave lanes idle (q|k|v, o and down at 7B; every matrix with
//     rows of 1024 .. 1920 k, as at 1.5B).  Described at the kernel.
//
// INT4 (W4A16).  A lane's 32 bytes are 64 consecutive 4-bit codes of one row,
// i.e. half of one 128-element group.  Each 32-bit word (codes of k..k+7) is
// turned into four half2 values without a conversion instruction: a nibble
// masked into mantissa bits 0-3 (or 4-7) of the binary16 constant 1024 (or
// 64) is the exact value 1024 + q (or 64 + q); one shift by 8 serves the upper
// nibble pairs.  Subtracting the packed constant c + z in fp16 is exact and
// leaves q - z in [-15, 15], so v_dot2_f32_f16 forms exact products
// (q - z) * x and the fp32 accumulation error is bounded by sum |(q - z) x|;
// the group scale multiplies the half-group sum once.  Per word: one shift,
// four and-or, four packed subtracts, four dot2 -- 1.6 VALU operations per
// weight at m = 1.
//
// FP8 (W8A16).  A lane's 32 bytes are 32 E4M3 codes; v_cvt_scalef32_pk_f16_fp8
// converts two codes to two exact binary16 values, v_dot2_f32_f16
// accumulates, and the per-row fp32 scale is applied once after the reduction.
#include "sq_device.hpp"
#include "sq_internal.hpp"

namespace sq {
namespace {

// rows of a task, at most: four for m <= 2, two for m <= 4, one above, where
// the activation fragments need the registers.  A launch takes fewer when the
// matrix is too short to give every wavefront several tasks (measured: one row
// for the 7B q|k|v / o / down shapes, two for gate|up, four for the LM head).
constexpr int max_rows_for(int m) { return m <= 2 ? 4 : (m <= 4 ? 2 : 1); }
constexpr int kLaneBytes = 32;              // code bytes per lane per row and step
constexpr size_t kLdsBudget = 64 * 1024;    // activation bytes one workgroup may stage
constexpr int kWavesPerCu = 16;            // resident wavefronts per CU in the persistent grid
constexpr int kTeamsMax = 4;               // teams per workgroup, at most (2 for 4-wavefront teams; measured)

template <int V>
struct IntC {
  static constexpr int value = V;
};

template <int R>
struct Frag {
  u32x4 c[R][2];
  uint32_t s[R];  // INT4 group scale bits
  uint32_t z[R];  // INT4 group zero bits
};

// Where a task's rows start.  The last task may hold fewer than R rows:
// its extra rows read row n - 1 again and are never stored.
struct TaskPtr {
  const uint8_t* codes;   // row0's codes at the slice start
  const uint16_t* scales; // row0's group scales at the slice start (INT4)
  const uint16_t* zeros;
  int last;               // index of the task's last real row (0 .. R-1)
};

// SILU (R = 2): task t is the gate row t and the up row t + n / 2, at a pitch
// of n / 2 rows (the caller's row_bytes / groups of load_frag).
template <bool W8, int R, bool SILU = false>
__device__ __forceinline__ TaskPtr task_ptr(const uint8_t* __restrict__ codes, const uint16_t* __restrict__ scales,
                                            const uint16_t* __restrict__ zeros, int64_t n, int64_t k, int64_t k0,
                                            int64_t task) {
  TaskPtr t;
  const int64_t row0 = SILU ? task : task * R;
  const int64_t left = n - 1 - row0;
  t.last = SILU ? 1 : (left < R - 1 ? (int)left : R - 1);
  t.codes = codes + row0 * (W8 ? k : (k >> 1)) + (W8 ? k0 : (k0 >> 1));
  t.scales = W8 ? nullptr : scales + row0 * (k >> 7) + (k0 >> 7);
  t.zeros = W8 ? nullptr : zeros + row0 * (k >> 7) + (k0 >> 7);
  return t;
}

// A row base the wavefront holds in common, as a global-memory pointer: a
// load then adds only a zero-extended 32-bit lane offset to the scalar base
// (no 64-bit address arithmetic per lane).  The cast keeps all 64 bits.
template <class T>
using gptr = __attribute__((address_space(1))) const T*;
template <class T>
__device__ __forceinline__ gptr<T> uniform_ptr(const T* p) {
  return (gptr<T>)p;
}

// Codes of a task's rows for the lane's chunk of step `it`.  The loads are
// unconditional: a lane past the end of the slice reads the slice's last chunk
// again (its contribution is dropped in the compute), and an FP8 slice that
// ends on half a chunk (k % 32 == 16) reads its first 16 bytes twice; the
// copy meets zero activations in LDS.
template <bool W8, int R>
__device__ __forceinline__ Frag<R> load_frag(const TaskPtr& t, int row_bytes, int groups, int64_t kl, int nchunk,
                                             int it, int lane) {
  Frag<R> f;
  int chunk = it * kWave + lane;
  chunk = chunk < nchunk ? chunk : nchunk - 1;
  const bool hi = W8 ? (chunk * 32 + 16 < kl) : true;
  // a uniform row base plus a zero-extended 32-bit lane offset: the loads take
  // the scalar-base form, with no 64-bit address arithmetic per lane
  const uint32_t coff = (uint32_t)chunk * (uint32_t)kLaneBytes, goff = (uint32_t)chunk >> 1;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int rr = r < t.last ? r : t.last;
    const gptr<u32x4> p = (gptr<u32x4>)(uniform_ptr(t.codes + (int64_t)rr * row_bytes) + coff);
    f.c[r][0] = p[0];
    f.c[r][1] = p[hi ? 1 : 0];
    if constexpr (!W8) {
      f.s[r] = uniform_ptr(t.scales + (int64_t)rr * groups)[goff];
      f.z[r] = uniform_ptr(t.zeros + (int64_t)rr * groups)[goff];
    } else {
      f.s[r] = 0u;
      f.z[r] = 0u;
    }
  }
  return f;
}

// INT4 LDS layout for a K slice of nchunk 64-element chunks (lane-consecutive
// chunks are consecutive 16-byte cells): xs [M][8 words][nchunk][8 halves],
// halves of word w in the order x[8w+0], x[8w+4], x[8w+1], x[8w+5], x[8w+2],
// x[8w+6], x[8w+3], x[8w+7] -- the nibble pairs of a code word.
// FP8 layout: xs [M][4 cells][nchunk][8 halves] in natural order.
// halves (x0,x1),(x2,x3),(x4,x5),(x6,x7) -> (x0,x4),(x1,x5),(x2,x6),(x3,x7):
// the nibble pairs of an INT4 code word
__device__ __forceinline__ u32x4 pair_order(u32x4 raw) {
  u32x4 out;
  out[0] = __builtin_amdgcn_perm(raw[2], raw[0], 0x05040100u);
  out[1] = __builtin_amdgcn_perm(raw[2], raw[0], 0x07060302u);
  out[2] = __builtin_amdgcn_perm(raw[3], raw[1], 0x05040100u);
  out[3] = __builtin_amdgcn_perm(raw[3], raw[1], 0x07060302u);
  return out;
}

template <int M, bool W8>
__device__ __forceinline__ u32x4 x_cell(const uint16_t* __restrict__ x, int64_t k, int64_t k0, int64_t kl, int c,
                                        int m, int w) {
  const int64_t kk = (int64_t)c * (W8 ? 32 : 64) + 8 * w;
  const u32x4 raw = kk < kl ? *reinterpret_cast<const u32x4*>(x + (int64_t)m * k + k0 + kk) : u32x4{0u, 0u, 0u, 0u};
  return W8 ? raw : pair_order(raw);
}

// The same cell from a normalised row (INT4 order): h and norm weights of
// row m at k index kk = 64 c + 8 w, converted by rms_cell once r is known.
struct NormCell {
  float4_t h0, h1;
  u32x4 w;
};

__device__ __forceinline__ NormCell norm_cell_load(const NormSrc& nr, int64_t k, int c, int m, int w) {
  const int64_t kk = (int64_t)c * 64 + 8 * w;
  const float* hr = nr.h + ((int64_t)m * nr.group + nr.group - 1) * k + kk;
  NormCell f;
  f.h0 = *reinterpret_cast<const float4_t*>(hr);
  f.h1 = *reinterpret_cast<const float4_t*>(hr + 4);
  f.w = *reinterpret_cast<const u32x4*>(nr.w + kk);
  return f;
}

// Activations staged in LDS by the whole workgroup.  The loads of the first
// batch (B cells per thread, all of x for up to B * blockDim.x cells) are
// issued before the weight prefetch, so that they do not queue behind it in
// HBM; their stores follow once the weight loads are in flight.
// NRM (INT4, one K slice, 256 threads): the cells come from normalised rows;
// load() fetches their h and norm weights, convert() forms them once the
// rows' 1 / rms are known (2 M cells per thread cover K <= 4096).
template <int M, bool W8, bool NRM = false>
struct XStage {
  static constexpr int kCells = W8 ? 4 : 8;  // 16-byte cells of x per chunk and row
  // fewer held cells where the activation fragments need registers
  static constexpr int B = NRM ? 2 * M : (M <= 4 ? 8 : 2);
  u32x4 v[B];
  NormCell nc[NRM ? B : 1];

  __device__ __forceinline__ void load(const uint16_t* __restrict__ x, int64_t k, int64_t k0, int64_t kl, int nchunk,
                                       int base, const NormSrc& nr) {
    const int total = nchunk * M * kCells, nthreads = (int)blockDim.x;
#pragma unroll
    for (int i = 0; i < B; ++i) {
      int idx = base + i * nthreads + (int)threadIdx.x;
      idx = idx < total ? idx : total - 1;
      const int c = idx / (M * kCells), rem = idx % (M * kCells);
      if constexpr (NRM)
        nc[i] = norm_cell_load(nr, k, c, rem / kCells, rem % kCells);
      else
        v[i] = x_cell<M, W8>(x, k, k0, kl, c, rem / kCells, rem % kCells);
    }
  }

  __device__ __forceinline__ void convert(int nchunk, int base, const float (&r)[M]) {
    if constexpr (NRM) {
      const int total = nchunk * M * kCells, nthreads = (int)blockDim.x;
#pragma unroll
      for (int i = 0; i < B; ++i) {
        int idx = base + i * nthreads + (int)threadIdx.x;
        idx = idx < total ? idx : total - 1;
        const int m = (idx % (M * kCells)) / kCells;
        float rm = r[0];
#pragma unroll
        for (int mm = 1; mm < M; ++mm) rm = m == mm ? r[mm] : rm;
        v[i] = pair_order(rms_cell(nc[i].h0, nc[i].h1, nc[i].w, rm));
      }
    }
  }

  __device__ __forceinline__ void store(int nchunk, int base, half_t* xs) const {
    const int total = nchunk * M * kCells, nthreads = (int)blockDim.x;
#pragma unroll
    for (int i = 0; i < B; ++i) {
      const int idx = base + i * nthreads + (int)threadIdx.x;
      if (idx < total) {
        const int c = idx / (M * kCells), rem = idx % (M * kCells), m = rem / kCells, w = rem % kCells;
        *reinterpret_cast<u32x4*>(xs + (((size_t)m * kCells + w) * nchunk + c) * 8) = v[i];
      }
    }
  }
};

// Output modes of the projection kernels: y fp32, y fp16, y fp32 added to, or
// (SILU, tasks of a gate and an up row) t = f16(silu(gate) * up) [m][n / 2].
enum : int { kOutF32 = 0, kOutF16 = 1, kOutAcc = 2, kOutSilu = 3 };

__device__ __forceinline__ void store_mode(void* y, int64_t idx, float v, int out_mode) {
  if (out_mode == kOutF16)
    reinterpret_cast<uint16_t*>(y)[idx] = f32_to_f16_bits(v);
  else if (out_mode == kOutAcc)
    reinterpret_cast<float*>(y)[idx] += v;
  else
    reinterpret_cast<float*>(y)[idx] = v;
}

template <int M, bool W8, int R, bool MULTI, bool XR, bool NRM, bool SILU>
__global__ __launch_bounds__(1024) void gemv_kernel(const uint16_t* __restrict__ x, int64_t k, int64_t kslice,
                                                       const uint8_t* __restrict__ codes,
                                                       const uint16_t* __restrict__ scales16,
                                                       const uint16_t* __restrict__ zeros16,
                                                       const float* __restrict__ scales32, int64_t n,
                                                       void* __restrict__ y, int out_mode,
                                                       float* __restrict__ partial, int nw_team, NormSrc nr) {
  extern __shared__ __align__(16) char smem[];
  // every argument in one batch of scalar loads, before the first address needs one
  asm volatile("" ::"s"(x), "s"(k), "s"(kslice), "s"(codes), "s"(scales16), "s"(zeros16), "s"(scales32), "s"(n),
               "s"(y), "s"(out_mode), "s"(partial), "s"(nw_team));
  constexpr int kCells = W8 ? 4 : 8;
  constexpr int kChunkK = W8 ? 32 : 64;  // weights per 32-byte lane chunk
  const int split = blockIdx.y;
  const int64_t k0 = (int64_t)split * kslice;
  const int64_t kl = (k - k0) < kslice ? (k - k0) : kslice;
  const int nchunk = (int)((kl + kChunkK - 1) / kChunkK);
  const int nit = (nchunk + kWave - 1) / kWave;  // >= nw by the host's choice of nw
  const int nw = MULTI ? nw_team : 1;            // wavefronts per team
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int team = wave / nw, wt = wave - team * nw;  // team in the workgroup, wavefront in the team
  const int nteam = (int)(blockDim.x >> 6) / nw;      // teams per workgroup
  const int64_t tstride = (int64_t)gridDim.x * nteam;  // teams in the grid: the task stride
  const int64_t ntask = SILU ? n / 2 : (n + R - 1) / R;
  // multi-wavefront teams meet at barriers, so every team of the grid runs
  // the same number of tasks (ntask_pad / tstride); single-wavefront teams
  // stop at ntask
  const int64_t ntask_pad = MULTI ? (ntask + tstride - 1) / tstride * tstride : ntask;
  int64_t task = (int64_t)blockIdx.x * nteam + team;
  int it = wt;
  half_t* xs = reinterpret_cast<half_t*>(smem);
  float* red = reinterpret_cast<float*>(smem + (size_t)M * kCells * nchunk * 16);  // [teams][nw][R][M]

  // distance between the rows of a task: one row, or n / 2 rows (SILU)
  const int row_bytes = (int)(W8 ? k : (k >> 1)) * (SILU ? (int)(n >> 1) : 1);
  const int groups = (int)(k >> 7) * (SILU ? (int)(n >> 1) : 1);

  // activations first, then the first fragment, so that x is not queued
  // behind the weight stream
  // NRM: the rows' sums of squares are loaded first, then the cells' h and
  // norm weights; 1 / rms meets in LDS (after the activation cells) before the
  // cells are formed
  RmsRows<NRM ? M : 1> rr;
  if constexpr (NRM) rr.load(nr.h + (int64_t)(nr.group - 1) * k, (int64_t)nr.group * k, M, (int)k);
  XStage<M, W8, NRM> xst;
  xst.load(x, k, k0, kl, nchunk, 0, nr);
  Frag<R> fa, fb;
  TaskPtr tp = task_ptr<W8, R, SILU>(codes, scales16, zeros16, n, k, k0, task < ntask ? task : ntask - 1);
  fa = load_frag<W8, R>(tp, row_bytes, groups, kl, nchunk, it, lane);
  if constexpr (NRM) {
    float* wsum = reinterpret_cast<float*>(smem + (size_t)M * kCells * nchunk * 16);  // [M][4]
    rr.finish(M, (int)k, wsum);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    float r[M];
#pragma unroll
    for (int m = 0; m < M; ++m) r[m] = rms_inverse(wsum + 4 * m, (int)k, nr.eps);
    xst.convert(nchunk, 0, r);
  }
  xst.store(nchunk, 0, xs);
  const int xtotal = nchunk * M * kCells, xbatch = XStage<M, W8, NRM>::B * (int)blockDim.x;
  for (int base = xbatch; !NRM && base < xtotal; base += xbatch) {  // activations beyond the first batch
    xst.load(x, k, k0, kl, nchunk, base, nr);
    xst.store(nchunk, base, xs);
  }
  __syncthreads();
  if (task >= ntask_pad) return;  // uniform across the wavefront; never for a multi-wavefront team

  // XR: a task is one step (K within 64 chunks), so a lane meets the same
  // activation chunk in every task; its cells are read from LDS once, here,
  // and stay in registers (measured: 7B gate|up 17.0 -> 16.5 us, LM head
  // 55.3 -> 54.6 us at m = 1)
  u32x4 xr[XR ? M : 1][XR ? kCells : 1];
  if constexpr (XR) {
    const int cc0 = lane < nchunk ? lane : nchunk - 1;
#pragma unroll
    for (int m = 0; m < M; ++m)
#pragma unroll
      for (int w = 0; w < kCells; ++w)
        xr[m][w] = *reinterpret_cast<const u32x4*>(xs + (((size_t)m * kCells + w) * nchunk + cc0) * 8);
  }

  // masks and magic numbers in VGPRs, so each mask-and-insert is one v_and_or_b32
  uint32_t mlo = 0x000F000Fu, mhi = 0x00F000F0u, k1024 = 0x64006400u, k64 = 0x54005400u;
  asm("" : "+v"(mlo), "+v"(mhi), "+v"(k1024), "+v"(k64));

  float acc[R][M];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int m = 0; m < M; ++m) acc[r][m] = 0.f;

  // One step (task, it): fetch this wavefront's next step into `nxt`, then
  // consume `cur`; after the task's last step the row sums are finished.
  // Returns false when the workgroup has no tasks left.
  auto step = [&](const Frag<R>& cur, Frag<R>& nxt) -> bool {
    int64_t task_n = task;
    int it_n = it + nw;
    if (it_n >= nit) {
      it_n = wt;
      task_n = task + tstride;
    }
    const TaskPtr tp_n = task_n == task ? tp : task_ptr<W8, R, SILU>(codes, scales16, zeros16, n, k, k0,
                                                             task_n < ntask ? task_n : ntask - 1);
    nxt = load_frag<W8, R>(tp_n, row_bytes, groups, kl, nchunk, it_n, lane);

    const int chunk = it * kWave + lane;
    const bool ok = chunk < nchunk;
    const int cc = ok ? chunk : nchunk - 1;
    float a[R][M];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int m = 0; m < M; ++m) a[r][m] = 0.f;

    if constexpr (!W8) {
      half2_t c1024[R], c64[R];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const uint32_t zb = cur.z[r];
        const half2_t z2 = __builtin_bit_cast(half2_t, zb | (zb << 16));
        c1024[r] = z2 + half2_t{(half_t)1024.0f, (half_t)1024.0f};
        c64[r] = z2 + half2_t{(half_t)64.0f, (half_t)64.0f};
      }
#pragma unroll
      for (int w = 0; w < 8; ++w) {
        half2_t xw[M][4];
#pragma unroll
        for (int m = 0; m < M; ++m) {
          const u32x4 v =
              XR ? xr[m][XR ? w : 0] : *reinterpret_cast<const u32x4*>(xs + (((size_t)m * kCells + w) * nchunk + cc) * 8);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const uint32_t e = v[i];  // bit-cast a scalar copy: the element lvalue itself is misread
            xw[m][i] = __builtin_bit_cast(half2_t, e);
          }
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
          const uint32_t q = cur.c[r][w >> 2][w & 3];
          const uint32_t q8 = q >> 8;
          const half2_t d0 = __builtin_bit_cast(half2_t, (q & mlo) | k1024) - c1024[r];   // q0 - z, q4 - z
          const half2_t d1 = __builtin_bit_cast(half2_t, (q & mhi) | k64) - c64[r];       // q1 - z, q5 - z
          const half2_t d2 = __builtin_bit_cast(half2_t, (q8 & mlo) | k1024) - c1024[r];  // q2 - z, q6 - z
          const half2_t d3 = __builtin_bit_cast(half2_t, (q8 & mhi) | k64) - c64[r];      // q3 - z, q7 - z
#pragma unroll
          for (int m = 0; m < M; ++m) {
            float t = a[r][m];
            t = __builtin_amdgcn_fdot2(d0, xw[m][0], t, false);
            t = __builtin_amdgcn_fdot2(d1, xw[m][1], t, false);
            t = __builtin_amdgcn_fdot2(d2, xw[m][2], t, false);
            t = __builtin_amdgcn_fdot2(d3, xw[m][3], t, false);
            a[r][m] = t;
          }
        }
      }
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const float s = ok ? f16_bits_to_f32((uint16_t)cur.s[r]) : 0.f;  // a lane past the end adds 0
#pragma unroll
        for (int m = 0; m < M; ++m) acc[r][m] += s * a[r][m];
      }
    } else {
#pragma unroll
      for (int cell = 0; cell < 4; ++cell) {
        half2_t xw[M][4];
#pragma unroll
        for (int m = 0; m < M; ++m) {
          const u32x4 v = *reinterpret_cast<const u32x4*>(xs + (((size_t)m * kCells + cell) * nchunk + cc) * 8);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const uint32_t e = v[i];  // bit-cast a scalar copy: the element lvalue itself is misread
            xw[m][i] = __builtin_bit_cast(half2_t, e);
          }
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
          const uint32_t q0 = cur.c[r][cell >> 1][2 * (cell & 1)];
          const uint32_t q1 = cur.c[r][cell >> 1][2 * (cell & 1) + 1];
          const half2_t w0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(q0, 1.0f, false);
          const half2_t w1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(q0, 1.0f, true);
          const half2_t w2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(q1, 1.0f, false);
          const half2_t w3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(q1, 1.0f, true);
#pragma unroll
          for (int m = 0; m < M; ++m) {
            float t = a[r][m];
            t = __builtin_amdgcn_fdot2(w0, xw[m][0], t, false);
            t = __builtin_amdgcn_fdot2(w1, xw[m][1], t, false);
            t = __builtin_amdgcn_fdot2(w2, xw[m][2], t, false);
            t = __builtin_amdgcn_fdot2(w3, xw[m][3], t, false);
            a[r][m] = t;
          }
        }
      }
#pragma unroll
      for (int r = 0; r < R; ++r)
#pragma unroll
        for (int m = 0; m < M; ++m) acc[r][m] += ok ? a[r][m] : 0.f;
    }

    if (task_n != task) {  // this wavefront's last step of the task
      constexpr int T = (R * M + 3) / 4;
      float v[4 * T];
#pragma unroll
      for (int i = 0; i < 4 * T; ++i) v[i] = i < R * M ? acc[i / M][i % M] : 0.f;
#pragma unroll
      for (int r = 0; r < R; ++r)
#pragma unroll
        for (int m = 0; m < M; ++m) acc[r][m] = 0.f;
      float w[T];
      wave_sums<T>(v, w);
      // lane 16 j holds value 4 t + (0, 2, 1, 3)[j] in w[t]
      const int rowsel = lane >> 4;
      const int which = rowsel == 0 ? 0 : (rowsel == 1 ? 2 : (rowsel == 2 ? 1 : 3));
      const bool lead = (lane & 15) == 0;
      auto emit = [&](int idx, float val) {
        const int r = idx / M, m = idx % M;
        const int64_t row = task * R + r;
        if (row >= n) return;  // also every row of a padding task (task >= ntask)
        if constexpr (W8) val *= scales32[row];
        if (partial)
          partial[((int64_t)split * M + m) * n + row] = val;
        else
          store_mode(y, (int64_t)m * n + row, val, out_mode);
      };
      if constexpr (SILU) {
        // gate of row m = 0 in lane 0 and (M = 2) of m = 1 in lane 32; its up
        // value 32 (M = 1) or 16 (M = 2) lanes above: t[m][task] = silu(g) u
        const float up = __shfl(w[0], lane + (M == 1 ? 32 : 16), kWave);
        if (lane == 0 || (M == 2 && lane == 32))
          reinterpret_cast<uint16_t*>(y)[(int64_t)(lane >> 5) * (n >> 1) + task] = silu_gate_bits(w[0], up);
      } else if constexpr (!MULTI) {
        if (lead) {
#pragma unroll
          for (int t = 0; t < T; ++t) {
            const int idx = 4 * t + which;
            if (idx < R * M) emit(idx, w[t]);
          }
        }
      } else {
        if (lead) {
#pragma unroll
          for (int t = 0; t < T; ++t) {
            const int idx = 4 * t + which;
            if (idx < R * M) red[wave * R * M + idx] = w[t];
          }
        }
        __syncthreads();
        if (wt == 0 && lane < R * M) {
          float out = red[(team * nw) * R * M + lane];
          for (int wv = 1; wv < nw; ++wv) out += red[(team * nw + wv) * R * M + lane];
          emit(lane, out);
        }
        __syncthreads();
      }
    }
    task = task_n;
    it = it_n;
    tp = tp_n;
    return task < ntask_pad;
  };

  while (step(fa, fb) && step(fb, fa)) {
  }
}

// INT4 GEMV over row blocks (k >= 1024, m <= 2).  A workgroup of NWV
// wavefronts (16 per CU in all) owns a contiguous block of rows, whose codes
// are one contiguous byte range of 32-byte pieces (64 codes, half a group).
// A wavefront walks a run of it in steps of 64 consecutive pieces.  The runs
// are whole steps, as even as the step count allows, and the odd steps go to
// the oldest wavefronts, which the memory system serves first (measured: runs
// of equal bytes, whose last step often held a few pieces, were up to 1.3 us
// slower on the 7B down projection).  D steps of loads are in flight (the
// host takes D = 1: with 16 wavefronts of a CU streaming, every deeper
// prefetch measured slower).  A row holds at least 16 pieces, so a step meets
// at most NA rows (five for 16 .. 21 pieces a row, four to 31, three to 63,
// two from 64 on): each lane adds its piece into the sum of its row, and when
// the walk leaves a row the wavefront reduces that row's sum into an LDS slot
// [wavefront][row].  After one
// barrier each row is the sum of its NWV slots in wavefront order
// (deterministic).  Activations are staged in LDS chunk-major with one pad
// cell per 64-element chunk (a 144-byte stride), so a lane reads its eight
// cells at immediate offsets and the 16 lanes of one read fall in different
// banks.
//
// FP8 (W8) takes the same walk with 32 codes to a piece: a lane converts its
// codes two at a time (v_cvt_scalef32_pk_f16_fp8, exact), the activations are
// staged in plain k order with four cells and one pad cell to a chunk (an
// 80-byte stride, again 16 lanes on distinct banks), and the row scale
// multiplies each finished row sum.  Up to four activation rows (m <= 4).
struct PieceFrag {
  u32x4 c[2];  // 32 bytes of codes
  uint32_t s;  // group scale bits (INT4)
  uint32_t z;  // group zero bits (INT4)
};

template <int M, bool W8, int D, int XB, int NA, int NWV, bool NRM>
__global__ __launch_bounds__(1024) void gemv_rows_kernel(const uint16_t* __restrict__ x, int64_t k,
                                                        const uint8_t* __restrict__ codes,
                                                        const uint16_t* __restrict__ scales16,
                                                        const uint16_t* __restrict__ zeros16, int64_t rows_q,
                                                        int rows_rem, const float* __restrict__ scales32,
                                                        int64_t n, void* __restrict__ y, int out_mode,
                                                        NormSrc nr) {
  extern __shared__ __align__(16) char smem[];
  // The arguments the first loads need come first: the library is built with
  // the first 14 argument dwords preloaded into scalar registers at dispatch,
  // so the activation and code loads issue without waiting for a kernel-
  // argument load.
  asm volatile("" ::"s"(x), "s"(k), "s"(codes), "s"(scales16), "s"(zeros16), "s"(rows_q), "s"(rows_rem));
  constexpr int kCPC = W8 ? 4 : 8;  // activation cells (8 halves) per chunk of a piece
  constexpr int kPad = kCPC + 1;    // LDS cells per chunk: the cells and one pad
  constexpr int nwave = NWV;        // wavefronts per workgroup, a power of two
  // no integer division on the way to the first load: block b holds rows_q
  // rows, plus one for b < rows_rem
  const int b = blockIdx.x;
  const int64_t r0 = (int64_t)b * rows_q + (b < rows_rem ? b : rows_rem);
  const int nrows = (int)rows_q + (b < rows_rem ? 1 : 0);
  const int ppr = (int)(k >> (W8 ? 5 : 6));  // pieces per row (and activation chunks)
  const int P = nrows * ppr;      // pieces of the block (< 2^27 by the host's check)
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // runs of whole steps: sb each, one more for the sx oldest wavefronts
  const int T = (P + 63) >> 6;  // steps of the block
  const int sb = T / nwave, sx = T - sb * nwave;  // nwave: a power of two
  const int ps0 = 64 * (wave * sb + (wave < sx ? wave : sx));
  const int ps = ps0 < P ? ps0 : P, pe0 = ps0 + 64 * (sb + (wave < sx ? 1 : 0)), pe = pe0 < P ? pe0 : P;
  const int nsteps = (pe - ps + 63) >> 6;
  half_t* xs = reinterpret_cast<half_t*>(smem);
  // NRM: the rows' wavefront sums of squares [M][4] after the activations, then the row sums
  float* wsum = reinterpret_cast<float*>(smem + (size_t)M * ppr * kPad * 16);
  float* red = reinterpret_cast<float*>(smem + (size_t)M * ppr * kPad * 16 + (NRM ? 64 : 0));  // [nwave][M][nrows]
  const uint8_t* bcodes = codes + r0 * (W8 ? k : (k >> 1));
  const uint16_t* bscales = W8 ? nullptr : scales16 + r0 * (k >> 7);
  const uint16_t* bzeros = W8 ? nullptr : zeros16 + r0 * (k >> 7);

  // piece p of the block: codes at 32 p, group p / 2 (rows hold whole groups);
  // a lane past the run reads the run's last piece again and adds nothing.
  // Every load is unconditional, so that the compiler can count the loads in
  // flight and wait only for the oldest.
  auto load = [&](int s) -> PieceFrag {
    PieceFrag f;
    int p = ps + 64 * s + lane;
    p = p < pe ? p : pe - 1;
    p = p > 0 ? p : 0;  // a run without pieces reads piece 0
    // a zero-extended 32-bit offset from the block base (p < 2^27): scalar-base loads
    const u32x4* cp = reinterpret_cast<const u32x4*>(bcodes + (uint32_t)p * 32u);
    f.c[0] = cp[0];
    f.c[1] = cp[1];
    if constexpr (!W8) {
      f.s = bscales[(uint32_t)p >> 1];
      f.z = bzeros[(uint32_t)p >> 1];
    } else {
      f.s = f.z = 0u;
    }
    return f;
  };

  // activations first (XB cells per thread cover all of x: the host's
  // choice), then the first D steps of codes
  const int cpm = ppr * kCPC, xtotal = M * cpm, nthr = (int)blockDim.x;  // cells per activation row, in all
  u32x4 xv[XB];
  // flat cell index -> (activation row, cell within the row); m <= 4
  auto xsplit = [&](int idx, int& m, int& rem) {
    m = 0;
    rem = idx;
#pragma unroll
    for (int i = 1; i < M; ++i)
      if (rem >= cpm) {
        rem -= cpm;
        ++m;
      }
  };
  NormCell xn[NRM ? XB : 1];
  auto xload = [&](int base) {
#pragma unroll
    for (int b = 0; b < XB; ++b) {
      int idx = base + b * nthr + (int)threadIdx.x;
      idx = idx < xtotal ? idx : xtotal - 1;
      int m, rem;
      xsplit(idx, m, rem);
      if constexpr (NRM)
        xn[b] = norm_cell_load(nr, k, rem / kCPC, m, rem % kCPC);
      else
        xv[b] = x_cell<M, W8>(x, k, 0, k, rem / kCPC, m, rem % kCPC);
    }
  };
  auto xstore = [&](int base) {
#pragma unroll
    for (int b = 0; b < XB; ++b) {
      const int idx = base + b * nthr + (int)threadIdx.x;
      if (idx < xtotal) {
        int m, rem;
        xsplit(idx, m, rem);
        *reinterpret_cast<u32x4*>(xs + (((size_t)m * ppr + rem / kCPC) * kPad + rem % kCPC) * 8) = xv[b];
      }
    }
  };
  RmsRows<1> rr;  // NRM: M <= 2 rows over groups of 256 threads (512 or 1024)
  if constexpr (NRM) rr.load(nr.h + (int64_t)(nr.group - 1) * k, (int64_t)nr.group * k, M, (int)k);
  xload(0);
  PieceFrag ring[D];
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
    for (int b = 0; b < XB; ++b) {
      int idx = b * nthr + (int)threadIdx.x;
      idx = idx < xtotal ? idx : xtotal - 1;
      int m, rem;
      xsplit(idx, m, rem);
      float rm = r[0];
#pragma unroll
      for (int mm = 1; mm < M; ++mm) rm = m == mm ? r[mm] : rm;
      xv[b] = pair_order(rms_cell(xn[b].h0, xn[b].h1, xn[b].w, rm));
    }
  }
  xstore(0);
  for (int i = (int)threadIdx.x; i < M * nrows * nwave; i += nthr) red[i] = 0.f;
  // an accumulated output: this thread's first value read now, its latency under the walk
  float yold = 0.f;
  if (out_mode == kOutAcc && (int)threadIdx.x < M * nrows) {
    int m = 0, row = (int)threadIdx.x;
#pragma unroll
    for (int i = 1; i < M; ++i)
      if (row >= nrows) {
        row -= nrows;
        ++m;
      }
    yold = reinterpret_cast<const float*>(y)[(int64_t)m * n + r0 + row];
  }
  // LDS writes done, then the barrier: no wait for the code loads in flight
  // (a full __syncthreads would wait for every outstanding global load)
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();

  uint32_t mlo = 0x000F000Fu, mhi = 0x00F000F0u, k1024 = 0x64006400u, k64 = 0x54005400u;
  asm("" : "+v"(mlo), "+v"(mhi), "+v"(k1024), "+v"(k64));

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
    float v[4] = {a[0], M > 1 ? a[1] : 0.f, M > 2 ? a[2] : 0.f, M > 3 ? a[3] : 0.f};
    float w[1];
    wave_sums<1>(v, w);
    // lane 16 j holds the total of v[(0, 2, 1, 3)[j]]
    if (lane == 0) red[wave * M * nrows + row] = w[0];
    if (M > 1 && lane == 32) red[(wave * M + 1) * nrows + row] = w[0];
    if (M > 2 && lane == 16) red[(wave * M + 2) * nrows + row] = w[0];
    if (M > 3 && lane == 48) red[(wave * M + 3) * nrows + row] = w[0];
  };

  auto compute = [&](const PieceFrag& f) {
    // the lane's row is crow + rel: a step of 64 pieces meets at most NA rows
    int chunk = coff + lane, rel = 0;
#pragma unroll
    for (int i = 1; i < NA; ++i)
      if (chunk >= ppr) {
        chunk -= ppr;
        rel = i;
      }
    const bool ok = cb + lane < pe;
    if constexpr (W8) {
      float a[M];
#pragma unroll
      for (int m = 0; m < M; ++m) a[m] = 0.f;
#pragma unroll
      for (int w = 0; w < 4; ++w) {  // cell w: codes 8 w .. 8 w + 7, the words 2 w and 2 w + 1
        const uint32_t q0 = f.c[w >> 1][2 * (w & 1)], q1 = f.c[w >> 1][2 * (w & 1) + 1];
        const half2_t h0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(q0, 1.0f, false);
        const half2_t h1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(q0, 1.0f, true);
        const half2_t h2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(q1, 1.0f, false);
        const half2_t h3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(q1, 1.0f, true);
#pragma unroll
        for (int m = 0; m < M; ++m) {
          const u32x4 v = *reinterpret_cast<const u32x4*>(xs + (((size_t)m * ppr + chunk) * kPad + w) * 8);
          const uint32_t e0 = v[0], e1 = v[1], e2 = v[2], e3 = v[3];  // scalar copies, as elsewhere
          float t = a[m];
          t = __builtin_amdgcn_fdot2(h0, __builtin_bit_cast(half2_t, e0), t, false);
          t = __builtin_amdgcn_fdot2(h1, __builtin_bit_cast(half2_t, e1), t, false);
          t = __builtin_amdgcn_fdot2(h2, __builtin_bit_cast(half2_t, e2), t, false);
          t = __builtin_amdgcn_fdot2(h3, __builtin_bit_cast(half2_t, e3), t, false);
          a[m] = t;
        }
      }
#pragma unroll
      for (int m = 0; m < M; ++m) {
        const float v = ok ? a[m] : 0.f;
#pragma unroll
        for (int i = 0; i < NA; ++i) acc[i][m] += rel == i ? v : 0.f;
      }
      return;
    }
    const uint32_t zb = f.z;
    const half2_t z2 = __builtin_bit_cast(half2_t, zb | (zb << 16));
    const half2_t c1024 = z2 + half2_t{(half_t)1024.0f, (half_t)1024.0f};
    const half2_t c64 = z2 + half2_t{(half_t)64.0f, (half_t)64.0f};
    float a[M];
#pragma unroll
    for (int m = 0; m < M; ++m) a[m] = 0.f;
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      const uint32_t q = f.c[w >> 2][w & 3];
      const uint32_t q8 = q >> 8;
      const half2_t d0 = __builtin_bit_cast(half2_t, (q & mlo) | k1024) - c1024;   // q0 - z, q4 - z
      const half2_t d1 = __builtin_bit_cast(half2_t, (q & mhi) | k64) - c64;       // q1 - z, q5 - z
      const half2_t d2 = __builtin_bit_cast(half2_t, (q8 & mlo) | k1024) - c1024;  // q2 - z, q6 - z
      const half2_t d3 = __builtin_bit_cast(half2_t, (q8 & mhi) | k64) - c64;      // q3 - z, q7 - z
#pragma unroll
      for (int m = 0; m < M; ++m) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(xs + (((size_t)m * ppr + chunk) * kPad + w) * 8);
        const uint32_t e0 = v[0], e1 = v[1], e2 = v[2], e3 = v[3];  // scalar copies, as elsewhere
        float t = a[m];
        t = __builtin_amdgcn_fdot2(d0, __builtin_bit_cast(half2_t, e0), t, false);
        t = __builtin_amdgcn_fdot2(d1, __builtin_bit_cast(half2_t, e1), t, false);
        t = __builtin_amdgcn_fdot2(d2, __builtin_bit_cast(half2_t, e2), t, false);
        t = __builtin_amdgcn_fdot2(d3, __builtin_bit_cast(half2_t, e3), t, false);
        a[m] = t;
      }
    }
    const float sc = f16_bits_to_f32((uint16_t)f.s);
#pragma unroll
    for (int m = 0; m < M; ++m) {
      const float v = ok ? sc * a[m] : 0.f;
#pragma unroll
      for (int i = 0; i < NA; ++i) acc[i][m] += rel == i ? v : 0.f;
    }
  };

  for (int s0 = 0; s0 < nsteps; s0 += D) {
#pragma unroll
    for (int j = 0; j < D; ++j) {
      const int s = s0 + j;
      if (s < nsteps) {
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
        compute(ring[j]);
        cb += 64;
        coff += 64;
        while (coff >= ppr) {
          coff -= ppr;
          ++crow;
        }
      }
      ring[j] = load(s + D);
    }
  }
  if (nsteps > 0) {
#pragma unroll
    for (int i = 0; i < NA; ++i)
      if (cur + i < nrows) flush(acc[i], cur + i);
  }
  __syncthreads();
  for (int t = (int)threadIdx.x; t < M * nrows; t += nthr) {
    int m = 0, row = t;
#pragma unroll
    for (int i = 1; i < M; ++i)
      if (row >= nrows) {
        row -= nrows;
        ++m;
      }
    float v = 0.f;
    for (int w = 0; w < nwave; ++w) v += red[w * M * nrows + t];  // consecutive threads, consecutive words
    if constexpr (W8) v *= scales32[r0 + row];
    const int64_t o = (int64_t)m * n + r0 + row;
    if (out_mode == kOutAcc && t == (int)threadIdx.x)  // the value read at the start
      reinterpret_cast<float*>(y)[o] = yold + v;
    else
      store_mode(y, o, v, out_mode);
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

template <int M, bool W8, int R, bool MULTI, bool XR, bool NRM, bool SILU = false>
hipError_t gemv_launch(const uint16_t* x, int64_t k, int64_t kslice, int splits, const uint8_t* codes,
                       const uint16_t* scales16, const uint16_t* zeros16, const float* scales32, int64_t n, void* y,
                       int out_mode, float* partial, int nw, const NormSrc& nr, hipStream_t stream) {
  constexpr int64_t chunk_k = W8 ? 32 : 64;
  const int64_t kfirst = kslice < k ? kslice : k;
  const int64_t nchunk = (kfirst + chunk_k - 1) / chunk_k;
  const int64_t ntask = SILU ? n / 2 : (n + R - 1) / R;
  const int64_t cus = cu_count();
  // teams: as many as the CUs hold (kWavesPerCu wavefronts each) or
  // as there are tasks; teams per workgroup: enough to cover the CUs once
  const int64_t per_cu = kWavesPerCu / nw > 0 ? kWavesPerCu / nw : 1;
  int64_t teams = ntask < cus * per_cu / splits ? ntask : cus * per_cu / splits;
  if (teams < 1) teams = 1;
  int64_t T = (teams + cus / splits - 1) / (cus / splits > 0 ? cus / splits : 1);
  if (T > per_cu) T = per_cu;
  // teams per workgroup: at most kTeamsMax (half that for teams of four or
  // more wavefronts), and a divisor of the teams per CU, so that workgroups tile the CUs
  int64_t tmax = nw >= 4 ? (kTeamsMax + 1) / 2 : kTeamsMax;
  while (tmax > 1 && per_cu % tmax != 0) --tmax;
  if (T > tmax) T = tmax;
  if (T < 1) T = 1;
  const int64_t blocks = (teams + T - 1) / T;
  // normalised rows: one K slice staged by 256 threads, 2 M cells each
  if (NRM && (splits != 1 || T * nw != 4 || nchunk > 64)) return hipErrorNotSupported;
  // SiLU pairs: rows t and t + n / 2 of a task, at a pitch that fits 32 bits
  if (SILU && (n % 2 != 0 || (n / 2) * (k / 2) >= (int64_t(1) << 31))) return hipErrorNotSupported;
  const size_t lds = (size_t)M * 2 * (size_t)(nchunk * chunk_k) + (MULTI ? (size_t)T * nw * R * M * 4 : 0) +
                     (NRM ? (size_t)M * 4 * sizeof(float) : 0);
  const dim3 grid((unsigned)blocks, (unsigned)splits);
  hipLaunchKernelGGL((gemv_kernel<M, W8, R, MULTI, XR, NRM, SILU>), grid, dim3((unsigned)(T * nw * 64)), lds, stream, x, k,
                     kslice, codes, scales16, zeros16, scales32, n, y, out_mode, partial, nw, nr);
  return hipGetLastError();
}

constexpr int64_t kRowsMinK = 1024;  // shortest rows the row-block kernel takes
constexpr int kRowsDepth = 1;        // steps of loads in flight per wavefront (measured: 1 < 2 < 3 < 4 in time)
constexpr size_t kRowsLdsMax = 150 * 1024;

// Host side of the row-block kernel (INT4 m <= 2, FP8 m <= 4): 16 wavefronts
// per CU (fewer workgroups than rows never), rows split evenly over the
// workgroups.  Returns hipErrorNotSupported when the shape is outside what it
// takes.
template <int M, bool W8, bool NRM>
hipError_t gemv_rows_m(const uint16_t* x, int64_t k, const uint8_t* codes, const uint16_t* scales16,
                       const uint16_t* zeros16, const float* scales32, int64_t n, void* y, int out_mode,
                       const NormSrc& nr, hipStream_t stream) {
  // whole pieces per row: 32 FP8 codes, or 64 INT4 codes (k % 128 == 0 already);
  // normalised rows (INT4) of at most 4096 values, two cells per thread at most
  if (M > (W8 ? 4 : 2) || k < kRowsMinK || (W8 && k % 32 != 0) || (NRM && (W8 || k > 4096)))
    return hipErrorNotSupported;
  // 16 wavefronts per CU: one workgroup of 16, or two of 8 for INT4 rows of
  // 8192 k and more (measured: 7B down 13.5 -> 12.8 us, q|k|v 5.8 -> 6.0 us)
  const int nwave = !W8 && k >= 8192 && M * k <= 8 * 8 * 512 ? 8 : 16, nthr = 64 * nwave;  // 8: x in one pass
  const int64_t wg_max = cu_count() * (16 / nwave);
  const int64_t blocks = n < wg_max ? n : wg_max;
  const int64_t rows_max = (n + blocks - 1) / blocks;
  const int64_t ppr = k >> (W8 ? 5 : 6);
  constexpr int64_t cpc = W8 ? 4 : 8;  // activation cells per chunk
  const size_t lds =
      (size_t)M * ppr * (cpc + 1) * 16 + (NRM ? 64 : 0) + (size_t)M * rows_max * nwave * sizeof(float);
  const int64_t xcells = M * ppr * cpc;  // 16-byte activation cells, staged by the workgroup at once
  if (lds > kRowsLdsMax || rows_max * ppr >= (int64_t(1) << 27) || xcells > (NRM ? 2 : 8) * nthr)
    return hipErrorNotSupported;
  constexpr int D = kRowsDepth;
  const int64_t q = n / blocks;
  const int rem = (int)(n % blocks);
  // workgroups of 8 wavefronts take over a third of the LDS, so that a CU holds
  // two of them (the registers would allow three)
  const size_t lds_launch = nwave == 8 && lds < 54 * 1024 ? 54 * 1024 : lds;
  auto go = [&](auto xb_tag, auto na_tag, auto nw_tag) {
    constexpr int XB = decltype(xb_tag)::value, NA = decltype(na_tag)::value, NWV = decltype(nw_tag)::value;
    hipLaunchKernelGGL((gemv_rows_kernel<M, W8, D, XB, NA, NWV, NRM>), dim3((unsigned)blocks), dim3(nthr),
                       lds_launch, stream, x, k, codes, scales16, zeros16, q, rem, scales32, n, y, out_mode, nr);
  };
  // the fewest activation cells per thread that cover the activations: the
  // loads past the end are redundant and delay the code loads behind them
  // (measured: 7B q|k|v 5.9 -> 5.5 us, o 5.45 -> 5.12 us with one cell)
  auto pick = [&](auto na_tag, auto nw_tag) {
    if (xcells <= nthr)
      go(IntC<1>{}, na_tag, nw_tag);
    else if constexpr (NRM)  // at most two cells (the host's check above)
      go(IntC<2>{}, na_tag, nw_tag);
    else if (xcells <= 2 * nthr)
      go(IntC<2>{}, na_tag, nw_tag);
    else if (xcells <= 4 * nthr)
      go(IntC<4>{}, na_tag, nw_tag);
    else
      go(IntC<8>{}, na_tag, nw_tag);
  };
  if (nwave == 8)  // INT4, k >= 8192: two rows per step at most
    pick(IntC<2>{}, IntC<8>{});
  else if (ppr < 22)  // rows of 16 .. 21 pieces: up to five rows
    pick(IntC<5>{}, IntC<16>{});
  else if (ppr < 32)  // rows of 22 .. 31 pieces: up to four rows
    pick(IntC<4>{}, IntC<16>{});
  else if (ppr < 64)  // rows of 32 .. 63 pieces: a step meets up to three rows
    pick(IntC<3>{}, IntC<16>{});
  else
    pick(IntC<2>{}, IntC<16>{});
  return hipGetLastError();
}

template <int M, bool W8>
hipError_t gemv_m(const uint16_t* x, int64_t k, const uint8_t* codes, const uint16_t* scales16,
                  const uint16_t* zeros16, const float* scales32, int64_t n, void* y, int out_mode,
                  const NormSrc* nrm, hipStream_t stream) {
  if (nrm && (W8 || M > 2)) return hipErrorNotSupported;
  const NormSrc nr = nrm ? *nrm : NormSrc{nullptr, nullptr, 0.f, 1};
  // the activations of a K slice sit in LDS (M * 2 bytes per k); slices are
  // whole 128-element groups
  const int64_t grain = 128;
  const int64_t kmax = (int64_t)(kLdsBudget / ((size_t)M * 2)) / grain * grain;
  const int splits = (int)((k + kmax - 1) / kmax);
  int64_t kslice = (k + splits - 1) / splits;
  kslice = (kslice + grain - 1) / grain * grain;
  // wavefronts per workgroup: one per step of a task, at most four
  const int64_t chunk_k = W8 ? 32 : 64;
  const int64_t kfirst = kslice < k ? kslice : k;
  const int64_t nit = ((kfirst + chunk_k - 1) / chunk_k + kWave - 1) / kWave;
  // the last slice may be shorter: nw must not exceed its step count either
  const int64_t klast = k - (int64_t)(splits - 1) * kslice;
  const int64_t nit_last = ((klast + chunk_k - 1) / chunk_k + kWave - 1) / kWave;
  const int64_t steps = nit < nit_last ? nit : nit_last;
  // rows per task: the most that still give each resident wavefront at least
  // two tasks (four rows: eight), one row otherwise
  const int64_t waves = (int64_t)cu_count() * kWavesPerCu;
  constexpr int RMAX = max_rows_for(M);
  int rows = 1;
  if (RMAX >= 4 && (n + 3) / 4 >= 8 * waves)
    rows = 4;
  else if (RMAX >= 2 && (n + 1) / 2 >= 2 * waves)
    rows = 2;
  // one wavefront per task when tasks outnumber the resident wavefronts;
  // otherwise a team of wavefronts splits each task's steps: four from four
  // steps, two from two (measured: at five steps, four-wavefront teams beat
  // teams of five, which leave a CU one wavefront short and pad more tasks)
  const int64_t ntask = (n + rows - 1) / rows;
  const int nw = ntask >= waves ? 1 : (steps >= 4 ? 4 : (steps >= 2 ? 2 : 1));
  if constexpr (!W8 && M <= 2) {
    // the row-block kernel, where it applies, when a task would be one row (no
    // activation reuse across rows to lose) or when the last step of a row
    // leaves more than a quarter of the lanes idle (measured crossover)
    const int64_t row_chunks = k / 64;
    const bool idle_lanes = 4 * row_chunks < 3 * 64 * ((row_chunks + 63) / 64);
    if ((rows == 1 || idle_lanes) && out_mode != kOutSilu) {
      const hipError_t e =
          nrm ? gemv_rows_m<M, false, true>(x, k, codes, scales16, zeros16, nullptr, n, y, out_mode, nr, stream)
              : gemv_rows_m<M, false, false>(x, k, codes, scales16, zeros16, nullptr, n, y, out_mode, nr, stream);
      if (e != hipErrorNotSupported) return e;
    }
  }
  if constexpr (W8 && M <= 4) {
    const hipError_t e =
        gemv_rows_m<M, true, false>(x, k, codes, nullptr, nullptr, scales32, n, y, out_mode, nr, stream);
    if (e != hipErrorNotSupported) return e;
  }
  // normalised rows and accumulated outputs: one K slice, one wavefront per task
  if ((nrm || out_mode == kOutAcc) && (splits != 1 || (nrm && nw != 1))) return hipErrorNotSupported;
  if (out_mode == kOutSilu) {  // tasks of the gate and up rows t, t + n / 2: two rows, one wavefront, one slice
    if constexpr (!W8 && M <= 2) {
      // only where the plain projection runs this kernel too (the same sums,
      // so the same bits as the projection followed by the SiLU kernel)
      const int64_t row_chunks = k / 64;
      const bool idle_lanes = 4 * row_chunks < 3 * 64 * ((row_chunks + 63) / 64);
      if (rows != 2 || nw != 1 || splits != 1 || idle_lanes) return hipErrorNotSupported;
      if constexpr (M == 1) {
        if (nit == 1)
          return nrm ? gemv_launch<M, false, 2, false, true, true, true>(x, k, kslice, splits, codes, scales16,
                                                                          zeros16, nullptr, n, y, out_mode, nullptr,
                                                                          nw, nr, stream)
                     : gemv_launch<M, false, 2, false, true, false, true>(x, k, kslice, splits, codes, scales16,
                                                                           zeros16, nullptr, n, y, out_mode, nullptr,
                                                                           nw, nr, stream);
      }
      return nrm ? gemv_launch<M, false, 2, false, false, true, true>(x, k, kslice, splits, codes, scales16, zeros16,
                                                                       nullptr, n, y, out_mode, nullptr, nw, nr,
                                                                       stream)
                 : gemv_launch<M, false, 2, false, false, false, true>(x, k, kslice, splits, codes, scales16, zeros16,
                                                                        nullptr, n, y, out_mode, nullptr, nw, nr,
                                                                        stream);
    }
    return hipErrorNotSupported;
  }
  // split-K partial sums: only the tasks-of-rows kernel needs them
  float* partial = nullptr;
  if (splits > 1) {
    void* ws = nullptr;
    const hipError_t e = workspace((size_t)splits * M * n * sizeof(float), stream, &ws);
    if (e != hipSuccess) return e;
    partial = static_cast<float*>(ws);
  }
  hipError_t err = hipErrorInvalidValue;
  auto go = [&](auto r_tag, auto multi_tag) {
    constexpr int RR = decltype(r_tag)::value;
    constexpr bool MM = decltype(multi_tag)::value != 0;
    // activations in registers where a task is one step (one row of 32
    // activation VGPRs beside the fragments: at most 128 VGPRs with four rows)
    constexpr bool XRok = !W8 && !MM && M == 1;
    constexpr bool NRok = !W8 && !MM && M <= 2;
    if (NRok && nrm) {
      if (XRok && nit == 1)
        err = gemv_launch<M, W8, RR, MM, XRok, NRok>(x, k, kslice, splits, codes, scales16, zeros16, scales32, n, y,
                                                     out_mode, partial, nw, nr, stream);
      else
        err = gemv_launch<M, W8, RR, MM, false, NRok>(x, k, kslice, splits, codes, scales16, zeros16, scales32, n, y,
                                                      out_mode, partial, nw, nr, stream);
    } else if (XRok && splits == 1 && nit == 1) {
      err = gemv_launch<M, W8, RR, MM, XRok, false>(x, k, kslice, splits, codes, scales16, zeros16, scales32, n, y,
                                                    out_mode, partial, nw, nr, stream);
    } else {
      err = gemv_launch<M, W8, RR, MM, false, false>(x, k, kslice, splits, codes, scales16, zeros16, scales32, n, y,
                                                     out_mode, partial, nw, nr, stream);
    }
  };
  auto with_nw = [&](auto r_tag) {
    if (nw > 1)
      go(r_tag, IntC<1>{});
    else
      go(r_tag, IntC<0>{});
  };
  if constexpr (RMAX >= 4) {
    if (rows == 4) with_nw(IntC<4>{});
  }
  if constexpr (RMAX >= 2) {
    if (rows == 2) with_nw(IntC<2>{});
  }
  if (rows == 1) with_nw(IntC<1>{});
  if (err != hipSuccess || splits == 1) return err;
  return launch_splitk_reduce(partial, splits, (int64_t)M * n, y, out_mode == kOutF16, stream);
}

template <bool W8>
hipError_t gemv_dispatch(const uint16_t* x, int m, int64_t k, const uint8_t* codes, const uint16_t* scales16,
                         const uint16_t* zeros16, const float* scales32, int64_t n, void* y, int out_mode,
                         const NormSrc* nrm, hipStream_t stream) {
  switch (m) {
    case 1: return gemv_m<1, W8>(x, k, codes, scales16, zeros16, scales32, n, y, out_mode, nrm, stream);
    case 2: return gemv_m<2, W8>(x, k, codes, scales16, zeros16, scales32, n, y, out_mode, nrm, stream);
    case 3: return gemv_m<3, W8>(x, k, codes, scales16, zeros16, scales32, n, y, out_mode, nrm, stream);
    case 4: return gemv_m<4, W8>(x, k, codes, scales16, zeros16, scales32, n, y, out_mode, nrm, stream);
    case 5: return gemv_m<5, W8>(x, k, codes, scales16, zeros16, scales32, n, y, out_mode, nrm, stream);
    case 6: return gemv_m<6, W8>(x, k, codes, scales16, zeros16, scales32, n, y, out_mode, nrm, stream);
    case 7: return gemv_m<7, W8>(x, k, codes, scales16, zeros16, scales32, n, y, out_mode, nrm, stream);
    case 8: return gemv_m<8, W8>(x, k, codes, scales16, zeros16, scales32, n, y, out_mode, nrm, stream);
    default: return hipErrorInvalidValue;
  }
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
                          const uint16_t* zeros, int64_t n, void* y, bool f16_out, hipStream_t stream,
                          const NormSrc* nrm, bool accum, bool silu) {
  const int mode = silu ? kOutSilu : (accum ? kOutAcc : (f16_out ? kOutF16 : kOutF32));
  return gemv_dispatch<false>(x, m, k, codes, scales, zeros, nullptr, n, y, mode, nrm, stream);
}

hipError_t launch_gemv_w8(const uint16_t* x, int m, int64_t k, const uint8_t* codes, const float* scales, int64_t n,
                          void* y, bool f16_out, hipStream_t stream) {
  return gemv_dispatch<true>(x, m, k, codes, nullptr, nullptr, scales, n, y, f16_out ? kOutF16 : kOutF32, nullptr,
                             stream);
}

}  // namespace sq

// LM-head softmax and speculative acceptance or correction (SpecQuant
// SS III-D.4 and the guess-set rule of SS III-A), stochastic (T > 0) and
// greedy (T = 0).
//
// Every vocabulary row is cut into chunks of kChunk logits so that a round's
// b * (2kd + 1) rows spread over the whole chip:
//   1. stats:    per (row, chunk) the max of z = l / T and sum exp(z - max),
//                fp64 (online-softmax partials, merged later in chunk order);
//   2. decide:   per (sequence, chunk) merge the row partials, take the kd
//                accept decisions u * q(x) < p(x) (one thread each), find the
//                first rejection n, and sum the chunk's share of the draw
//                weights R = rint(r * 2^60) in int64 (exact, so the total
//                does not depend on the summation order);
//   3. draw:     per sequence, locate the chunk holding t = floor(u Z / 2^24)
//                with a block scan of the chunk totals, then block-scan that
//                chunk.
// Probabilities are computed in fp64 and held in fp32 (prob32), the values
// q_out / p_out hand back; the decisions and the draw weights are formed in
// fp64 from those fp32 values, so that they can be reproduced exactly from
// q_out / p_out.  A -inf logit is a masked token (probability 0).  A row
// holding a NaN or +inf logit, or no finite logit, has no distribution: its
// sequence gets n_accepted = next_token = -1 (and NaN rows in q_out / p_out).
// Greedy uses per-chunk (max, first index) pairs and one decision pass.
#include <math.h>

#include <mutex>

#include "sq_device.hpp"
#include "sq_internal.hpp"

#pragma clang fp contract(off)

namespace sq {
namespace {

constexpr int kThreads = 256;
constexpr int kChunk = kAcceptChunk;  // 1024: a 152k-token row spreads over 149 workgroups
constexpr int kPer = kChunk / kThreads;  // logits per thread and chunk

struct SeqInfo {
  int n;
  int pad;
  double lp, sp, lq, sq;  // merged (max, sum) of the draw rows p_n and q_n
};

struct ArgMax {
  float v;
  int i;
};

__device__ __forceinline__ double zval(float l, float t) { return t == 1.0f ? (double)l : (double)l / (double)t; }

__device__ __forceinline__ int64_t grid_weight(double r) { return llrint(ldexp(r, 60)); }

// A probability exp(z - L) / S in fp64, held in fp32: the one expression
// behind q_out / p_out, the decisions and the draw weights.
__device__ __forceinline__ float prob32(float l, float t, double L, double S) {
  return (float)(exp(zval(l, t) - L) / S);
}

// Deterministic block reductions over 256 threads (4 wavefronts).
__device__ double block_max(double v, double* sh) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmax(v, __shfl_xor(v, off, 64));
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  __syncthreads();
  v = fmax(fmax(sh[0], sh[1]), fmax(sh[2], sh[3]));
  __syncthreads();
  return v;
}

__device__ double block_sum(double v, double* sh) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  __syncthreads();
  v = (sh[0] + sh[1]) + (sh[2] + sh[3]);
  __syncthreads();
  return v;
}

__device__ int64_t block_sum_i64(int64_t v, int64_t* sh) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  __syncthreads();
  v = (sh[0] + sh[1]) + (sh[2] + sh[3]);
  __syncthreads();
  return v;
}

// Row r of the combined row space: target rows first ([b][kd+1] order), then
// draft rows ([kd][b] order); both arrays are contiguous in that order.
__device__ __forceinline__ const float* row_ptr(const float* draft, const float* target, int64_t rows_t, int64_t r,
                                                int v) {
  return r < rows_t ? target + r * v : draft + (r - rows_t) * v;
}

// Exclusive prefix sum of v over the 256 threads in thread order; `total`
// receives the block's sum.  Integer, so exact.
__device__ int64_t block_exclusive_scan_i64(int64_t v, int64_t* sh, int64_t& total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int64_t x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int64_t y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  if (lane == 63) sh[w] = x;
  __syncthreads();
  int64_t base = 0;
  for (int i = 0; i < w; ++i) base += sh[i];
  total = (sh[0] + sh[1]) + (sh[2] + sh[3]);
  __syncthreads();
  return base + x - v;
}

// One wavefront merges a row's chunk partials: L = max over chunks, S = the
// sum of S_c exp(L_c - L), each lane taking every 64th chunk in increasing
// order and the lanes combined in a fixed shuffle tree.  A fully masked chunk
// (S_c = 0) adds nothing; a chunk marked invalid (S_c NaN), or a row without
// any mass, gives L = S = NaN.  Every lane returns the values.
//
// The first kCells chunks of each lane are loaded ahead (load_cells: lane l
// chunks l, l + 64, ..., a chunk past the row's end replaced by the row's
// last one and ignored), so that a kernel can issue them beside its other
// independent loads.  Rows of more than 64 kCells chunks take the rest from
// memory (kWide); without kWide the code holds no loop over memory, so that
// the compiler's load counters wait for exactly the loads a value needs.
constexpr int kCells = 4;

__device__ __forceinline__ void load_cells(const double2* st, int nchunk, double2 (&e)[kCells]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int i = 0; i < kCells; ++i) e[i] = st[min(lane + 64 * i, nchunk - 1)];
}

template <bool kWide>
__device__ void merge_cells(const double2* st, int nchunk, const double2 (&e)[kCells], double& L, double& S) {
  const int lane = threadIdx.x & 63;
  double mx = -INFINITY;
  int bad = 0;
#pragma unroll
  for (int i = 0; i < kCells; ++i) {
    const bool in = lane + 64 * i < nchunk;
    bad |= in && isnan(e[i].y) ? 1 : 0;
    if (in && e[i].y > 0.0) mx = fmax(mx, e[i].x);
  }
  if constexpr (kWide) {
    for (int c = lane + 64 * kCells; c < nchunk; c += 64) {
      const double2 f = st[c];
      bad |= isnan(f.y) ? 1 : 0;
      if (f.y > 0.0) mx = fmax(mx, f.x);
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    mx = fmax(mx, __shfl_xor(mx, off, 64));
    bad |= __shfl_xor(bad, off, 64);
  }
  double s = 0.0;
#pragma unroll
  for (int i = 0; i < kCells; ++i)
    if (lane + 64 * i < nchunk && e[i].y > 0.0) s += e[i].y * exp(e[i].x - mx);
  if constexpr (kWide) {
    for (int c = lane + 64 * kCells; c < nchunk; c += 64) {
      const double2 f = st[c];
      if (f.y > 0.0) s += f.y * exp(f.x - mx);
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off, 64);
  if (bad || !(s > 0.0)) {
    mx = NAN;
    s = NAN;
  }
  L = mx;
  S = s;
}

__device__ void wave_merge(const double2* st, int nchunk, double& L, double& S) {
  double2 e[kCells];
  load_cells(st, nchunk, e);
  merge_cells<true>(st, nchunk, e, L, S);
}

// 1. per (row, chunk): (max z, sum exp(z - max z)).  blockIdx.x = row * nchunk + chunk.
__global__ __launch_bounds__(kThreads) void stats_kernel(const float* __restrict__ draft,
                                                         const float* __restrict__ target, int64_t rows_t, int v,
                                                         float temp, int nchunk, double2* __restrict__ stats) {
  __shared__ double sh[4];
  const int64_t row = blockIdx.x / nchunk;
  const int c = blockIdx.x % nchunk;
  const float* l = row_ptr(draft, target, rows_t, row, v);
  const int beg = c * kChunk;
  double z[kPer];
  double mx = -INFINITY;
  int bad = 0;
#pragma unroll
  for (int e = 0; e < kPer; ++e) {
    const int j = beg + e * kThreads + threadIdx.x;
    const float lj = j < v ? l[j] : -INFINITY;
    bad |= (isnan(lj) || lj == INFINITY) ? 1 : 0;
    z[e] = zval(lj, temp);
    if (!isnan(z[e])) mx = fmax(mx, z[e]);
  }
  bad = __syncthreads_or(bad);
  mx = block_max(mx, sh);
  double s = 0.0;
  if (mx > -INFINITY && !bad) {  // uniform across the block
#pragma unroll
    for (int e = 0; e < kPer; ++e) s += exp(z[e] - mx);  // masked and padded cells add exp(-inf) = 0
  }
  s = block_sum(s, sh);
  // (max, sum); a fully masked chunk is (-inf, 0); an invalid one (NaN, NaN)
  if (threadIdx.x == 0) stats[row * nchunk + c] = bad ? make_double2(NAN, NAN) : make_double2(mx, s);
}

// Optional copies of the distributions: p or q = exp(z - L) / S as fp32.
__global__ __launch_bounds__(kThreads) void probs_kernel(const float* __restrict__ draft,
                                                         const float* __restrict__ target, int64_t rows_t, int v,
                                                         float temp, int nchunk, const double2* __restrict__ stats,
                                                         float* __restrict__ q_out, float* __restrict__ p_out) {
  __shared__ double sL, sS;
  const int64_t row = blockIdx.x / nchunk;
  const int c = blockIdx.x % nchunk;
  float* out = row < rows_t ? (p_out ? p_out + row * v : nullptr) : (q_out ? q_out + (row - rows_t) * v : nullptr);
  if (!out) return;  // uniform across the block
  if (threadIdx.x < 64) {
    double L, S;
    wave_merge(stats + row * nchunk, nchunk, L, S);
    if (threadIdx.x == 0) {
      sL = L;
      sS = S;
    }
  }
  __syncthreads();
  const double L = sL, S = sS;  // NaN for a row without a distribution: NaN out
  const float* l = row_ptr(draft, target, rows_t, row, v);
  for (int e = 0; e < kPer; ++e) {
    const int j = c * kChunk + e * kThreads + threadIdx.x;
    if (j < v) out[j] = prob32(l[j], temp, L, S);
  }
}

// 2. per (sequence, chunk): decisions, first rejection, chunk share of the draw weights.
// zs[(s * nchunk + c) * 2 + 0] = sum of R over the chunk for the draw row
// (residual max(0, p_n - q_n) when n < kd, else p_kd); [.. + 1] = sum of R for
// p_n (the fallback when the residual mass is zero).  A sequence with a row
// without a distribution gets n = -1 and zero weights.
// blockIdx.x = s * nchunk + c.
// Loads that wait for nothing computed here go out together, so that their
// round trips overlap: the draft tokens and their uniforms, the first rows of
// chunk partials, the logits at the tokens, and this chunk of p_0 and q_0
// (the draw rows when the first draft token is rejected, or when kd = 0).
// Every one of them is unconditional (indices clamped, the value ignored
// where it does not apply).
template <bool kWide>
__global__ __launch_bounds__(kThreads) void decide_kernel(const float* __restrict__ draft,
                                                          const float* __restrict__ target,
                                                          const int32_t* __restrict__ tokens,
                                                          const uint32_t* __restrict__ u24, int b, int kd, int v,
                                                          float temp, int nchunk, const double2* __restrict__ stats,
                                                          int64_t* __restrict__ zs, SeqInfo* __restrict__ info) {
  constexpr int kBatch = 3;  // rows of partials a wavefront holds at once
  __shared__ double sL[129], sS[129];
  __shared__ int sAcc[64];
  __shared__ int sN;
  __shared__ int64_t shi[4];
  const int s = blockIdx.x / nchunk;
  const int c = blockIdx.x % nchunk;
  const int w = threadIdx.x >> 6;
  const int nrows = 2 * kd + 1;
  const int64_t rows_t = (int64_t)b * (kd + 1);
  const float* trow = target + (int64_t)s * (kd + 1) * v;  // p_0 of the sequence
  // row rr of the sequence: target rows 0..kd, then draft rows 0..kd-1
  auto row_of = [&](int rr) -> int64_t {
    return rr <= kd ? (int64_t)s * (kd + 1) + rr : rows_t + (int64_t)(rr - kd - 1) * b + s;
  };
  // thread i < kd: draft position i; the other threads read position 0 (or,
  // with kd = 0, the sequence's uniform) and ignore it
  const bool dlane = (int)threadIdx.x < kd;
  const int di = dlane ? (int)threadIdx.x : 0;
  const int32_t* tp = kd > 0 ? tokens + (int64_t)di * b + s : (const int32_t*)(u24 + (int64_t)s * (kd + 1));
  const int32_t xraw = *tp;
  const uint32_t ut = u24[(int64_t)s * (kd + 1) + di];
  // the 2kd + 1 rows' statistics, one wavefront per row, kBatch rows in flight
  double2 e[kBatch][kCells];
  auto load_batch = [&](int r0) {
#pragma unroll
    for (int j = 0; j < kBatch; ++j)
      load_cells(stats + row_of(min(r0 + 4 * j, nrows - 1)) * nchunk, nchunk, e[j]);
  };
  load_batch(w);
  // this chunk of p_0 and q_0 (of p_0 twice when kd = 0), thread t holding
  // logits t, t + 256, ...
  float pv[kPer], qv[kPer];
  const float* q0 = kd > 0 ? draft + (int64_t)s * v : trow;
  auto load_chunk = [&](const float* row, float (&dst)[kPer]) {
#pragma unroll
    for (int k = 0; k < kPer; ++k) dst[k] = row[min(c * kChunk + k * kThreads + (int)threadIdx.x, v - 1)];
  };
  load_chunk(trow, pv);
  load_chunk(q0, qv);
  const bool tok_ok = dlane && xraw >= 0 && xraw < v;
  const int xi = tok_ok ? xraw : 0;
  const float lpt = trow[(int64_t)di * v + xi];
  const float lqt = kd > 0 ? draft[((int64_t)di * b + s) * v + xi] : trow[xi];
  auto merge_batch = [&](int r0) {
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int rr = r0 + 4 * j;
      if (rr < nrows) {
        double L, S;
        merge_cells<kWide>(stats + row_of(rr) * nchunk, nchunk, e[j], L, S);
        if ((threadIdx.x & 63) == 0) {
          sL[rr] = L;
          sS[rr] = S;
        }
      }
    }
  };
  merge_batch(w);
  for (int r0 = w + 4 * kBatch; r0 < nrows; r0 += 4 * kBatch) {  // kd >= 6
    load_batch(r0);
    merge_batch(r0);
  }
  __syncthreads();
  int invalid = 0;
  for (int rr = threadIdx.x; rr < nrows; rr += kThreads) invalid |= isnan(sS[rr]) ? 1 : 0;
  invalid = __syncthreads_or(invalid);
  if (dlane && !invalid) {
    const int i = threadIdx.x;
    int acc = 0;
    if (tok_ok) {
      // fp32 probabilities; u (24 bits) times q (24 bits) is exact in fp64
      const float p = prob32(lpt, temp, sL[i], sS[i]);
      const float q = prob32(lqt, temp, sL[kd + 1 + i], sS[kd + 1 + i]);
      const double u = ldexp((double)(ut & 0xFFFFFFu), -24);
      acc = (u * (double)q < (double)p) ? 1 : 0;
    }
    sAcc[i] = acc;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int n = kd;
    for (int i = 0; i < kd; ++i)
      if (!sAcc[i]) {
        n = i;
        break;
      }
    sN = invalid ? -1 : n;
  }
  __syncthreads();
  const int n = sN;
  if (n < 0) {  // uniform across the block
    if (threadIdx.x == 0) {
      zs[((int64_t)s * nchunk + c) * 2 + 0] = 0;
      zs[((int64_t)s * nchunk + c) * 2 + 1] = 0;
      if (c == 0) {
        SeqInfo si;
        si.n = -1;
        si.pad = 0;
        si.lp = si.sp = si.lq = si.sq = 0.0;
        info[s] = si;
      }
    }
    return;
  }
  const double Lp = sL[n], Sp = sS[n];
  const bool resid = n < kd;
  const double Lq = resid ? sL[kd + 1 + n] : 0.0, Sq = resid ? sS[kd + 1 + n] : 1.0;
  if (n > 0) {  // uniform across the block; n = 0 uses the rows loaded ahead
    load_chunk(trow + (int64_t)n * v, pv);
    if (resid) load_chunk(draft + ((int64_t)n * b + s) * v, qv);
  }
  int64_t z0 = 0, z1 = 0;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int j = c * kChunk + k * kThreads + threadIdx.x;
    if (j >= v) break;
    const float p = prob32(pv[k], temp, Lp, Sp);
    if (resid) {
      const float q = prob32(qv[k], temp, Lq, Sq);
      const double r = (double)p - (double)q;
      z0 += grid_weight(r > 0.0 ? r : 0.0);
      z1 += grid_weight((double)p);
    } else {
      z0 += grid_weight((double)p);
    }
  }
  z0 = block_sum_i64(z0, shi);
  z1 = block_sum_i64(z1, shi);
  if (threadIdx.x == 0) {
    zs[((int64_t)s * nchunk + c) * 2 + 0] = z0;
    zs[((int64_t)s * nchunk + c) * 2 + 1] = z1;
    if (c == 0) {
      SeqInfo si;
      si.n = n;
      si.pad = 0;
      si.lp = Lp;
      si.sp = Sp;
      si.lq = Lq;
      si.sq = Sq;
      info[s] = si;
    }
  }
}

// 3. per sequence: the draw.  The chunk holding t is found with a block scan
// over the chunk totals (256 chunks at a time), then the chunk is scanned
// with kPer consecutive logits per thread, so that the block's exclusive scan
// of the thread sums orders them.  All sums are int64, so exact.  The
// sequence's record, its uniform and the first 256 chunk totals are loaded
// together at the start (none waits for another).
__global__ __launch_bounds__(kThreads) void draw_kernel(const float* __restrict__ draft,
                                                        const float* __restrict__ target,
                                                        const uint32_t* __restrict__ u24, int b, int kd, int v,
                                                        float temp, int nchunk, const int64_t* __restrict__ zs,
                                                        const SeqInfo* __restrict__ info,
                                                        int32_t* __restrict__ n_accepted,
                                                        int32_t* __restrict__ next_token) {
  __shared__ int64_t sOff;
  __shared__ int sChunk;
  __shared__ int64_t shi[4];
  const int s = blockIdx.x;
  const int64_t* z = zs + (int64_t)s * nchunk * 2;
  const SeqInfo si = info[s];
  const uint32_t us = u24[(int64_t)s * (kd + 1) + kd];
  // thread t holds chunk t's totals (a thread past the last chunk reads the
  // last one and takes 0)
  const int tc = min((int)threadIdx.x, nchunk - 1);
  const int64_t ra = z[2 * tc], rb = z[2 * tc + 1];
  const bool first = (int)threadIdx.x < nchunk;
  const int64_t za = first ? ra : 0, zb = first ? rb : 0;

  // the total mass Z of the draw row (the residual's, else p_n's when that is zero on the grid)
  int64_t part = za;
  for (int c = threadIdx.x + kThreads; c < nchunk; c += kThreads) part += z[2 * c];
  int64_t Z = block_sum_i64(part, shi);
  const int n = si.n;
  if (n < 0) {  // a row without a distribution (uniform across the block)
    if (threadIdx.x == 0) {
      n_accepted[s] = -1;
      next_token[s] = -1;
    }
    return;
  }
  int which = 0;
  if (Z == 0 && n < kd) {  // uniform across the block
    which = 1;
    part = zb;
    for (int c = threadIdx.x + kThreads; c < nchunk; c += kThreads) part += z[2 * c + 1];
    Z = block_sum_i64(part, shi);
  }
  if (Z == 0) {  // no mass on the fixed-point grid
    if (threadIdx.x == 0) {
      n_accepted[s] = n;
      next_token[s] = -1;
    }
    return;
  }
  const uint64_t uu = us & 0xFFFFFFu;
  const uint64_t lo = uu * (uint64_t)Z;
  const uint64_t hi = __umul64hi(uu, (uint64_t)Z);
  const int64_t t = (int64_t)((hi << 40) | (lo >> 24));  // floor(u * Z / 2^24) < Z

  // the chunk c with run(c) <= t < run(c) + z_c, 256 chunks at a time
  if (threadIdx.x == 0) sChunk = -1;
  int64_t run = 0;
  for (int c0 = 0; c0 < nchunk; c0 += kThreads) {
    const int c = c0 + (int)threadIdx.x;
    const int64_t zc = c0 == 0 ? (which ? zb : za) : c < nchunk ? z[2 * c + which] : 0;
    int64_t tile;
    const int64_t pre = run + block_exclusive_scan_i64(zc, shi, tile);
    if (zc > 0 && pre <= t && t < pre + zc) {
      sChunk = c;
      sOff = t - pre;
    }
    __syncthreads();
    if (sChunk >= 0) break;  // uniform across the block
    run += tile;
  }
  const int chunk = sChunk;
  if (chunk < 0) {  // cannot happen (t < Z); kept so that no index can leave the row
    if (threadIdx.x == 0) {
      n_accepted[s] = n;
      next_token[s] = -1;
    }
    return;
  }
  const int64_t off = sOff;
  const bool resid = n < kd && which == 0;
  const float* lp = target + ((int64_t)s * (kd + 1) + n) * v;
  const float* lq = resid ? draft + ((int64_t)n * b + s) * v : nullptr;
  int64_t R[kPer];
  int64_t local = 0;
  const int beg = chunk * kChunk + threadIdx.x * kPer;
  float pv[kPer], qv[kPer];  // every load of the chunk in flight at once
#pragma unroll
  for (int e = 0; e < kPer; ++e) {
    const int j = beg + e;
    pv[e] = j < v ? lp[j] : 0.0f;
    qv[e] = resid && j < v ? lq[j] : 0.0f;
  }
#pragma unroll
  for (int e = 0; e < kPer; ++e) {
    const int j = beg + e;
    int64_t w = 0;
    if (j < v) {
      const float p = prob32(pv[e], temp, si.lp, si.sp);
      if (resid) {
        const float q = prob32(qv[e], temp, si.lq, si.sq);
        const double r = (double)p - (double)q;
        w = grid_weight(r > 0.0 ? r : 0.0);
      } else {
        w = grid_weight((double)p);
      }
    }
    R[e] = w;
    local += w;
  }
  int64_t tot;
  const int64_t pre = block_exclusive_scan_i64(local, shi, tot);
  if (local > 0 && pre <= off && off < pre + local) {
    int64_t acc = pre;
    int tok = beg;
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
      acc += R[e];
      if (acc > off) {
        tok = beg + e;
        break;
      }
    }
    next_token[s] = tok;
    n_accepted[s] = n;
  }
}

// Greedy: per (target row, chunk) the max finite logit and its smallest
// index (index kNone when the chunk has no finite logit, kBad when it holds a
// NaN or +inf).
constexpr int kNone = 0x7FFFFFFF;
constexpr int kBad = -1;

__global__ __launch_bounds__(kThreads) void argmax_kernel(const float* __restrict__ target, int v, int nchunk,
                                                          ArgMax* __restrict__ out) {
  __shared__ float sv[4];
  __shared__ int si[4];
  const int64_t row = blockIdx.x / nchunk;
  const int c = blockIdx.x % nchunk;
  const float* l = target + row * v;
  float best = -INFINITY;
  int bi = kNone;
  int bad = 0;
  for (int e = 0; e < kPer; ++e) {
    const int j = c * kChunk + e * kThreads + threadIdx.x;
    if (j < v) {
      const float x = l[j];
      bad |= (isnan(x) || x == INFINITY) ? 1 : 0;
      if (isfinite(x) && (bi == kNone || x > best || (x == best && j < bi))) {
        best = x;
        bi = j;
      }
    }
  }
  bad = __syncthreads_or(bad);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(best, off, 64);
    const int oi = __shfl_xor(bi, off, 64);
    if (oi != kNone && (bi == kNone || ov > best || (ov == best && oi < bi))) {
      best = ov;
      bi = oi;
    }
  }
  if ((threadIdx.x & 63) == 0) {
    sv[threadIdx.x >> 6] = best;
    si[threadIdx.x >> 6] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w)
      if (si[w] != kNone && (bi == kNone || sv[w] > best || (sv[w] == best && si[w] < bi))) {
        best = sv[w];
        bi = si[w];
      }
    ArgMax a;
    a.v = best;
    a.i = bad ? kBad : bi;
    out[row * nchunk + c] = a;
  }
}

__global__ __launch_bounds__(kThreads) void greedy_kernel(const int32_t* __restrict__ tokens, int b, int kd, int v,
                                                          int nchunk, const ArgMax* __restrict__ am,
                                                          int32_t* __restrict__ n_accepted,
                                                          int32_t* __restrict__ next_token) {
  __shared__ int sArg[65];
  const int s = blockIdx.x;
  for (int i = threadIdx.x; i <= kd; i += kThreads) {
    const ArgMax* a = am + ((int64_t)s * (kd + 1) + i) * nchunk;
    float best = -INFINITY;
    int bi = kNone;
    bool bad = false;
    for (int c = 0; c < nchunk; ++c) {
      const ArgMax e = a[c];
      bad |= e.i == kBad;
      if (e.i != kBad && e.i != kNone && (bi == kNone || e.v > best)) {  // chunks ascend: ties keep the earlier
        best = e.v;
        bi = e.i;
      }
    }
    sArg[i] = (bad || bi == kNone) ? -1 : bi;  // -1: the row has no greedy target
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    bool invalid = false;
    for (int i = 0; i <= kd; ++i) invalid |= sArg[i] < 0;
    if (invalid) {
      n_accepted[s] = -1;
      next_token[s] = -1;
      return;
    }
    int n = kd;
    for (int i = 0; i < kd; ++i) {
      const int32_t xt = tokens[(int64_t)i * b + s];
      if (xt < 0 || xt >= v || xt != sArg[i]) {
        n = i;
        break;
      }
    }
    n_accepted[s] = n;
    next_token[s] = sArg[n];
  }
}

// ----------------------------------------------------- several draft chains
// Multi-candidate acceptance: each sequence has c draft chains of kd tokens;
// target rows [b][c][kd+1], draft rows [kd][b][c], tokens [kd][b][c],
// uniforms [b][c kd + 1] (u[d c + j] tests chain j at depth d, u[c kd] drives
// the final draw).  The fp32 distributions are materialised first (probs
// kernel); then one workgroup of kMThreads per sequence walks the chains'
// prefix tree with recursive rejection sampling on the int64 grid:
//   first candidate at a node:   u q(x) < p(x) in fp64 (exact);
//   its rejection:               R = rint(max(0, p - q) 2^60), Z = sum R;
//   later candidates:            u q(x) Z < R(x), exact in 128-bit integers;
//   their rejection:             R <- max(0, R - floor(q Z)), Z = sum R;
//   Z == 0 after an update:      R = rint(p 2^60) (the node's p);
//   all alive candidates fail:   draw from R; after kd accepted: from p_kd.
// Integer sums do not depend on their order, so the results are those of the
// same rule applied to the fp32 distributions in any order.
constexpr int kMThreads = 1024;
constexpr int kMWaves = kMThreads / 64;

__device__ __forceinline__ int64_t mblock_sum_i64(int64_t v, int64_t* sh) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  __syncthreads();  // sh may still be read by an earlier call
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  __syncthreads();
  int64_t t = 0;
  for (int w = 0; w < kMWaves; ++w) t += sh[w];
  return t;
}

// q = m 2^e exactly (m < 2^24), from the bits of a finite q >= 0.
__device__ __forceinline__ void split_f32(float q, uint64_t& m, int& e) {
  const uint32_t bits = __float_as_uint(q);
  const uint32_t ex = (bits >> 23) & 0xFFu, man = bits & 0x7FFFFFu;
  if (ex == 0) {
    m = man;
    e = -149;
  } else {
    m = man | 0x800000u;
    e = (int)ex - 150;
  }
}

// floor(q Z), q in [0, 1], 0 <= Z < 2^62, exactly.
__device__ __forceinline__ int64_t floor_qz(float q, int64_t z) {
  uint64_t m;
  int e;
  split_f32(q, m, e);
  if (m == 0 || z == 0) return 0;
  const uint64_t lo = m * (uint64_t)z, hi = __umul64hi(m, (uint64_t)z);
  const int sh = -e;  // >= 23 for q <= 1
  if (sh >= 128) return 0;
  if (sh >= 64) return (int64_t)(hi >> (sh - 64));
  return (int64_t)((hi << (64 - sh)) | (lo >> sh));
}

// u24 / 2^24 q Z < R, exactly.
__device__ __forceinline__ bool test_grid(uint32_t u24, float q, int64_t z, int64_t r) {
  if (r <= 0) return false;
  uint64_t m;
  int e;
  split_f32(q, m, e);
  const uint64_t a = (uint64_t)(u24 & 0xFFFFFFu) * m;  // < 2^48
  const uint64_t llo = a * (uint64_t)z, lhi = __umul64hi(a, (uint64_t)z);
  const int sh = 24 - e;  // >= 47 for q <= 1
  const int bits = 64 - __clzll((unsigned long long)r);
  if (bits + sh >= 127) return true;  // r 2^sh >= 2^126 > lhs
  uint64_t rhi, rlo;
  if (sh >= 64) {
    rhi = (uint64_t)r << (sh - 64);
    rlo = 0;
  } else {
    rhi = (uint64_t)r >> (64 - sh);
    rlo = (uint64_t)r << sh;
  }
  return lhi < rhi || (lhi == rhi && llo < rlo);
}

__global__ __launch_bounds__(kMThreads) void multi_kernel(const float* __restrict__ p32, const float* __restrict__ q32,
                                                          const int32_t* __restrict__ tokens,
                                                          const uint32_t* __restrict__ u24, int b, int c, int kd,
                                                          int v, int nchunk, const double2* __restrict__ stats,
                                                          int64_t* __restrict__ grid, int32_t* __restrict__ n_accepted,
                                                          int32_t* __restrict__ next_token,
                                                          int32_t* __restrict__ chain) {
  __shared__ int64_t sh[kMWaves];
  __shared__ int sBad;
  __shared__ int64_t sR;
  __shared__ int sTok;
  const int s = blockIdx.x;
  const int t = threadIdx.x;
  const int64_t rows_t = (int64_t)b * c * (kd + 1);
  // every row of the sequence must have a distribution (its merged statistics finite)
  if (t == 0) sBad = 0;
  __syncthreads();
  for (int rr = t >> 6; rr < c * (2 * kd + 1); rr += kMWaves) {
    int64_t row;
    if (rr < c * (kd + 1)) {
      row = (int64_t)s * c * (kd + 1) + rr;
    } else {
      const int k2 = rr - c * (kd + 1);  // draft row d * c + j
      row = rows_t + ((int64_t)(k2 / c) * b + s) * c + k2 % c;
    }
    double L, S;
    wave_merge(stats + row * nchunk, nchunk, L, S);
    if ((t & 63) == 0 && isnan(S)) atomicOr(&sBad, 1);
  }
  __syncthreads();
  if (sBad) {
    if (t == 0) n_accepted[s] = next_token[s] = chain[s] = -1;
    return;
  }
  int64_t* R = grid + (int64_t)s * v;
  const uint32_t* u = u24 + (int64_t)s * (c * kd + 1);
  const uint64_t all = c == 64 ? ~0ull : ((1ull << c) - 1ull);
  uint64_t alive = all;
  int n = kd;
  int64_t z = 0;
  auto tok_of = [&](int d, int j) { return tokens[((int64_t)d * b + s) * c + j]; };
  auto grid_p = [&](const float* p) -> int64_t {  // R = rint(p 2^60), returns Z
    int64_t part = 0;
    for (int y = t; y < v; y += kMThreads) {
      const int64_t w = grid_weight((double)p[y]);
      R[y] = w;
      part += w;
    }
    return mblock_sum_i64(part, sh);
  };
  for (int d = 0; d < kd; ++d) {
    const int j0 = __ffsll((unsigned long long)alive) - 1;
    const float* p = p32 + (((int64_t)s * c + j0) * (kd + 1) + d) * v;
    const float* q = q32 + (((int64_t)d * b + s) * c + j0) * v;
    int accepted = -1;
    bool first = true;
    for (uint64_t rest = alive; rest; rest &= rest - 1) {
      const int j = __ffsll((unsigned long long)rest) - 1;
      const int32_t x = tok_of(d, j);
      const uint32_t uj = u[d * c + j];
      bool acc = false;
      if (x >= 0 && x < v) {
        if (first) {
          acc = ldexp((double)(uj & 0xFFFFFFu), -24) * (double)q[x] < (double)p[x];
        } else {
          if (t == 0) sR = R[x];
          __syncthreads();
          acc = test_grid(uj, q[x], z, sR);
          __syncthreads();
        }
      }
      if (acc) {  // uniform: every thread took the same decision
        accepted = x;
        break;
      }
      int64_t part = 0;
      if (first) {
        for (int y = t; y < v; y += kMThreads) {
          const double r = (double)p[y] - (double)q[y];
          const int64_t w = grid_weight(r > 0.0 ? r : 0.0);
          R[y] = w;
          part += w;
        }
      } else {
        const int64_t z0 = z;
        for (int y = t; y < v; y += kMThreads) {
          const int64_t w0 = R[y] - floor_qz(q[y], z0);
          const int64_t w = w0 > 0 ? w0 : 0;
          R[y] = w;
          part += w;
        }
      }
      z = mblock_sum_i64(part, sh);  // its barrier also publishes R to the workgroup
      if (z == 0) z = grid_p(p);     // no residual mass on the grid: back to p
      first = false;
    }
    if (accepted < 0) {
      n = d;
      break;
    }
    uint64_t keep = 0;
    for (uint64_t rest = alive; rest; rest &= rest - 1) {
      const int j = __ffsll((unsigned long long)rest) - 1;
      if (tok_of(d, j) == accepted) keep |= 1ull << j;
    }
    alive = keep;
  }
  const int jf = __ffsll((unsigned long long)alive) - 1;
  if (n == kd) z = grid_p(p32 + (((int64_t)s * c + jf) * (kd + 1) + kd) * v);
  // the draw: t = floor(u Z / 2^24); thread i owns a contiguous segment of the row
  if (t == 0) sTok = -1;
  __syncthreads();
  if (z > 0) {
    const uint64_t uu = u[c * kd] & 0xFFFFFFu;
    const int64_t tt = (int64_t)((__umul64hi(uu, (uint64_t)z) << 40) | ((uu * (uint64_t)z) >> 24));
    const int seg = (v + kMThreads - 1) / kMThreads;
    const int beg = t * seg, end = beg + seg < v ? beg + seg : v;
    int64_t local = 0;
    for (int y = beg; y < end; ++y) local += R[y];
    // exclusive scan of the segment totals in thread order
    const int lane = t & 63, w = t >> 6;
    int64_t x = local;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int64_t yv = __shfl_up(x, off, 64);
      if (lane >= off) x += yv;
    }
    __syncthreads();
    if (lane == 63) sh[w] = x;
    __syncthreads();
    int64_t base = 0;
    for (int i = 0; i < w; ++i) base += sh[i];
    const int64_t pre = base + x - local;
    if (local > 0 && pre <= tt && tt < pre + local) {
      int64_t acc = pre;
      for (int y = beg; y < end; ++y) {
        acc += R[y];
        if (acc > tt) {
          sTok = y;
          break;
        }
      }
    }
  }
  __syncthreads();
  if (t == 0) {
    n_accepted[s] = n;
    next_token[s] = sTok;
    chain[s] = jf;
  }
}

// Greedy (T = 0) over several chains: per sequence, the argmax of the lowest
// alive chain's row at each depth is accepted when an alive chain drafted it.
__global__ __launch_bounds__(kThreads) void multi_greedy_kernel(const int32_t* __restrict__ tokens, int b, int c,
                                                                int kd, int nchunk, const ArgMax* __restrict__ am,
                                                                int32_t* __restrict__ n_accepted,
                                                                int32_t* __restrict__ next_token,
                                                                int32_t* __restrict__ chain) {
  __shared__ int sArg[64 * 65];
  const int s = blockIdx.x;
  const int rows = c * (kd + 1);
  for (int r = threadIdx.x; r < rows; r += kThreads) {
    const ArgMax* a = am + ((int64_t)s * rows + r) * nchunk;
    float best = -INFINITY;
    int bi = kNone;
    bool bad = false;
    for (int k = 0; k < nchunk; ++k) {
      const ArgMax e = a[k];
      bad |= e.i == kBad;
      if (e.i != kBad && e.i != kNone && (bi == kNone || e.v > best)) {  // chunks ascend: ties keep the earlier
        best = e.v;
        bi = e.i;
      }
    }
    sArg[r] = (bad || bi == kNone) ? -1 : bi;
  }
  __syncthreads();
  if (threadIdx.x != 0) return;
  for (int r = 0; r < rows; ++r)
    if (sArg[r] < 0) {
      n_accepted[s] = next_token[s] = chain[s] = -1;
      return;
    }
  uint64_t alive = c == 64 ? ~0ull : ((1ull << c) - 1ull);
  int n = kd, tok = -1;
  for (int d = 0; d <= kd; ++d) {
    const int j0 = __ffsll((unsigned long long)alive) - 1;
    const int g = sArg[j0 * (kd + 1) + d];
    if (d == kd) {
      tok = g;
      break;
    }
    uint64_t keep = 0;
    for (uint64_t rest = alive; rest; rest &= rest - 1) {
      const int j = __ffsll((unsigned long long)rest) - 1;
      if (tokens[((int64_t)d * b + s) * c + j] == g) keep |= 1ull << j;
    }
    if (!keep) {
      n = d;
      tok = g;
      break;
    }
    alive = keep;
  }
  n_accepted[s] = n;
  next_token[s] = tok;
  chain[s] = __ffsll((unsigned long long)alive) - 1;
}

}  // namespace

namespace {

// Scratch of one call: the greedy pairs, or the row statistics, the chunk
// weights and the per-sequence state (each part 256-byte aligned).
struct AcceptScratch {
  size_t st_bytes, zs_bytes, in_bytes;
  size_t total() const { return st_bytes + zs_bytes + in_bytes; }
};

AcceptScratch accept_scratch(int b, int kd, int v, float temperature) {
  const int64_t nchunk = (v + kChunk - 1) / kChunk;
  const int64_t rows_t = (int64_t)b * (kd + 1);
  AcceptScratch a;
  if (temperature == 0.0f) {
    a.st_bytes = ((size_t)rows_t * nchunk * sizeof(ArgMax) + 255) / 256 * 256;
    a.zs_bytes = a.in_bytes = 0;
    return a;
  }
  const int64_t rows = rows_t + (int64_t)b * kd;
  a.st_bytes = ((size_t)rows * nchunk * sizeof(double2) + 255) / 256 * 256;
  a.zs_bytes = ((size_t)b * nchunk * 2 * sizeof(int64_t) + 255) / 256 * 256;
  a.in_bytes = (size_t)b * sizeof(SeqInfo);
  return a;
}

// The accept kernels on the scratch `ws` (at least accept_scratch().total() bytes).
hipError_t enqueue_accept(const float* draft, const float* target, const int32_t* tokens, const uint32_t* u24, int b,
                          int kd, int v, float temperature, int32_t* n_accepted, int32_t* next_token, float* q_out,
                          float* p_out, char* ws, hipStream_t stream) {
  const int nchunk = (v + kChunk - 1) / kChunk;
  const int64_t rows_t = (int64_t)b * (kd + 1);
  const AcceptScratch a = accept_scratch(b, kd, v, temperature);
  if (temperature == 0.0f) {
    ArgMax* am = reinterpret_cast<ArgMax*>(ws);
    hipLaunchKernelGGL(argmax_kernel, dim3((unsigned)(rows_t * nchunk)), dim3(kThreads), 0, stream, target, v, nchunk,
                       am);
    hipLaunchKernelGGL(greedy_kernel, dim3((unsigned)b), dim3(kThreads), 0, stream, tokens, b, kd, v, nchunk, am,
                       n_accepted, next_token);
    return hipGetLastError();
  }
  const int64_t rows = rows_t + (int64_t)b * kd;
  double2* stats = reinterpret_cast<double2*>(ws);
  int64_t* zs = reinterpret_cast<int64_t*>(ws + a.st_bytes);
  SeqInfo* info = reinterpret_cast<SeqInfo*>(ws + a.st_bytes + a.zs_bytes);
  hipLaunchKernelGGL(stats_kernel, dim3((unsigned)(rows * nchunk)), dim3(kThreads), 0, stream, draft, target, rows_t, v,
                     temperature, nchunk, stats);
  if (p_out || q_out)
    hipLaunchKernelGGL(probs_kernel, dim3((unsigned)(rows * nchunk)), dim3(kThreads), 0, stream, draft, target, rows_t,
                       v, temperature, nchunk, stats, q_out, p_out);
  if (nchunk > 64 * kCells)
    hipLaunchKernelGGL(decide_kernel<true>, dim3((unsigned)((int64_t)b * nchunk)), dim3(kThreads), 0, stream, draft,
                       target, tokens, u24, b, kd, v, temperature, nchunk, stats, zs, info);
  else
    hipLaunchKernelGGL(decide_kernel<false>, dim3((unsigned)((int64_t)b * nchunk)), dim3(kThreads), 0, stream, draft,
                       target, tokens, u24, b, kd, v, temperature, nchunk, stats, zs, info);
  hipLaunchKernelGGL(draw_kernel, dim3((unsigned)b), dim3(kThreads), 0, stream, draft, target, u24, b, kd, v,
                     temperature, nchunk, zs, info, n_accepted, next_token);
  return hipGetLastError();
}

// The scratch of the allocation-free entry point: one static array per GPU,
// held until the process ends.  Host code never passes `scratch` itself to a
// kernel (on the host it names a stand-in, not device memory): it uses the
// device address taken once per device with hipGetSymbolAddress.
static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_addr[kMaxDevices];

hipError_t noalloc_scratch(char** out) {
  *out = nullptr;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_addr[dev]) {  // first call on this device, which is current
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      (void)hipGetLastError();
      return e != hipSuccess ? e : hipErrorInvalidSymbol;
    }
    g_scratch_addr[dev] = p;
  }
  *out = static_cast<char*>(g_scratch_addr[dev]);
  return hipSuccess;
}

}  // namespace

size_t spec_accept_scratch_bytes(int b, int kd, int v, float temperature) {
  return accept_scratch(b, kd, v, temperature).total();
}

hipError_t launch_spec_accept(const float* draft, const float* target, const int32_t* tokens, const uint32_t* u24,
                              int b, int kd, int v, float temperature, int32_t* n_accepted, int32_t* next_token,
                              float* q_out, float* p_out, hipStream_t stream) {
  void* ws = nullptr;
  const hipError_t e = workspace(accept_scratch(b, kd, v, temperature).total(), stream, &ws);
  if (e != hipSuccess) return e;
  return enqueue_accept(draft, target, tokens, u24, b, kd, v, temperature, n_accepted, next_token, q_out, p_out,
                        static_cast<char*>(ws), stream);
}

hipError_t launch_spec_accept_noalloc(const float* draft, const float* target, const int32_t* tokens,
                                      const uint32_t* u24, int b, int kd, int v, float temperature,
                                      int32_t* n_accepted, int32_t* next_token, float* q_out, float* p_out,
                                      hipStream_t stream) {
  if (accept_scratch(b, kd, v, temperature).total() > kNoAllocScratchBytes) return hipErrorInvalidValue;
  char* ws = nullptr;
  const hipError_t e = noalloc_scratch(&ws);
  if (e != hipSuccess) return e;
  return enqueue_accept(draft, target, tokens, u24, b, kd, v, temperature, n_accepted, next_token, q_out, p_out, ws,
                        stream);
}


size_t spec_accept_multi_scratch_bytes(int b, int c, int kd, int v, float temperature, bool have_q, bool have_p) {
  const int64_t nchunk = (v + kChunk - 1) / kChunk;
  const int64_t rows_t = (int64_t)b * c * (kd + 1);
  if (temperature == 0.0f) return ((size_t)rows_t * nchunk * sizeof(ArgMax) + 255) / 256 * 256;
  const int64_t rows_d = (int64_t)kd * b * c;
  size_t bytes = ((size_t)(rows_t + rows_d) * nchunk * sizeof(double2) + 255) / 256 * 256;  // stats
  bytes += ((size_t)b * v * sizeof(int64_t) + 255) / 256 * 256;                              // residual grid
  if (!have_p) bytes += ((size_t)rows_t * v * sizeof(float) + 255) / 256 * 256;
  if (!have_q) bytes += ((size_t)rows_d * v * sizeof(float) + 255) / 256 * 256;
  return bytes;
}

hipError_t launch_spec_accept_multi(const float* draft, const float* target, const int32_t* tokens,
                                    const uint32_t* u24, int b, int c, int kd, int v, float temperature,
                                    int32_t* n_accepted, int32_t* next_token, int32_t* chain, float* q_out,
                                    float* p_out, hipStream_t stream) {
  void* wsv = nullptr;
  const hipError_t e =
      workspace(spec_accept_multi_scratch_bytes(b, c, kd, v, temperature, q_out != nullptr, p_out != nullptr), stream,
                &wsv);
  if (e != hipSuccess) return e;
  char* ws = static_cast<char*>(wsv);
  const int nchunk = (v + kChunk - 1) / kChunk;
  const int64_t rows_t = (int64_t)b * c * (kd + 1);
  if (temperature == 0.0f) {
    ArgMax* am = reinterpret_cast<ArgMax*>(ws);
    hipLaunchKernelGGL(argmax_kernel, dim3((unsigned)(rows_t * nchunk)), dim3(kThreads), 0, stream, target, v, nchunk,
                       am);
    hipLaunchKernelGGL(multi_greedy_kernel, dim3((unsigned)b), dim3(kThreads), 0, stream, tokens, b, c, kd, nchunk, am,
                       n_accepted, next_token, chain);
    return hipGetLastError();
  }
  const int64_t rows_d = (int64_t)kd * b * c, rows = rows_t + rows_d;
  double2* stats = reinterpret_cast<double2*>(ws);
  ws += ((size_t)rows * nchunk * sizeof(double2) + 255) / 256 * 256;
  int64_t* grid = reinterpret_cast<int64_t*>(ws);
  ws += ((size_t)b * v * sizeof(int64_t) + 255) / 256 * 256;
  float* p32 = p_out;
  if (!p32) {
    p32 = reinterpret_cast<float*>(ws);
    ws += ((size_t)rows_t * v * sizeof(float) + 255) / 256 * 256;
  }
  float* q32 = q_out;
  if (!q32 && rows_d > 0) q32 = reinterpret_cast<float*>(ws);
  hipLaunchKernelGGL(stats_kernel, dim3((unsigned)(rows * nchunk)), dim3(kThreads), 0, stream, draft, target, rows_t,
                     v, temperature, nchunk, stats);
  hipLaunchKernelGGL(probs_kernel, dim3((unsigned)(rows * nchunk)), dim3(kThreads), 0, stream, draft, target, rows_t,
                     v, temperature, nchunk, stats, q32, p32);
  hipLaunchKernelGGL(multi_kernel, dim3((unsigned)b), dim3(kMThreads), 0, stream, p32, q32, tokens, u24, b, c, kd, v,
                     nchunk, stats, grid, n_accepted, next_token, chain);
  return hipGetLastError();
}

}  // namespace sq

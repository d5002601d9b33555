// The decoder layer around the projections of a SpecQuant pass (draft
// generation, SS III-D.2; parent verification, SS III-D.3) for the Qwen2.5
// family the paper evaluates (SS IV), and the commit that restarts a
// sequence at its first rejected token (SS III-D.4):
//   embed_kernel        h = table[token] (fp32 residual stream)
//   add_rmsnorm_kernel  h += delta; x = f16(h / sqrt(mean(h^2) + eps) * w)
//   rope_kv_kernel      bias, rotary embedding of q and k, cache write of k, v
//   attn_chunk_kernel   causal grouped-query attention over a slot of 64-position
//                       chunks of the cache on the matrix cores (partial softmax)
//   attn_merge_kernel   merge of the slots in slot order
//   attn_chunk_lds_kernel<true>  the chunk kernel that also does rope_kv_kernel's
//                       work for its block (one launch less per layer)
//   silu_mul_kernel     t = f16(g / (1 + exp(-g)) * u)
//   commit_kernel       emitted tokens, next pending token, position
//   kv_adopt_kernel, commit_multi_kernel  the same with several draft chains per sequence
//
// Cache layout, per model and layer: keys [b][hkv][capacity][128] (a key is
// 256 contiguous bytes) and values position-minor, [b][hkv][128][capacity],
// so that the matrix-core product P.V reads each value fragment as two 8-byte
// runs of positions.  A row of a block of rows_per_seq rows of sequence b sits
// at position pos_base[b] + pos_offset + j.  The round never moves cache data:
// removing the rejected part of a block only moves pos_base, and the entries
// past it are overwritten before any row can attend to them.
#include "sq_device.hpp"
#include "sq_internal.hpp"

namespace sq {
namespace {

constexpr int kHd = 128;    // head dimension of the family
constexpr int kChunk = 64;  // cache positions per attention wavefront

// device status bits (the SQ_DEV_* values of the C header)
constexpr int32_t kBadToken = 1, kBadPos = 2, kOverflow = 4, kNoDist = 8;

typedef _Float16 half4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void flag(int32_t* status, int32_t bit) {
  if (status) atomicOr(status, bit);
}

constexpr uint16_t kNanF16 = 0x7E00;

// ------------------------------------------------------------------ embed
__global__ __launch_bounds__(256) void embed_kernel(const uint16_t* __restrict__ table, int64_t vocab, int hidden,
                                                    const int32_t* __restrict__ first,
                                                    const int32_t* __restrict__ rest, int b, int kd,
                                                    float* __restrict__ h, int32_t* __restrict__ status) {
  const int row = blockIdx.x;  // row = bi * (kd + 1) + j
  const int bi = row / (kd + 1), j = row - bi * (kd + 1);
  const int32_t tok = j == 0 ? first[bi] : rest[(int64_t)(j - 1) * b + bi];
  float* out = h + (int64_t)row * hidden;
  if (tok < 0 || tok >= vocab) {
    for (int c = threadIdx.x; c < hidden; c += blockDim.x) out[c] = __builtin_nanf("");
    if (threadIdx.x == 0) flag(status, kBadToken);
    return;
  }
  const uint16_t* src = table + (int64_t)tok * hidden;
  for (int c = threadIdx.x * 8; c < hidden; c += blockDim.x * 8) {
    const half8_t v = *reinterpret_cast<const half8_t*>(src + c);
    float4_t lo = {(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
    float4_t hi = {(float)v[4], (float)v[5], (float)v[6], (float)v[7]};
    *reinterpret_cast<float4_t*>(out + c) = lo;
    *reinterpret_cast<float4_t*>(out + c + 4) = hi;
  }
}

// ---------------------------------------------------- residual add + norm
// One workgroup of 256 threads per row of h; thread i holds the float4 cells
// i, i + 256, ... of the row in registers (NV of them: hidden <= 1024 NV).
// Every global load (the row of h, of delta and the norm weights) is issued
// before the first use, so the kernel waits for memory once.  Every row gets
// the residual add; the rows r * group + group - 1 are normalised into output
// row r (the arithmetic of rms_cell_sq / rms_inverse / rms_scale, shared with
// the projections that normalise their own input: the same bits).
template <int NV>
__global__ __launch_bounds__(256) void add_rmsnorm_kernel(float* __restrict__ h, const float* __restrict__ delta,
                                                          int hidden, const uint16_t* __restrict__ w, float eps,
                                                          int group, uint16_t* __restrict__ x) {
  __shared__ float red[4];
  const int64_t row = blockIdx.x;
  float* hr = h + row * hidden;
  const bool out_row = (row % group) == group - 1;
  const int n4 = hidden >> 2;
  float4_t v[NV], d[NV];
  uint2 wv[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = (int)threadIdx.x + 256 * i;
    const bool ok = c < n4;
    v[i] = ok ? reinterpret_cast<const float4_t*>(hr)[c] : float4_t{0.f, 0.f, 0.f, 0.f};
    d[i] = ok && delta ? reinterpret_cast<const float4_t*>(delta + row * hidden)[c] : float4_t{0.f, 0.f, 0.f, 0.f};
    wv[i] = ok && out_row ? reinterpret_cast<const uint2*>(w)[c] : uint2{0u, 0u};
  }
  if (delta) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int c = (int)threadIdx.x + 256 * i;
      if (c < n4) {
        v[i] += d[i];
        reinterpret_cast<float4_t*>(hr)[c] = v[i];
      }
    }
  }
  if (!out_row) return;  // uniform across the workgroup
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = (int)threadIdx.x + 256 * i;
    if (c < n4) ss += rms_cell_sq(v[i]);
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float r = rms_inverse(red, hidden, eps);
  uint16_t* xr = x + (row / group) * hidden;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = (int)threadIdx.x + 256 * i;
    if (c < n4) {
      const half4_t wh = __builtin_bit_cast(half4_t, wv[i]);
      half4_t o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = rms_scale(v[i][e], r, wh[e]);
      reinterpret_cast<uint2*>(xr)[c] = __builtin_bit_cast(uint2, o);
    }
  }
}

// ------------------------------------------------- bias + RoPE + cache write
// The rotation shared by rope_kv_kernel and the attention that rotates its own
// query rows and new cache entries (the same bits): pair (t, t + 64) of a head
// turns by pos * theta^(-2t/128), the angle and its cosine and sine in fp64,
// the turn itself in fp32 with every product rounded on its own.
__device__ __forceinline__ double rope_freq(int t, double theta) {
  return pow(theta, -2.0 * (double)t / (double)kHd);
}

__device__ __forceinline__ float2 rope_cos_sin(int64_t pos, double freq) {
  double sn, cs;
  sincos((double)pos * freq, &sn, &cs);
  return make_float2((float)cs, (float)sn);
}

__device__ __forceinline__ void rope_turn(float a, float e, float2 cs, float& ra, float& re) {
#pragma clang fp contract(off)
  ra = a * cs.x - e * cs.y;
  re = e * cs.x + a * cs.y;
}

// One wavefront per (row, head); lane t handles the pair (t, t + 64).
__global__ __launch_bounds__(64) void rope_kv_kernel(const float* __restrict__ qkv, const uint16_t* __restrict__ bias,
                                                     int hq, int hkv, int rps, const int32_t* __restrict__ pos_base,
                                                     int pos_offset, int64_t len_bound, int64_t capacity, double theta,
                                                     uint16_t* __restrict__ q_out, uint16_t* __restrict__ kc,
                                                     uint16_t* __restrict__ vc, int32_t* __restrict__ status) {
  const int r = blockIdx.x, hh = blockIdx.y;
  const int bi = r / rps, j = r - bi * rps;
  const int t = threadIdx.x;
  const int nh = hq + 2 * hkv;
  // the loads first (their addresses do not depend on the position), and the
  // frequency theta^(-2t/128) while they are in flight
  const int64_t pos = (int64_t)pos_base[bi] + pos_offset + j;
  const float* src = qkv + ((int64_t)r * nh + hh) * kHd;
  float a = src[t], e = src[t + 64];
  float ba = 0.f, be = 0.f;
  if (bias) {
    ba = f16_bits_to_f32(bias[hh * kHd + t]);
    be = f16_bits_to_f32(bias[hh * kHd + t + 64]);
  }
  const bool rot = hh < hq + hkv;
  const double freq = rot ? rope_freq(t, theta) : 0.0;
  if (pos < 0 || pos >= len_bound) {
    if (hh < hq) {
      q_out[((int64_t)r * hq + hh) * kHd + t] = kNanF16;
      q_out[((int64_t)r * hq + hh) * kHd + t + 64] = kNanF16;
    }
    if (t == 0 && hh == 0) flag(status, kBadPos);
    return;
  }
  if (bias) {
    a += ba;
    e += be;
  }
  if (rot) {
    float ra, re;
    rope_turn(a, e, rope_cos_sin(pos, freq), ra, re);
    uint16_t* dst = hh < hq ? q_out + ((int64_t)r * hq + hh) * kHd
                            : kc + (((int64_t)bi * hkv + (hh - hq)) * capacity + pos) * kHd;
    dst[t] = f32_to_f16_bits(ra);
    dst[t + 64] = f32_to_f16_bits(re);
  } else {
    uint16_t* vo = vc + ((int64_t)bi * hkv + (hh - hq - hkv)) * kHd * capacity + pos;
    vo[(int64_t)t * capacity] = f32_to_f16_bits(a);
    vo[(int64_t)(t + 64) * capacity] = f32_to_f16_bits(e);
  }
}

// ------------------------------------------------------------- attention
// Query rows of a block, per (sequence bi, kv head g): the block's rows of bi
// times the G = hq / hkv heads of g, ordered qi = j * G + gg, in tiles of 16.
// A wavefront takes one tile over a run of 64-position chunks of the cache,
// on the matrix cores (v_mfma_f32_16x16x32_f16; lane l holds A[l%16][8(l/16)
// .. +8) and B[8(l/16) .. +8)[l%16], D[4(l/16) + i][l%16]):
//   S^T = K . Q^T  -- A: 16 keys x 32 of the head dimension (lane l: key l%16,
//                     dims 32(l/16) + 8s .. +8 for step s), B: the same dims of
//                     16 query rows; lane l ends with the scores of keys
//                     4(l/16) + i of query l%16;
//   O = P . V      -- the lane's 8 scores of two adjacent key tiles are
//                     exactly its A fragment of P (keys 4(l/16) + i and
//                     16 + 4(l/16) + i of query l%16), and B takes the values
//                     of the same 8 keys at dim l%16 (+16 per output tile)
//                     from the position-minor value cache.
// Across its chunks the wavefront keeps, per query row, the running maximum m
// of the scaled scores (log2 units), l = sum of the weights p = 2^(s - m) and
// O = sum p v, rescaled by 2^(m_old - m_new) when m grows.  Keys after a row's
// position get p = 0.  Partial results (m, l, O) of several wavefronts merge
// as out = sum_w 2^(m_w - M) O_w / sum_w 2^(m_w - M) l_w, M = max_w m_w.
struct AttnTile {
  int hq, rps, G, nq;
};

__device__ __forceinline__ void attn_load_q(const uint16_t* __restrict__ q, const AttnTile& a, int bi, int g, int qt,
                                            int li, int lg, half8_t (&qf)[4]) {
  const half8_t zero8 = {0, 0, 0, 0, 0, 0, 0, 0};
  const int qi = 16 * qt + li;
  const bool qok = qi < a.nq;
  const int j = qok ? qi / a.G : 0, gg = qok ? qi - (qi / a.G) * a.G : 0;
  const half8_t* qp =
      reinterpret_cast<const half8_t*>(q + (((int64_t)bi * a.rps + j) * a.hq + g * a.G + gg) * kHd + 32 * lg);
#pragma unroll
  for (int s = 0; s < 4; ++s) qf[s] = qok ? qp[s] : zero8;
}

// A chunk's key and value fragments, loaded whole (the caller keeps key0 + 63
// inside the cache).
__device__ __forceinline__ void attn_load_kv(const uint16_t* __restrict__ kc, const uint16_t* __restrict__ vc,
                                             int64_t bg, int64_t capacity, int64_t key0, int li, int lg,
                                             half8_t (&kf)[4][4], half8_t (&vf)[2][8]) {
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) {
    const int64_t key = key0 + 16 * kt + li;
    const half8_t* kp = reinterpret_cast<const half8_t*>(kc + (bg * capacity + key) * kHd + 32 * lg);
#pragma unroll
    for (int s = 0; s < 4; ++s) kf[kt][s] = kp[s];
  }
#pragma unroll
  for (int t2 = 0; t2 < 2; ++t2) {
    const int64_t ka = key0 + 32 * t2 + 4 * lg, kb = ka + 16;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      const uint16_t* vp = vc + (bg * kHd + 16 * dt + li) * capacity;
      const half4_t a = *reinterpret_cast<const half4_t*>(vp + ka);
      const half4_t b = *reinterpret_cast<const half4_t*>(vp + kb);
      half8_t f;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        f[e] = a[e];
        f[4 + e] = b[e];
      }
      vf[t2][dt] = f;
    }
  }
}

// Zero the values of keys after the last row's position: stale entries may
// hold anything, and a zero weight times a NaN value is NaN.  Their keys need
// no mask: such a key's score only reaches its own entry of S, which the
// causal mask replaces by -inf.
__device__ __forceinline__ void attn_mask_v(int64_t key0, int64_t pmax, int lg, half8_t (&vf)[2][8]) {
  if (key0 + kChunk - 1 <= pmax) return;  // uniform: every key of the chunk is read
#pragma unroll
  for (int t2 = 0; t2 < 2; ++t2) {
    const int64_t ka = key0 + 32 * t2 + 4 * lg, kb = ka + 16;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      half8_t f = vf[t2][dt];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        f[e] = ka + e <= pmax ? f[e] : (half_t)0;
        f[4 + e] = kb + e <= pmax ? f[4 + e] : (half_t)0;
      }
      vf[t2][dt] = f;
    }
  }
}

// One chunk (keys key0 .. key0 + 63) into tile qt's running (m, l, O); the
// key fragment (kt, s) and value fragment (t2, dt) come from kfrag / vfrag,
// each called where the matrix cores take it.
template <class KF, class VF>
__device__ __forceinline__ void attn_update_src(const AttnTile& a, int64_t p0, int qt, int li, int lg,
                                                const half8_t (&qf)[4], KF kfrag, VF vfrag, int64_t key0, float& m,
                                                float& l, float4_t (&o)[8]) {
  const float sl2 = 1.4426950408889634f * 0.08838834764831845f;  // log2(e) / sqrt(128)
  const int qi = 16 * qt + li;
  const bool qok = qi < a.nq;
  const int j = qok ? qi / a.G : 0;
  float4_t st[4];
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) {
    float4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 4; ++s) acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(kfrag(kt, s), qf[s], acc, 0, 0, 0);
    st[kt] = acc;
  }
  const int64_t qpos = p0 + j;
  float cm = -__builtin_inff();
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t key = key0 + 16 * kt + 4 * lg + i;
      const float v = (qok && key <= qpos) ? st[kt][i] * sl2 : -__builtin_inff();
      st[kt][i] = v;
      cm = fmaxf(cm, v);
    }
  cm = fmaxf(cm, __shfl_xor(cm, 16, kWave));
  cm = fmaxf(cm, __shfl_xor(cm, 32, kWave));
  const float mn = fmaxf(m, cm);
  const bool none = mn == -__builtin_inff();  // no key of this row so far
  const float alpha = none ? 1.f : exp2f(m - mn);
  // p = hi + lo, both binary16 (hi = f16(p), lo = f16(p - hi), the difference
  // exact in fp32): two products with the values carry p to about 2^-22
  float psum = 0.f;
  half8_t pf[2], pl[2];
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float p = none ? 0.f : exp2f(st[kt][i] - mn);
      const half_t ph = (half_t)p;
      psum += p;
      pf[kt >> 1][(kt & 1) * 4 + i] = ph;
      pl[kt >> 1][(kt & 1) * 4 + i] = (half_t)(p - (float)ph);
    }
  psum += __shfl_xor(psum, 16, kWave);
  psum += __shfl_xor(psum, 32, kWave);
  l = l * alpha + psum;
  m = mn;
  // rows 4 lg + i of the output tile take the factor of query 4 lg + i
  float ar[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) ar[i] = __shfl(alpha, 4 * lg + i, kWave);
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) {
    float4_t acc = o[dt];
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] *= ar[i];
    const half8_t v0 = vfrag(0, dt), v1 = vfrag(1, dt);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(pl[0], v0, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(pl[1], v1, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(pf[0], v0, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(pf[1], v1, acc, 0, 0, 0);
    o[dt] = acc;
  }
}

__device__ __forceinline__ void attn_update(const AttnTile& a, int64_t p0, int qt, int li, int lg,
                                            const half8_t (&qf)[4], const half8_t (&kf)[4][4],
                                            const half8_t (&vf)[2][8], int64_t key0, float& m, float& l,
                                            float4_t (&o)[8]) {
  attn_update_src(
      a, p0, qt, li, lg, qf, [&](int kt, int s) { return kf[kt][s]; }, [&](int t2, int dt) { return vf[t2][dt]; },
      key0, m, l, o);
}

// One workgroup per (slot, sequence bi, kv head g); slot s covers the `span`
// consecutive chunks s * span .. s * span + span - 1, its tiles one per
// wavefront (up to 4 wavefronts, which read the same cache fragments; with
// more tiles, span 1 and each wavefront takes every 4th tile).  The slot's
// (m, l, O) go to global partials that attn_merge_kernel merges in slot
// order.
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void attn_chunk_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc, const uint16_t* __restrict__ vc, int hq, int hkv,
    int rps, int64_t capacity, const int32_t* __restrict__ pos_base, int pos_offset, int nslots, int span, int nq_pad,
    float* __restrict__ part_o, float2* __restrict__ part_ml) {
  const int slot = blockIdx.x;
  const int bg = blockIdx.y;  // bi * hkv + g
  const int bi = bg / hkv, g = bg - bi * hkv;
  const AttnTile a{hq, rps, hq / hkv, rps * (hq / hkv)};
  const int64_t p0 = (int64_t)pos_base[bi] + pos_offset;
  const int64_t pmax = p0 + rps - 1;
  // slot0 < len_bound <= capacity, so the slot's first chunk lies in the cache
  // whatever the positions: its loads are issued before the positions arrive
  const int64_t slot0 = (int64_t)slot * span * kChunk;
  const int lane = threadIdx.x & 63, li = lane & 15, lg = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nwave = blockDim.x >> 6;
  const int nqt = (a.nq + 15) >> 4;
  half8_t kf[4][4], vf[2][8];

  float* po = part_o + ((int64_t)bg * nslots + slot) * nq_pad * kHd;
  float2* pml = part_ml + ((int64_t)bg * nslots + slot) * nq_pad;
  auto store = [&](int qt, float m, float l, const float4_t(&o)[8]) {
#pragma unroll
    for (int dt = 0; dt < 8; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) po[(int64_t)(16 * qt + 4 * lg + i) * kHd + 16 * dt + li] = o[dt][i];
    if (lg == 0) pml[16 * qt + li] = make_float2(m, l);
  };

  if (nqt <= nwave) {  // one query tile per wavefront, its running sums kept across the slot's chunks
    const int qt = wave;
    half8_t qf[4];
    attn_load_q(q, a, bi, g, qt, li, lg, qf);
    attn_load_kv(kc, vc, bg, capacity, slot0, li, lg, kf, vf);
    if (slot0 > pmax) return;  // no row reads this slot (uniform); rows at negative positions mask every key
    float m = -__builtin_inff(), l = 0.f;
    float4_t o[8];
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[dt] = float4_t{0.f, 0.f, 0.f, 0.f};
    for (int t = 0; t < span; ++t) {
      const int64_t key0 = slot0 + (int64_t)t * kChunk;
      if (key0 > pmax || key0 >= capacity) break;  // uniform; rows past the cache read none of it
      if (t > 0) attn_load_kv(kc, vc, bg, capacity, key0, li, lg, kf, vf);
      attn_mask_v(key0, pmax, lg, vf);
      attn_update(a, p0, qt, li, lg, qf, kf, vf, key0, m, l, o);
    }
    store(qt, m, l, o);
  } else {  // more query tiles than wavefronts: span 1, tiles wave, wave + nwave, ...
    attn_load_kv(kc, vc, bg, capacity, slot0, li, lg, kf, vf);
    if (slot0 > pmax) return;
    attn_mask_v(slot0, pmax, lg, vf);
    for (int qt = wave; qt < nqt; qt += nwave) {
      half8_t qf[4];
      attn_load_q(q, a, bi, g, qt, li, lg, qf);
      float m = -__builtin_inff(), l = 0.f;
      float4_t o[8];
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) o[dt] = float4_t{0.f, 0.f, 0.f, 0.f};
      attn_update(a, p0, qt, li, lg, qf, kf, vf, slot0, m, l, o);
      store(qt, m, l, o);
    }
  }
}

// The same slots with the chunks staged through LDS, for blocks of 2 .. 4
// query tiles (whose wavefronts would otherwise each load the same key and
// value fragments) and for slots of several chunks: the workgroup's four
// wavefronts load each chunk once, as 16-byte cells of contiguous memory
// (keys: 16 KB in a row; values: 128 rows of 128 B), into one of two LDS
// buffers, while the wavefronts that own a query tile work on the previous
// chunk from the other buffer; each reads its fragments from LDS.  Rows are
// padded (keys to 272 B, values to 144 B), so that the lanes of one fragment
// read fall in distinct banks.  One barrier per chunk: it follows the issue
// of the next chunk's loads and waits only for the LDS writes.
constexpr int kLdsKeyStride = 136;  // halves per key row in LDS (128 + 8)
constexpr int kLdsValStride = 72;   // halves per value row in LDS (64 positions + 8)
constexpr int kLdsChunk = 64 * kLdsKeyStride + kHd * kLdsValStride;  // halves per chunk buffer
constexpr int kLdsThreads = 256;
constexpr int kLdsCells = 2 * kChunk * kHd * 2 / 16 / kLdsThreads;  // 16-byte cells per thread and chunk: 8

// The attention that also does rope_kv_kernel's work for its block: the
// sources of the rotation (the q|k|v projection rows) and where the new keys
// and values go.  At most 64 query rows per (sequence, kv head) and 16 rows
// per sequence.
struct RopeSrc {
  const float* qkv;      // [b rps][(hq + 2 hkv) * 128] fp32
  const uint16_t* bias;  // [(hq + 2 hkv) * 128] fp16, or null
  double theta;
  int64_t len_bound;
  uint16_t* kc;  // the caches, written at the block's valid positions
  uint16_t* vc;
  int32_t* status;
};
constexpr int kRopeMaxRows = 16;
// rotation items (row-head, four pairs) per thread: (64 query rows + 2 * 16) * 16 / 256
constexpr int kRopeItems = (64 + 2 * kRopeMaxRows) * 16 / kLdsThreads;

__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
}

// With ROPE, the workgroup first rotates its block's query rows (into LDS
// buffer 1, which holds no chunk until the second one is staged) and the new
// keys and values of kv head g (into LDS after the two buffers) with
// rope_kv_kernel's arithmetic, from q|k|v rows it loads before the positions
// arrive; the cosines and sines of (row, pair) are computed once, into buffer
// 1.  The workgroup whose slot holds a valid position of the block writes its
// new key and value to the caches (once each), and a staged chunk that holds
// such positions gets their new entries patched over the stale cells it read.
// Without ROPE, q is read as rope_kv_kernel wrote it.
template <bool ROPE>
__global__ __launch_bounds__(kLdsThreads) __attribute__((amdgpu_waves_per_eu(2))) void attn_chunk_lds_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc, const uint16_t* __restrict__ vc, int hq, int hkv,
    int rps, int64_t capacity, const int32_t* __restrict__ pos_base, int pos_offset, int nslots, int span, int nq_pad,
    float* __restrict__ part_o, float2* __restrict__ part_ml, RopeSrc rs) {
  extern __shared__ __align__(16) char smem[];
  half_t* lbuf = reinterpret_cast<half_t*>(smem);  // [2][kLdsChunk], then (ROPE) new keys and values [2][rps][128]
  const int slot = blockIdx.x;
  const int bg = blockIdx.y;  // bi * hkv + g
  const int bi = bg / hkv, g = bg - bi * hkv;
  const AttnTile a{hq, rps, hq / hkv, rps * (hq / hkv)};
  const int tid = threadIdx.x, lane = tid & 63, li = lane & 15, lg = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nqt = (a.nq + 15) >> 4;
  const int64_t slot0 = (int64_t)slot * span * kChunk;  // < len_bound <= capacity

  // cells of chunk key0 for this thread: i < 4 keys (key c / 16, part c % 16),
  // i >= 4 values (dim c' / 8, positions 8 (c' % 8) .. +8), c = tid + 256 i
  u32x4 pre[kLdsCells];
  auto load_chunk = [&](int64_t key0) {
#pragma unroll
    for (int i = 0; i < kLdsCells; ++i) {
      const int c = tid + kLdsThreads * i;
      if (i < kLdsCells / 2) {
        pre[i] = *reinterpret_cast<const u32x4*>(kc + ((int64_t)bg * capacity + key0 + (c >> 4)) * kHd + (c & 15) * 8);
      } else {
        const int c2 = c - kChunk * kHd / 8;
        pre[i] = *reinterpret_cast<const u32x4*>(vc + ((int64_t)bg * kHd + (c2 >> 3)) * capacity + key0 + (c2 & 7) * 8);
      }
    }
  };

  load_chunk(slot0);  // before the positions arrive: the slot's first chunk lies in the cache
  // ROPE: item idx = tid + 256 it is row-head r = idx / 16 (query rows qi < nq
  // of kv head g, then row j's key, then row j's value) and pairs 4 (idx % 16)
  // .. +4; its q|k|v sources do not depend on the positions
  const int nh = hq + 2 * hkv;
  const int nitems = ROPE ? (a.nq + 2 * rps) * 16 : 0;
  float4_t ulo[ROPE ? kRopeItems : 1], uhi[ROPE ? kRopeItems : 1];
  half4_t blo[ROPE ? kRopeItems : 1], bhi[ROPE ? kRopeItems : 1];
  auto item = [&](int idx, int& j, int& head, int& kind) {  // kind 0 query, 1 key, 2 value
    const int r = idx >> 4;
    if (r < a.nq) {
      j = r / a.G;
      head = g * a.G + (r - j * a.G);
      kind = 0;
    } else if (r < a.nq + rps) {
      j = r - a.nq;
      head = hq + g;
      kind = 1;
    } else {
      j = r - a.nq - rps;
      head = hq + hkv + g;
      kind = 2;
    }
  };
  if constexpr (ROPE) {
#pragma unroll
    for (int it = 0; it < kRopeItems; ++it) {
      const int idx = tid + kLdsThreads * it;
      if (idx < nitems) {
        int j, head, kind;
        item(idx, j, head, kind);
        const float* src = rs.qkv + ((int64_t)(bi * rps + j) * nh + head) * kHd + 4 * (idx & 15);
        ulo[it] = *reinterpret_cast<const float4_t*>(src);
        uhi[it] = *reinterpret_cast<const float4_t*>(src + 64);
        if (rs.bias) {
          const uint16_t* bp = rs.bias + head * kHd + 4 * (idx & 15);
          blo[it] = *reinterpret_cast<const half4_t*>(bp);
          bhi[it] = *reinterpret_cast<const half4_t*>(bp + 64);
        }
      }
    }
  }
  const int64_t p0 = (int64_t)pos_base[bi] + pos_offset;
  // the pair of every table entry this thread fills is tid % 64 (256 threads a row step)
  const double freq = ROPE ? rope_freq(tid & 63, rs.theta) : 0.0;
  const int64_t pmax = p0 + rps - 1;
  if constexpr (ROPE) {
    if (slot == 0 && g == 0 && tid < rps && (p0 + tid < 0 || p0 + tid >= rs.len_bound)) flag(rs.status, kBadPos);
  }
  if (slot0 > pmax) return;  // uniform across the workgroup: no row reads this slot
  const int64_t klast = pmax < capacity - 1 ? pmax : capacity - 1;  // rows past the cache read none of it
  const int64_t nt64 = (klast - slot0) / kChunk + 1;
  const int nt = nt64 < span ? (int)nt64 : span;  // chunks of the slot with a key at or before pmax
  const bool owner = wave < nqt;
  half8_t qf[4];
  half_t* newkv = lbuf + 2 * kLdsChunk;  // [2][rps][128]: the block's keys, then its values
  // a valid position of the block, in this slot: its new entry goes to the caches from here
  auto store_kv = [&](int64_t pos) {
    return pos >= 0 && pos < rs.len_bound && pos >= slot0 && pos < slot0 + (int64_t)span * kChunk;
  };
  if constexpr (ROPE) {
    half_t* qb = lbuf + kLdsChunk;                        // [nq][128] rotated query rows
    float2* tab = reinterpret_cast<float2*>(qb + 64 * kHd);  // [rps][64] cosine, sine of (row, pair)
    for (int e = tid; e < rps * 64; e += kLdsThreads) tab[e] = rope_cos_sin(p0 + (e >> 6), freq);
    lds_barrier();
#pragma unroll
    for (int it = 0; it < kRopeItems; ++it) {
      const int idx = tid + kLdsThreads * it;
      if (idx < nitems) {
        int j, head, kind;
        item(idx, j, head, kind);
        const int t0 = 4 * (idx & 15);
        half4_t lo, hi;
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          float u = ulo[it][x], v = uhi[it][x];
          if (rs.bias) {
            u += (float)blo[it][x];
            v += (float)bhi[it][x];
          }
          if (kind < 2) rope_turn(u, v, tab[j * 64 + t0 + x], u, v);
          const half_t hu = (half_t)u, hv = (half_t)v;  // scalar copies: vector element lvalues are
          lo[x] = hu;                                   // misread by bit_cast
          hi[x] = hv;
          if (kind == 2 && store_kv(p0 + j)) {
            uint16_t* vo = rs.vc + ((int64_t)bg * kHd + t0 + x) * capacity + p0 + j;
            vo[0] = __builtin_bit_cast(uint16_t, hu);
            vo[(int64_t)64 * capacity] = __builtin_bit_cast(uint16_t, hv);
          }
        }
        half_t* dst = kind == 0 ? qb + (idx >> 4) * kHd : newkv + ((kind - 1) * rps + j) * kHd;
        *reinterpret_cast<half4_t*>(dst + t0) = lo;
        *reinterpret_cast<half4_t*>(dst + t0 + 64) = hi;
        if (kind == 1 && store_kv(p0 + j)) {
          uint16_t* ko = rs.kc + ((int64_t)bg * capacity + p0 + j) * kHd + t0;
          *reinterpret_cast<half4_t*>(ko) = lo;
          *reinterpret_cast<half4_t*>(ko + 64) = hi;
        }
      }
    }
    lds_barrier();
    if (owner) {
      const half8_t zero8 = {0, 0, 0, 0, 0, 0, 0, 0};
      const int qi = 16 * wave + li;
#pragma unroll
      for (int s4 = 0; s4 < 4; ++s4)
        qf[s4] = qi < a.nq ? *reinterpret_cast<const half8_t*>(qb + qi * kHd + 32 * lg + 8 * s4) : zero8;
    }
  } else {
    if (owner) attn_load_q(q, a, bi, g, wave, li, lg, qf);
  }
  auto store_chunk = [&](half_t* b) {
#pragma unroll
    for (int i = 0; i < kLdsCells; ++i) {
      const int c = tid + kLdsThreads * i;
      if (i < kLdsCells / 2) {
        *reinterpret_cast<u32x4*>(b + (c >> 4) * kLdsKeyStride + (c & 15) * 8) = pre[i];
      } else {
        const int c2 = c - kChunk * kHd / 8;
        *reinterpret_cast<u32x4*>(b + 64 * kLdsKeyStride + (c2 >> 3) * kLdsValStride + (c2 & 7) * 8) = pre[i];
      }
    }
  };
  // ROPE: a staged chunk that holds valid positions of the block gets their
  // new entries over the stale ones read from the cache (after a barrier, so
  // that every plain cell is written first; a short rolled loop, off the
  // common path)
  auto patch_chunk = [&](half_t* b, int64_t key0) {
    if (!(ROPE && key0 + kChunk - 1 >= p0 && key0 <= pmax)) return;  // uniform
    lds_barrier();
#pragma unroll 1
    for (int e = tid; e < rps * (16 + kHd); e += kLdsThreads) {
      const bool key = e < rps * 16;
      const int j = key ? e >> 4 : (e - rps * 16) >> 7;
      const int64_t pos = p0 + j;
      if (pos < key0 || pos >= key0 + kChunk || pos < 0 || pos >= rs.len_bound) continue;
      const int r = (int)(pos - key0);
      if (key) {
        const int part = e & 15;
        *reinterpret_cast<u32x4*>(b + r * kLdsKeyStride + part * 8) =
            *reinterpret_cast<const u32x4*>(newkv + j * kHd + part * 8);
      } else {
        const int dv = (e - rps * 16) & (kHd - 1);
        b[64 * kLdsKeyStride + dv * kLdsValStride + r] = newkv[(rps + j) * kHd + dv];
      }
    }
  };
  store_chunk(lbuf);
  patch_chunk(lbuf, slot0);
  float m = -__builtin_inff(), l = 0.f;
  float4_t o[8];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) o[dt] = float4_t{0.f, 0.f, 0.f, 0.f};
  for (int t = 0; t < nt; ++t) {
    const int64_t key0 = slot0 + (int64_t)t * kChunk;
    if (t + 1 < nt) load_chunk(key0 + kChunk);
    // the LDS writes of buffer t % 2 are done; the next chunk's loads stay in flight
    lds_barrier();
    const half_t* b = lbuf + (t & 1) * kLdsChunk;
    if (owner) {
      const bool tail = key0 + kChunk - 1 > pmax;  // values of keys after pmax are zeroed (stale entries)
      auto kfrag = [&](int kt, int s4) {
        return *reinterpret_cast<const half8_t*>(b + (16 * kt + li) * kLdsKeyStride + 32 * lg + 8 * s4);
      };
      auto vfrag = [&](int t2, int dt) {
        const int ka = 32 * t2 + 4 * lg, kb = ka + 16;
        const half_t* vr = b + 64 * kLdsKeyStride + (16 * dt + li) * kLdsValStride;
        const half4_t va = *reinterpret_cast<const half4_t*>(vr + ka);
        const half4_t vb = *reinterpret_cast<const half4_t*>(vr + kb);
        half8_t f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          f[e] = (!tail || key0 + ka + e <= pmax) ? va[e] : (half_t)0;
          f[4 + e] = (!tail || key0 + kb + e <= pmax) ? vb[e] : (half_t)0;
        }
        return f;
      };
      attn_update_src(a, p0, wave, li, lg, qf, kfrag, vfrag, key0, m, l, o);
    }
    // buffer (t + 1) % 2 was last read before this chunk's barrier
    if (t + 1 < nt) {
      store_chunk(lbuf + ((t + 1) & 1) * kLdsChunk);
      patch_chunk(lbuf + ((t + 1) & 1) * kLdsChunk, key0 + kChunk);
    }
  }
  if (!owner) return;
  float* po = part_o + ((int64_t)bg * nslots + slot) * nq_pad * kHd;
  float2* pml = part_ml + ((int64_t)bg * nslots + slot) * nq_pad;
#pragma unroll
  for (int dt = 0; dt < 8; ++dt)
#pragma unroll
    for (int i = 0; i < 4; ++i) po[(int64_t)(16 * wave + 4 * lg + i) * kHd + 16 * dt + li] = o[dt][i];
  if (lg == 0) pml[16 * wave + li] = make_float2(m, l);
}

// One wavefront per (row, query head): the slots 0 .. pos / (64 span), in
// order, out = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s, M = max_s m_s.
// Lane c (mod 64) reads slot c's (m, l); lane t then sums dims 2t, 2t + 1
// over the slots, the loads of several slots in flight at once.
__global__ __launch_bounds__(64) void attn_merge_kernel(const float* __restrict__ part_o,
                                                        const float2* __restrict__ part_ml, int hq, int hkv, int rps,
                                                        int nch, int span, int nq_pad,
                                                        const int32_t* __restrict__ pos_base,
                                                        int pos_offset, int64_t len_bound,
                                                        uint16_t* __restrict__ out) {
  const int r = blockIdx.x, hh = blockIdx.y, lane = threadIdx.x;
  const int bi = r / rps, j = r - bi * rps;
  const int G = hq / hkv, g = hh / G, gg = hh - g * G;
  const int qi = j * G + gg;
  const int64_t pos = (int64_t)pos_base[bi] + pos_offset + j;
  const int64_t bg = (int64_t)bi * hkv + g;
  const float2* ml = part_ml + bg * nch * nq_pad + qi;
  const float* po = part_o + (bg * nch * nq_pad + qi) * kHd + 2 * lane;
  // the first 64 slots' (m, l) and the first slot's O before the position
  // arrives (slots past the row's last one are ignored below)
  const float2 ml0 = ml[(int64_t)(lane < nch ? lane : nch - 1) * nq_pad];
  const float2 o0 = *reinterpret_cast<const float2*>(po);
  uint16_t* o = out + ((int64_t)r * hq + hh) * kHd + 2 * lane;
  if (pos < 0 || pos >= len_bound) {
    o[0] = kNanF16;
    o[1] = kNanF16;
    return;
  }
  const int last = (int)(pos / kChunk / span);  // the last slot holding a key of this row
  float mx = lane <= last ? ml0.x : -__builtin_inff();
  for (int c = lane + 64; c <= last; c += 64) mx = fmaxf(mx, ml[(int64_t)c * nq_pad].x);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, kWave));
  float l = 0.f, a0 = 0.f, a1 = 0.f;
  if (last == 0) {  // one slot: O / l (what the sums below give with one slot)
    const float l0 = __shfl(ml0.y, 0, kWave);
    o[0] = f32_to_f16_bits(o0.x / l0);
    o[1] = f32_to_f16_bits(o0.y / l0);
    return;
  }
  for (int c0 = 0; c0 <= last; c0 += 64) {
    const int c = c0 + lane;
    float wl = 0.f;
    if (c <= last) {
      const float2 v = c0 == 0 ? ml0 : ml[(int64_t)c * nq_pad];
      wl = exp2f(v.x - mx);
      l += v.y * wl;
    }
    const int n = last - c0 + 1 < 64 ? last - c0 + 1 : 64;
    int i = 0;
    for (; i + 4 <= n; i += 4) {
      float2 p[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) p[u] = *reinterpret_cast<const float2*>(po + (int64_t)(c0 + i + u) * nq_pad * kHd);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float wc = __shfl(wl, i + u, kWave);
        a0 += p[u].x * wc;
        a1 += p[u].y * wc;
      }
    }
    for (; i < n; ++i) {
      const float2 p = *reinterpret_cast<const float2*>(po + (int64_t)(c0 + i) * nq_pad * kHd);
      const float wc = __shfl(wl, i, kWave);
      a0 += p.x * wc;
      a1 += p.y * wc;
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) l += __shfl_xor(l, off, kWave);
  o[0] = f32_to_f16_bits(a0 / l);
  o[1] = f32_to_f16_bits(a1 / l);
}

// ------------------------------------------------------------- SiLU . up
__global__ __launch_bounds__(256) void silu_mul_kernel(const float* __restrict__ gu, int64_t m, int64_t inter,
                                                       uint16_t* __restrict__ t) {
  const int64_t total = m * inter;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = i / inter, col = i - row * inter;
    const float gv = gu[row * 2 * inter + col], uv = gu[row * 2 * inter + inter + col];
    t[i] = silu_gate_bits(gv, uv);
  }
}

// ---------------------------------------------------------------- commit
__global__ __launch_bounds__(256) void commit_kernel(const int32_t* __restrict__ n_accepted,
                                                     const int32_t* __restrict__ next_token,
                                                     const int32_t* __restrict__ drafts, int b, int kd,
                                                     int32_t* __restrict__ pending, int32_t* __restrict__ prev,
                                                     int32_t* __restrict__ pos_base, int32_t* __restrict__ out_tokens,
                                                     int64_t out_capacity, int32_t* __restrict__ out_len,
                                                     int32_t* __restrict__ status) {
  const int bi = blockIdx.x * blockDim.x + threadIdx.x;
  if (bi >= b) return;
  const int n = n_accepted[bi];
  if (n < 0 || n > kd) {  // the round had no distribution for this sequence
    flag(status, kNoDist);
    return;
  }
  if (out_tokens) {
    const int64_t len = out_len[bi];
    int32_t* dst = out_tokens + (int64_t)bi * out_capacity;
    for (int i = 0; i <= n; ++i) {
      const int32_t tok = i < n ? drafts[(int64_t)i * b + bi] : next_token[bi];
      if (len + i >= 0 && len + i < out_capacity)
        dst[len + i] = tok;
      else
        flag(status, kOverflow);
    }
    out_len[bi] = (int32_t)(len + n + 1);
  }
  prev[bi] = n >= 1 ? drafts[(int64_t)(n - 1) * b + bi] : pending[bi];
  pending[bi] = next_token[bi];
  pos_base[bi] += n + 1;
}

// ------------------------------------------------ several chains per sequence
// Sequence s drafts c chains, held as cache rows s * c + j of every layer
// ([layers][b c][hkv][capacity][128] keys, [layers][b c][hkv][128][capacity]
// values).  After acceptance the chain `chain[s]` holds the accepted prefix;
// its entries at positions pos + lo_offset .. pos + n + hi_offset are copied
// to the other chains of s (one workgroup per (layer, destination row, kv
// head), lane d one dimension), so that every chain continues from it.
__global__ __launch_bounds__(128) void kv_adopt_kernel(uint16_t* __restrict__ kc, uint16_t* __restrict__ vc, int bc,
                                                       int c, int hkv, int64_t capacity,
                                                       const int32_t* __restrict__ chain,
                                                       const int32_t* __restrict__ n_accepted,
                                                       const int32_t* __restrict__ pos_base, int lo_offset,
                                                       int hi_offset) {
  const int l = blockIdx.x, dst = blockIdx.y, g = blockIdx.z, d = threadIdx.x;
  const int s = dst / c;
  const int src_j = chain[s], n = n_accepted[s];
  if (src_j < 0 || src_j >= c || n < 0 || dst == s * c + src_j) return;
  const int src = s * c + src_j;
  const int64_t pos = pos_base[src];
  int64_t lo = pos + lo_offset, hi = pos + n + hi_offset;
  lo = lo < 0 ? 0 : lo;
  hi = hi >= capacity ? capacity - 1 : hi;
  const int64_t kl = (int64_t)l * bc * hkv;
  const uint16_t* ks = kc + ((kl + (int64_t)src * hkv + g) * capacity) * kHd;
  uint16_t* kd_ = kc + ((kl + (int64_t)dst * hkv + g) * capacity) * kHd;
  const uint16_t* vs = vc + ((kl + (int64_t)src * hkv + g) * kHd + d) * capacity;
  uint16_t* vd = vc + ((kl + (int64_t)dst * hkv + g) * kHd + d) * capacity;
  for (int64_t p = lo; p <= hi; ++p) {
    kd_[p * kHd + d] = ks[p * kHd + d];
    vd[p] = vs[p];
  }
}

// The commit with c chains per sequence: the accepted chain's drafts, then
// the next token, are emitted; every chain of the sequence restarts from it.
__global__ __launch_bounds__(256) void commit_multi_kernel(const int32_t* __restrict__ n_accepted,
                                                           const int32_t* __restrict__ next_token,
                                                           const int32_t* __restrict__ chain,
                                                           const int32_t* __restrict__ drafts, int b, int c, int kd,
                                                           int32_t* __restrict__ pending, int32_t* __restrict__ prev,
                                                           int32_t* __restrict__ pos_base,
                                                           int32_t* __restrict__ out_tokens, int64_t out_capacity,
                                                           int32_t* __restrict__ out_len,
                                                           int32_t* __restrict__ status) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= b) return;
  const int n = n_accepted[s], src = chain[s];
  if (n < 0 || n > kd || src < 0 || src >= c) {  // the round had no distribution for this sequence
    flag(status, kNoDist);
    return;
  }
  auto draft = [&](int i) { return drafts[((int64_t)i * b + s) * c + src]; };
  if (out_tokens) {
    const int64_t len = out_len[s];
    int32_t* dst = out_tokens + (int64_t)s * out_capacity;
    for (int i = 0; i <= n; ++i) {
      const int32_t tok = i < n ? draft(i) : next_token[s];
      if (len + i >= 0 && len + i < out_capacity)
        dst[len + i] = tok;
      else
        flag(status, kOverflow);
    }
    out_len[s] = (int32_t)(len + n + 1);
  }
  const int32_t pv = n >= 1 ? draft(n - 1) : pending[s * c + src];
  const int32_t nx = next_token[s];
  const int32_t pb = pos_base[s * c + src] + n + 1;
  for (int j = 0; j < c; ++j) {
    prev[s * c + j] = pv;
    pending[s * c + j] = nx;
    pos_base[s * c + j] = pb;
  }
}

}  // namespace

hipError_t launch_embed_block(const uint16_t* table, int64_t vocab, int hidden, const int32_t* first,
                              const int32_t* rest, int b, int kd, float* h, int32_t* status, hipStream_t stream) {
  hipLaunchKernelGGL(embed_kernel, dim3((unsigned)(b * (kd + 1))), dim3(256), 0, stream, table, vocab, hidden, first,
                     rest, b, kd, h, status);
  return hipGetLastError();
}

hipError_t launch_add_rmsnorm(float* h, const float* delta, int64_t m, int hidden, const uint16_t* w, float eps,
                              int group, uint16_t* x, hipStream_t stream) {
  const int n4 = hidden / 4;
  const dim3 grid((unsigned)m), block(256);
  if (n4 <= 256)
    hipLaunchKernelGGL(add_rmsnorm_kernel<1>, grid, block, 0, stream, h, delta, hidden, w, eps, group, x);
  else if (n4 <= 512)
    hipLaunchKernelGGL(add_rmsnorm_kernel<2>, grid, block, 0, stream, h, delta, hidden, w, eps, group, x);
  else if (n4 <= 1024)
    hipLaunchKernelGGL(add_rmsnorm_kernel<4>, grid, block, 0, stream, h, delta, hidden, w, eps, group, x);
  else if (n4 <= 2048)
    hipLaunchKernelGGL(add_rmsnorm_kernel<8>, grid, block, 0, stream, h, delta, hidden, w, eps, group, x);
  else
    hipLaunchKernelGGL(add_rmsnorm_kernel<16>, grid, block, 0, stream, h, delta, hidden, w, eps, group, x);
  return hipGetLastError();
}

hipError_t launch_rope_kv(const float* qkv, const uint16_t* bias, int m, int hq, int hkv, int rps,
                          const int32_t* pos_base, int pos_offset, int64_t len_bound, int64_t capacity, double theta,
                          uint16_t* q_out, uint16_t* kc, uint16_t* vc, int32_t* status, hipStream_t stream) {
  hipLaunchKernelGGL(rope_kv_kernel, dim3((unsigned)m, (unsigned)(hq + 2 * hkv)), dim3(64), 0, stream, qkv, bias, hq,
                     hkv, rps, pos_base, pos_offset, len_bound, capacity, theta, q_out, kc, vc, status);
  return hipGetLastError();
}

namespace {
// Chunks per wavefront: about 512 wavefronts in all (two per CU) once the
// cache is long enough, at most 16 chunks each; a single chunk when the
// block has more than 4 query tiles.
int attention_span(int b, int hq, int hkv, int rps, int64_t len_bound) {
  const int64_t nch = (len_bound + kChunk - 1) / kChunk;
  const int nqt = (rps * (hq / hkv) + 15) / 16;
  if (nqt > 4) return 1;
  int64_t span = nch * b * hkv / 512;
  span = span < 1 ? 1 : (span > 16 ? 16 : span);
  return (int)span;
}
}  // namespace

size_t attention_workspace_bytes(int b, int hq, int hkv, int rps, int64_t len_bound) {
  const int span = attention_span(b, hq, hkv, rps, len_bound);
  const int64_t nslots = ((len_bound + kChunk - 1) / kChunk + span - 1) / span;
  const int nq_pad = (rps * (hq / hkv) + 15) / 16 * 16;
  return (size_t)b * hkv * nslots * nq_pad * (kHd * sizeof(float) + sizeof(float2));
}

hipError_t launch_attention(const uint16_t* q, const uint16_t* kc, const uint16_t* vc, int b, int rps, int hq,
                            int hkv, int64_t capacity, const int32_t* pos_base, int pos_offset, int64_t len_bound,
                            uint16_t* out, hipStream_t stream) {
  const int span = attention_span(b, hq, hkv, rps, len_bound);
  const int nslots = (int)(((len_bound + kChunk - 1) / kChunk + span - 1) / span);
  const int nq_pad = (rps * (hq / hkv) + 15) / 16 * 16;
  void* ws = nullptr;
  const hipError_t e = workspace(attention_workspace_bytes(b, hq, hkv, rps, len_bound), stream, &ws);
  if (e != hipSuccess) return e;
  float* part_o = static_cast<float*>(ws);
  float2* part_ml = reinterpret_cast<float2*>(part_o + (size_t)b * hkv * nslots * nq_pad * kHd);
  const int nqt = nq_pad / 16;
  if ((nqt >= 2 && nqt <= 4) || (nqt == 1 && span >= 2)) {
    // chunks through LDS: loaded once for the block's tiles, the next one in flight
    const size_t lds = (size_t)2 * kLdsChunk * sizeof(uint16_t);
    hipLaunchKernelGGL(attn_chunk_lds_kernel<false>, dim3((unsigned)nslots, (unsigned)(b * hkv)), dim3(kLdsThreads),
                       lds, stream, q, kc, vc, hq, hkv, rps, capacity, pos_base, pos_offset, nslots, span, nq_pad,
                       part_o, part_ml, RopeSrc{});
  } else {
    const int waves = nqt < 4 ? nqt : 4;  // one query tile per wavefront (16 rows each), at most 4
    hipLaunchKernelGGL(attn_chunk_kernel, dim3((unsigned)nslots, (unsigned)(b * hkv)), dim3(64 * waves), 0, stream, q,
                       kc, vc, hq, hkv, rps, capacity, pos_base, pos_offset, nslots, span, nq_pad, part_o, part_ml);
  }
  hipLaunchKernelGGL(attn_merge_kernel, dim3((unsigned)(b * rps), (unsigned)hq), dim3(64), 0, stream, part_o,
                     part_ml, hq, hkv, rps, nslots, span, nq_pad, pos_base, pos_offset, len_bound, out);
  return hipGetLastError();
}

hipError_t launch_rope_attention(const float* qkv, const uint16_t* bias, int b, int rps, int hq, int hkv,
                                 int64_t capacity, const int32_t* pos_base, int pos_offset, int64_t len_bound,
                                 double theta, uint16_t* kc, uint16_t* vc, uint16_t* out, int32_t* status,
                                 hipStream_t stream) {
  if (rps > kRopeMaxRows || rps * (hq / hkv) > 64) return hipErrorNotSupported;
  const int span = attention_span(b, hq, hkv, rps, len_bound);
  const int nslots = (int)(((len_bound + kChunk - 1) / kChunk + span - 1) / span);
  const int nq_pad = (rps * (hq / hkv) + 15) / 16 * 16;
  void* ws = nullptr;
  const hipError_t e = workspace(attention_workspace_bytes(b, hq, hkv, rps, len_bound), stream, &ws);
  if (e != hipSuccess) return e;
  float* part_o = static_cast<float*>(ws);
  float2* part_ml = reinterpret_cast<float2*>(part_o + (size_t)b * hkv * nslots * nq_pad * kHd);
  const size_t lds = ((size_t)2 * kLdsChunk + (size_t)2 * rps * kHd) * sizeof(uint16_t);
  const RopeSrc rs{qkv, bias, theta, len_bound, kc, vc, status};
  hipLaunchKernelGGL(attn_chunk_lds_kernel<true>, dim3((unsigned)nslots, (unsigned)(b * hkv)), dim3(kLdsThreads), lds,
                     stream, nullptr, kc, vc, hq, hkv, rps, capacity, pos_base, pos_offset, nslots, span, nq_pad,
                     part_o, part_ml, rs);
  hipLaunchKernelGGL(attn_merge_kernel, dim3((unsigned)(b * rps), (unsigned)hq), dim3(64), 0, stream, part_o,
                     part_ml, hq, hkv, rps, nslots, span, nq_pad, pos_base, pos_offset, len_bound, out);
  return hipGetLastError();
}

hipError_t launch_silu_mul(const float* gu, int64_t m, int64_t inter, uint16_t* t, hipStream_t stream) {
  const int64_t total = m * inter;
  int64_t blocks = (total + 255) / 256;
  const int64_t cap = (int64_t)cu_count() * 8;
  if (blocks > cap) blocks = cap;
  hipLaunchKernelGGL(silu_mul_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, gu, m, inter, t);
  return hipGetLastError();
}

hipError_t launch_spec_commit(const int32_t* n_accepted, const int32_t* next_token, const int32_t* drafts, int b,
                              int kd, int32_t* pending, int32_t* prev, int32_t* pos_base, int32_t* out_tokens,
                              int64_t out_capacity, int32_t* out_len, int32_t* status, hipStream_t stream) {
  hipLaunchKernelGGL(commit_kernel, dim3((unsigned)((b + 255) / 256)), dim3(256), 0, stream, n_accepted, next_token,
                     drafts, b, kd, pending, prev, pos_base, out_tokens, out_capacity, out_len, status);
  return hipGetLastError();
}

}  // namespace sq

namespace sq {

hipError_t launch_kv_adopt(uint16_t* kc, uint16_t* vc, int layers, int b, int c, int hkv, int64_t capacity,
                           const int32_t* chain, const int32_t* n_accepted, const int32_t* pos_base, int lo_offset,
                           int hi_offset, hipStream_t stream) {
  hipLaunchKernelGGL(kv_adopt_kernel, dim3((unsigned)layers, (unsigned)(b * c), (unsigned)hkv), dim3(kHd), 0, stream,
                     kc, vc, b * c, c, hkv, capacity, chain, n_accepted, pos_base, lo_offset, hi_offset);
  return hipGetLastError();
}

hipError_t launch_spec_commit_multi(const int32_t* n_accepted, const int32_t* next_token, const int32_t* chain,
                                    const int32_t* drafts, int b, int c, int kd, int32_t* pending, int32_t* prev,
                                    int32_t* pos_base, int32_t* out_tokens, int64_t out_capacity, int32_t* out_len,
                                    int32_t* status, hipStream_t stream) {
  hipLaunchKernelGGL(commit_multi_kernel, dim3((unsigned)((b + 255) / 256)), dim3(256), 0, stream, n_accepted,
                     next_token, chain, drafts, b, c, kd, pending, prev, pos_base, out_tokens, out_capacity, out_len,
                     status);
  return hipGetLastError();
}

}  // namespace sq

/*
 * specquant.h -- C ABI of the SpecQuant hot path on MI355X (gfx950).
 *
 * SpecQuant (arXiv 2609.21704) derives low-precision draft parents from one
 * FP16 parent (Q4 = f(W16, 4), Q8 = f(W16, 8), Q16 = W16; SS III-A), drafts
 * tokens with a quantized parent (SS III-D.2), verifies the drafted block with
 * the FP16 parent (SS III-D.3) and accepts or corrects tokens (SS III-D.4 and
 * the guess-set rule of SS III-A).  This library provides the data-parallel
 * steps of one such round as asynchronous HIP kernels:
 *
 *   sq_quantize_int4_g128  FP16 parent -> INT4 group-128 draft copy (offline)
 *   sq_quantize_fp8_e4m3   FP16 parent -> FP8 E4M3 draft copy (offline)
 *   sq_qgemv_w4a16         draft projection y = x . W4'^T, m <= 8 rows
 *   sq_qgemv_w8a16         draft projection y = x . W8'^T, m <= 8 rows
 *   sq_verify_gemm_f16     parent verification y = x . W16^T, m <= 64 rows
 *   sq_spec_accept         LM-head softmax + accept / reject / resample
 *
 * Conventions shared by every call
 *   - Matrices are row-major and contiguous.  A weight matrix is W[n][k]
 *     (n output features, k reduction features); activations are x[m][k];
 *     outputs are y[m][n] = sum_c x[m][c] * W'[n][c].
 *   - binary16 (fp16) data is passed as uint16_t bit patterns.
 *   - Every array argument is a DEVICE pointer owned by the caller; the library
 *     never frees or retains caller memory.  Pointers to x, codes and w16 must
 *     be 16-byte aligned; every other pointer must be aligned to its element.
 *   - Each call validates its arguments on the host, enqueues its kernels on
 *     `stream` and returns without synchronising.  A non-SQ_OK status means
 *     nothing was enqueued (SQ_ERR_DEVICE: a launch or an allocation failed).
 *   - Outputs must not overlap inputs or each other (SQ_ERR_ALIAS).
 *   - Some kernels use a library-owned device workspace (split-K partial sums,
 *     K-slice meeting slots, softmax row statistics), one per device.  It is
 *     allocated on first use and grows when a call needs more; a buffer it
 *     outgrows is kept, never freed, until the process ends, because a graph
 *     captured while it was current keeps using it.  The library never
 *     allocates while `stream` is being captured: a call that would need a
 *     larger workspace then returns SQ_ERR_CAPTURE and enqueues nothing (run
 *     the same call once outside capture first).  The workspace is shared by
 *     all calls on a device, so calls on one device must be ordered on one
 *     stream (calls on concurrently running streams of a device race on it).
 *   - Results are deterministic: the same inputs give the same bits.
 */
#ifndef SPECQUANT_H
#define SPECQUANT_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SQ_ABI_VERSION 2

typedef enum sq_status {
  SQ_OK = 0,
  SQ_ERR_NULL = 1,        /* a required pointer is NULL                              */
  SQ_ERR_SHAPE = 2,       /* a size is outside the supported range                   */
  SQ_ERR_ALIGN = 3,       /* a pointer is misaligned                                 */
  SQ_ERR_ALIAS = 4,       /* an output overlaps an input or another output           */
  SQ_ERR_NONFINITE = 5,   /* a scalar argument is NaN or infinite (temperature)      */
  SQ_ERR_UNSUPPORTED = 6, /* a dtype or mode the call does not support (y_dtype,
                             T < 0, q_out / p_out requested at T = 0)                */
  SQ_ERR_DEVICE = 7,      /* the HIP runtime reported an error; nothing enqueued     */
  SQ_ERR_CAPTURE = 8      /* the workspace would have to grow while `stream` is
                             being captured; nothing enqueued                        */
} sq_status;

typedef enum sq_dtype { SQ_F16 = 0, SQ_F32 = 1 } sq_dtype;

/* INT4 group-128 quantization of the FP16 parent: the low-precision parent
 * Q4 = f(W16, 4) of SS III-A.1 (the paper states no formula; this is
 * asymmetric round-to-nearest-even per group of 128 consecutive k):
 *   for each row r and group g (k = 128g .. 128g+127):
 *     lo = min(0, min w), hi = max(0, max w)
 *     all-zero group: s = 1, z = 0, q = 0
 *     else  s = smallest fp16 >= (hi - lo) / 15          (computed in fp64)
 *           z = clamp(rint(-lo / s), 0, 15)
 *           q = clamp(rint(w / s) + z, 0, 15)            (ties to even)
 *   dequantized weight w' = (q - z) * s, |w - w'| <= s / 2.
 * w16    [n][k] fp16 (16-B aligned), k % 128 == 0, 1 <= n, 128 <= k <= 2^20
 * codes  [n][k/2] u8 out: element 2j in the low nibble of byte j (16-B aligned)
 * scales [n][k/128] fp16 out; zeros [n][k/128] fp16 out (integers 0..15)
 * nonfinite_flag: nullable int32 device word; set to 1 (never cleared) when a
 *   group holds NaN or Inf.  Such a group gets codes 0, scale NaN, zero 0. */
sq_status sq_quantize_int4_g128(const uint16_t* w16, int64_t n, int64_t k, uint8_t* codes,
                                uint16_t* scales, uint16_t* zeros, int32_t* nonfinite_flag,
                                hipStream_t stream);

/* FP8 E4M3 quantization of the FP16 parent, one fp32 scale per output row:
 * the medium-precision parent Q8 = f(W16, 8) of SS III-A.2 (format: OCP E4M3,
 * bias 7, max 448, no infinities):
 *   s_r = fl32(amax_r / 448) (1.0 for an all-zero row), amax in fp64
 *   c   = RNE-encode(w / s_r) computed in fp64, saturating to +-448, the sign
 *         of zero kept; dequantized weight w' = decode(c) * s_r.
 * w16 [n][k] fp16 (16-B aligned), k % 16 == 0, 1 <= n, 16 <= k <= 2^20
 * codes [n][k] u8 out (16-B aligned); scales [n] f32 out
 * nonfinite_flag: as for the INT4 call; such a row gets codes 0, scale NaN. */
sq_status sq_quantize_fp8_e4m3(const uint16_t* w16, int64_t n, int64_t k, uint8_t* codes,
                               float* scales, int32_t* nonfinite_flag, hipStream_t stream);

/* Draft projection with the INT4 parent (draft generation, SS III-D.2):
 *   y[i][r] = sum_c x[i][c] * (q[r][c] - z[r][c/128]) * s[r][c/128]
 * dequantized in registers; fp32 accumulation; y rounded once to y_dtype.
 * x [m][k] fp16, 1 <= m <= 8; k % 128 == 0, 128 <= k <= 2^20
 * codes/scales/zeros as produced by sq_quantize_int4_g128 for an [n][k] matrix
 * y [m][n] of y_dtype (SQ_F16 or SQ_F32), 1 <= n <= 2^31 - 1. */
sq_status sq_qgemv_w4a16(const uint16_t* x, int64_t m, int64_t k, const uint8_t* codes,
                         const uint16_t* scales, const uint16_t* zeros, int64_t n, void* y,
                         sq_dtype y_dtype, hipStream_t stream);

/* Draft projection with the FP8 parent (draft generation, SS III-D.2):
 *   y[i][r] = s[r] * sum_c x[i][c] * decode(codes[r][c])
 * x [m][k] fp16, 1 <= m <= 8, k % 16 == 0, 16 <= k <= 2^20;
 * codes [n][k] u8, scales [n] f32 as produced by sq_quantize_fp8_e4m3;
 * y [m][n] of y_dtype. */
sq_status sq_qgemv_w8a16(const uint16_t* x, int64_t m, int64_t k, const uint8_t* codes,
                         const float* scales, int64_t n, void* y, sq_dtype y_dtype,
                         hipStream_t stream);

/* Parent verification of the drafted block with Q16 = W16 (SS III-D.3): the
 * FP16 parent processes the m = b * (kd + 1) drafted positions in one pass.
 *   y[i][r] = sum_c x[i][c] * w16[r][c]        (fp32 accumulation of exact products)
 * x [m][k] fp16, 1 <= m <= 64, k % 8 == 0, 8 <= k <= 2^20;
 * w16 [n][k] fp16; y [m][n] of y_dtype. */
sq_status sq_verify_gemm_f16(const uint16_t* x, int64_t m, int64_t k, const uint16_t* w16,
                             int64_t n, void* y, sq_dtype y_dtype, hipStream_t stream);

/* LM-head softmax and speculative acceptance or correction (SS III-D.4; the
 * guess-set rule of SS III-A), for b sequences with kd drafted tokens each:
 *   q_i = softmax(draft_logits_i / T), p_i = softmax(target_logits_i / T),
 *   computed in fp64 (z = l / T, exp(z - max z) / sum exp(z - max z)) and held
 *   in fp32 -- the values q_out / p_out return.  Decisions and draw weights
 *   are formed in fp64 from those fp32 values, so q_out / p_out reproduce them
 *   exactly.
 * T > 0 (stochastic): position i (0 <= i < kd) with draft token x_i is
 *   accepted iff u_i * q_i(x_i) < p_i(x_i), u_i = (u24[s][i] & 0xFFFFFF) / 2^24;
 *   n_accepted = index of the first rejection (kd if none).  At a rejection the
 *   emitted token is drawn from max(0, p_n - q_n) renormalised (from p_n if
 *   that mass is zero on the fixed-point grid); otherwise the bonus token is
 *   drawn from p_kd.  Draws use u24[s][kd]: weights r are put on the grid
 *   R = rint(r * 2^60) (int64), Z = sum R, t = floor(u24 * Z / 2^24), and the
 *   token is the smallest j whose running sum of R exceeds t.  A draft token
 *   outside [0, v) is rejected.
 * Logits of -inf are masked tokens (probability 0).  A row holding a NaN or
 *   +inf logit, or no finite logit, has no distribution: its sequence gets
 *   n_accepted = next_token = -1 (T > 0: any of its 2 kd + 1 rows; T = 0: its
 *   kd + 1 target rows), and its rows of q_out / p_out are NaN.
 * T = 0 (greedy, the paper's "if parent agrees" rule): position i is accepted
 *   iff x_i == argmax p_i (smallest index on ties); the emitted token is the
 *   argmax of the first disagreeing row, or of row kd.  u24 may be NULL.
 * kd = 0 turns the call into a plain sampler of target row 0 (draft sampling).
 * draft_logits  [kd][b][v] f32 (position-major: one draft step for all b;
 *               may be NULL when kd == 0)
 * target_logits [b][kd+1][v] f32 (sequence-major: the parent's verify rows)
 * draft_tokens  [kd][b] int32 (position-major like draft_logits; NULL allowed
 *               when kd == 0)
 * u24           [b][kd+1] uint32
 * n_accepted [b] int32 out; next_token [b] int32 out.  The emitted tokens of
 *   sequence s are draft_tokens[0 .. n_accepted[s])[s] then next_token[s].
 * q_out [kd][b][v] f32, p_out [b][kd+1][v] f32: optional (nullable) copies of
 *   the distributions, T > 0 only.
 * Limits: 1 <= b < 2^24, 0 <= kd <= 64, 1 <= v <= 2^26,
 *   b * (2 kd + 1) * ceil(v / 4096) < 2^24; T finite and >= 0. */
sq_status sq_spec_accept(const float* draft_logits, const float* target_logits,
                         const int32_t* draft_tokens, const uint32_t* u24, int32_t b, int32_t kd,
                         int32_t v, float temperature, int32_t* n_accepted, int32_t* next_token,
                         float* q_out, float* p_out, hipStream_t stream);

/* The accept call of sq_spec_accept for callers that cannot allocate device
 * memory: code under HIP graph capture, serving loops and harnesses that
 * forbid allocation.  Same arguments, kernels and results as sq_spec_accept,
 * but the call allocates nothing: its scratch (row statistics, chunk weights,
 * per-sequence state) is a static device array of SQ_NOALLOC_SCRATCH_BYTES
 * per GPU, held by the library until the process ends.  A call needs
 *   T > 0: 16 * (b * (2 kd + 1) * C) + 16 * (b * C) + 40 * b bytes,
 *   T = 0: 8 * (b * (kd + 1) * C) bytes, C = ceil(v / 4096),
 * each term rounded up to a multiple of 256 (the 40 b term excepted); a call
 * that needs more than SQ_NOALLOC_SCRATCH_BYTES returns SQ_ERR_SHAPE and
 * enqueues nothing (e.g. 4 sequences, kd = 8, v = 151936 need 44 KB; 256
 * sequences at kd = 8 need 2.8 MB).  Every call on a GPU shares that GPU's
 * array, and nothing in it needs to start at zero; calls that overlap on one
 * GPU (concurrently running streams) race on it, so order them on one
 * stream. */
#define SQ_NOALLOC_SCRATCH_BYTES (4u << 20)
sq_status sq_spec_accept_noalloc(const float* draft_logits, const float* target_logits,
                                 const int32_t* draft_tokens, const uint32_t* u24, int32_t b,
                                 int32_t kd, int32_t v, float temperature, int32_t* n_accepted,
                                 int32_t* next_token, float* q_out, float* p_out,
                                 hipStream_t stream);

/* Streaming-read probe (a measurement aid beside the method, not one of its
 * steps): reads `bytes` bytes of src once with 16-byte loads in grid-stride
 * order and nothing else, so that the duration of the call on the stream is a
 * plain read of that many bytes: the measured ceiling that the HBM-bound GEMVs
 * are compared against.
 * src   device memory, 16-B aligned; bytes a multiple of 16, 16 <= bytes <= 2^40
 * sink  [SQ_PROBE_SINK_WORDS] uint32 device out: word j is the XOR of the
 *       32-bit words workgroup j read, so the XOR of all the sink words is the
 *       XOR of every 32-bit word of src.  Must not overlap src. */
#define SQ_PROBE_SINK_WORDS 2048
sq_status sq_probe_stream_read(const void* src, int64_t bytes, uint32_t* sink, hipStream_t stream);

/* Human-readable name of a status code (static storage). */
const char* sq_status_str(sq_status status);

/* SQ_ABI_VERSION of the built library. */
int32_t sq_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SPECQUANT_H */

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
 *   sq_qgemv_w4a16         draft projection y = x . W4'^T, m <= 64 rows
 *   sq_qgemv_w8a16         draft projection y = x . W8'^T, m <= 64 rows
 *   sq_verify_gemm_f16     parent verification y = x . W16^T, m <= 64 rows
 *   sq_spec_accept         LM-head softmax + accept / reject / resample
 *
 * and the decoder layer around those projections, for the Qwen2.5 family the
 * paper evaluates (SS IV), with a key/value cache that the round rolls back by
 * position (SS III-D.4):
 *
 *   sq_embed_block_f16     token embedding of a speculative block
 *   sq_add_rmsnorm_f16     residual add + RMS normalisation
 *   sq_rope_kv_f16         q|k|v bias + rotary embedding + cache write
 *   sq_attention_f16       causal grouped-query attention over the cache
 *   sq_rope_attention_f16  the two above in one call (the chunk kernel rotates
 *                          its own query rows and new cache entries)
 *   sq_silu_mul_f16        SiLU-gated product of the gate|up projection
 *   sq_qgemv_w4a16_rmsnorm, sq_verify_gemm_f16_rmsnorm
 *                          a projection of RMS-normalised rows of h (the norm
 *                          inside the projection's activation staging)
 *   sq_qgemv_w4a16_rmsnorm_silu
 *                          the draft gate|up projection of normalised rows
 *                          with the SiLU-gated product applied to its outputs
 *   sq_qgemv_w4a16_acc, sq_verify_gemm_f16_acc
 *                          a projection added into the residual stream
 *   sq_spec_commit         emitted tokens and restart position of a round
 *
 * and several draft chains per sequence (multi-candidate drafting, SS III-D.2):
 *
 *   sq_spec_accept_multi   accept / correct over c chains (recursive rejection)
 *   sq_kv_adopt_f16        the accepted chain's cache entries to the other chains
 *   sq_spec_commit_multi   emitted tokens and restart position with c chains
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

#define SQ_ABI_VERSION 7

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
 * x [m][k] fp16, 1 <= m <= 64 (m <= 8: the draft GEMV; above, the matrix
 * cores, for passes over many rows such as a prompt's); k % 128 == 0,
 * 128 <= k <= 2^20
 * codes/scales/zeros as produced by sq_quantize_int4_g128 for an [n][k] matrix
 * y [m][n] of y_dtype (SQ_F16 or SQ_F32), 1 <= n <= 2^31 - 1. */
sq_status sq_qgemv_w4a16(const uint16_t* x, int64_t m, int64_t k, const uint8_t* codes,
                         const uint16_t* scales, const uint16_t* zeros, int64_t n, void* y,
                         sq_dtype y_dtype, hipStream_t stream);

/* Draft projection with the FP8 parent (draft generation, SS III-D.2):
 *   y[i][r] = s[r] * sum_c x[i][c] * decode(codes[r][c])
 * x [m][k] fp16, 1 <= m <= 64, k % 16 == 0, 16 <= k <= 2^20;
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
 *   b * (2 kd + 1) * ceil(v / 1024) < 2^24; T finite and >= 0. */
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
 *   T = 0: 8 * (b * (kd + 1) * C) bytes, C = ceil(v / 1024),
 * each term rounded up to a multiple of 256 (the 40 b term excepted); a call
 * that needs more than SQ_NOALLOC_SCRATCH_BYTES returns SQ_ERR_SHAPE and
 * enqueues nothing (e.g. 4 sequences, kd = 8, v = 151936 need 168 KB; 64
 * sequences at kd = 8 need 2.7 MB).  Every call on a GPU shares that GPU's
 * array, and nothing in it needs to start at zero; calls that overlap on one
 * GPU (concurrently running streams) race on it, so order them on one
 * stream. */
#define SQ_NOALLOC_SCRATCH_BYTES (4u << 20)
sq_status sq_spec_accept_noalloc(const float* draft_logits, const float* target_logits,
                                 const int32_t* draft_tokens, const uint32_t* u24, int32_t b,
                                 int32_t kd, int32_t v, float temperature, int32_t* n_accepted,
                                 int32_t* next_token, float* q_out, float* p_out,
                                 hipStream_t stream);

/* ------------------------------------------------------------------------
 * The decoder layer (SS III-D.2 / III-D.3 for the Qwen2.5 family of SS IV;
 * the paper describes neither the layer nor the cache, so these are the
 * textbook operations of that family).  Activations between calls: the
 * residual stream h is fp32 [m][hidden]; projection inputs are fp16; the
 * projection outputs these calls take are fp32 (y_dtype SQ_F32).  Heads are
 * 128 wide.  Rows come in blocks: row r = s * rows_per_seq + j of sequence s
 * sits at position pos_base[s] + pos_offset + j (pos_base a device array, so
 * that a captured graph follows the positions the round moves).
 *
 * Key/value cache of one model and layer (caller-owned, fp16):
 *   keys   k_cache [b][hkv][capacity][128]
 *   values v_cache [b][hkv][128][capacity]   (position-minor)
 * capacity % 64 == 0.  A row attends to the positions 0 .. its own position
 * of its sequence, which must all hold written entries; rolling back a
 * rejected block is moving pos_base (sq_spec_commit): entries past it are
 * rewritten before any later row can attend to them.
 *
 * Device status word (int32, nullable, caller-owned): the kernels OR these
 * bits into it for conditions the host cannot see; it is never cleared. */
#define SQ_DEV_BAD_TOKEN 1 /* a token outside [0, vocab): its row is NaN             */
#define SQ_DEV_BAD_POS 2   /* a position outside [0, len_bound): nothing written for
                              that row, its q / attention output NaN                */
#define SQ_DEV_OVERFLOW 4  /* emitted tokens past out_capacity were not stored      */
#define SQ_DEV_NO_DIST 8   /* a round with n_accepted < 0: that sequence kept its
                              state                                                 */

/* Token embedding of a block: h[s][j] = table[tok(s, j)] widened to fp32, with
 * tok(s, 0) = first[s] and tok(s, 1 + i) = rest[i][s] (rest position-major
 * [kd][b], as draft_tokens of sq_spec_accept): the pending token followed by
 * the drafted ones is the block the parent verifies.
 * table [vocab][hidden] fp16 (16-B aligned), hidden % 8 == 0, hidden <= 16384,
 * 1 <= vocab < 2^31; first [b]; rest [kd][b] (NULL when kd == 0);
 * h [b][kd+1][hidden] f32 out (16-B aligned); 1 <= b, 0 <= kd <= 63. */
sq_status sq_embed_block_f16(const uint16_t* table, int64_t vocab, int64_t hidden, const int32_t* first,
                             const int32_t* rest, int32_t b, int32_t kd, float* h, int32_t* status,
                             hipStream_t stream);

/* Residual add and RMS normalisation (eps inside the root):
 *   h[i] += delta[i] for every row i (when delta is not NULL);
 *   x[r] = f16(h[i] / sqrt(mean_c h[i][c]^2 + eps) * w), i = r * group + group - 1,
 * so group = rows_per_seq normalises only the last row of each sequence (the
 * row whose logits a draft step needs).  Sum of squares in fp32, the
 * reciprocal root in fp64.
 * h [m][hidden] f32 in/out; delta [m][hidden] f32 or NULL; w [hidden] fp16;
 * x [m / group][hidden] fp16 out.  hidden % 8 == 0, 8 <= hidden <= 16384,
 * 1 <= m < 2^31, m % group == 0; eps finite, >= 0.  16-B aligned arrays. */
sq_status sq_add_rmsnorm_f16(float* h, const float* delta, int64_t m, int64_t hidden, const uint16_t* w,
                             float eps, int32_t group, uint16_t* x, hipStream_t stream);

/* Bias, rotary position embedding and cache write of a block of m = b *
 * rows_per_seq rows: with u = qkv[r] + bias (fp32; bias NULL for none) split
 * into hq query heads, hkv key heads and hkv value heads of 128,
 *   q_out[r][h] = f16(rope(u_q[h], pos)),  k_cache[s][g][pos] = f16(rope(u_k[g], pos)),
 *   v_cache[s][g][:][pos] = f16(u_v[g]),
 * rope pairing element t with t + 64 and turning the pair by
 * pos * theta^(-2t/128) (angle, cosine and sine in fp64, the turn in fp32).
 * qkv [m][(hq + 2 hkv) * 128] f32; bias [(hq + 2 hkv) * 128] fp16;
 * pos_base [b]; q_out [m][hq][128] fp16 out; caches as above.
 * 1 <= hkv <= hq, hq % hkv == 0, hq <= 128; 1 <= rows_per_seq <= 64;
 * 64 <= capacity < 2^31, capacity % 64 == 0; 1 <= len_bound <= capacity (an
 * upper bound on every position + 1 of the call); theta > 1 finite.
 * A row at a position outside [0, len_bound) writes nothing to the caches, gets
 * NaN in q_out and sets SQ_DEV_BAD_POS. */
sq_status sq_rope_kv_f16(const float* qkv, const uint16_t* bias, int32_t b, int32_t rows_per_seq, int32_t hq,
                         int32_t hkv, const int32_t* pos_base, int32_t pos_offset, int64_t len_bound,
                         int64_t capacity, double theta, uint16_t* q_out, uint16_t* k_cache, uint16_t* v_cache,
                         int32_t* status, hipStream_t stream);

/* Causal grouped-query attention of a block over the cache: for row r of
 * sequence s at position p and query head h (kv head g = h / (hq / hkv)),
 *   out[r][h] = f16( sum_{t <= p} e_t v_t / sum_{t <= p} e_t ),
 *   e_t = exp(q[r][h] . k_t / sqrt(128) - max),
 * computed per 64-position chunk on the matrix cores (scores in fp32; each
 * weight e_t enters the product with the values as the sum of two fp16 terms,
 * accurate to about 2^-22; fp32 sums) and merged in chunk order.  q [m][hq][128] fp16 (as sq_rope_kv_f16 writes it);
 * out [m][hq][128] fp16 out; limits as sq_rope_kv_f16.  Uses the library
 * workspace (b * hkv * ceil(len_bound / 64) * 16 ceil(rows_per_seq * hq / hkv
 * / 16) * 520 bytes).  A row at a position outside [0, len_bound) gets NaN. */
sq_status sq_attention_f16(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, int32_t b,
                           int32_t rows_per_seq, int32_t hq, int32_t hkv, const int32_t* pos_base,
                           int32_t pos_offset, int64_t len_bound, int64_t capacity, uint16_t* out,
                           hipStream_t stream);

/* sq_rope_kv_f16 followed by sq_attention_f16 of its q_out, in one call: the
 * same out, the same cache entries and the same status, bit for bit.  The
 * attention's chunk kernel rotates the block's query rows and new keys from
 * qkv itself (the arithmetic of sq_rope_kv_f16), uses those new entries
 * where a chunk holds the block's positions instead of reading them back, and
 * writes them to the caches; no q_out is written.  Arguments and limits as the two calls;
 * rows_per_seq <= 16 and rows_per_seq * hq / hkv <= 64 (other blocks return
 * SQ_ERR_UNSUPPORTED and enqueue nothing).  The caches are read and written;
 * out must not overlap them. */
sq_status sq_rope_attention_f16(const float* qkv, const uint16_t* bias, int32_t b, int32_t rows_per_seq, int32_t hq,
                                int32_t hkv, const int32_t* pos_base, int32_t pos_offset, int64_t len_bound,
                                int64_t capacity, double theta, uint16_t* k_cache, uint16_t* v_cache, uint16_t* out,
                                int32_t* status, hipStream_t stream);

/* The projections of a decoder layer with the residual add and the RMS
 * normalisation folded in (one launch instead of two at every norm):
 *
 * sq_qgemv_w4a16_rmsnorm / sq_verify_gemm_f16_rmsnorm: sq_qgemv_w4a16 /
 * sq_verify_gemm_f16 of x = the rows sq_add_rmsnorm_f16(h, w = norm_w, eps,
 * group, delta = NULL) would write, bit for bit the same x and y: row r of x
 * is h row r * group + group - 1 ([m * group][k] f32, 16-B aligned), normalised
 * with the same fp32 sum of squares, fp64 reciprocal root and fp32 products,
 * inside the projection's activation staging.  k <= 4096; m <= 2 (INT4) or
 * m <= 8 (FP16, matrices of the row-block kernel: 2 n k >= 4 MiB and
 * n <= 32768).  Other shapes return SQ_ERR_UNSUPPORTED and enqueue nothing.
 *
 * sq_qgemv_w4a16_acc / sq_verify_gemm_f16_acc: y[i][r] += the projection
 * (y [m][n] f32 in/out; one fp32 add per value, as sq_add_rmsnorm_f16 adds
 * delta), for the output and down projections that feed the residual
 * stream.  m <= 8 (INT4) or the FP16 row-block shapes above; one K slice for
 * INT4 (k * m * 2 <= 64 KiB); other shapes return SQ_ERR_UNSUPPORTED.
 * Other arguments and limits as the plain calls. */
sq_status sq_qgemv_w4a16_rmsnorm(const float* h, int32_t group, const uint16_t* norm_w, float eps, int64_t m,
                                 int64_t k, const uint8_t* codes, const uint16_t* scales, const uint16_t* zeros,
                                 int64_t n, void* y, sq_dtype y_dtype, hipStream_t stream);
sq_status sq_verify_gemm_f16_rmsnorm(const float* h, int32_t group, const uint16_t* norm_w, float eps, int64_t m,
                                     int64_t k, const uint16_t* w16, int64_t n, void* y, sq_dtype y_dtype,
                                     hipStream_t stream);
sq_status sq_qgemv_w4a16_acc(const uint16_t* x, int64_t m, int64_t k, const uint8_t* codes, const uint16_t* scales,
                             const uint16_t* zeros, int64_t n, float* y, hipStream_t stream);

/* sq_qgemv_w4a16_rmsnorm of the fused gate|up matrix (rows [0, n / 2) the
 * gate, [n / 2, n) the up projection) followed by sq_silu_mul_f16 of its fp32
 * outputs, as one call: t[i][c] = f16(g / (1 + exp(-g)) * u) with g, u the
 * fp32 outputs of rows c and n / 2 + c (the same bits as the two calls).
 * t [m][n / 2] fp16 out; n even; m <= 2 with two rows per task of the INT4
 * GEMV (gate|up shapes of at least 2 x 16384 rows, k <= 4096); other shapes
 * return SQ_ERR_UNSUPPORTED and enqueue nothing. */
sq_status sq_qgemv_w4a16_rmsnorm_silu(const float* h, int32_t group, const uint16_t* norm_w, float eps, int64_t m,
                                      int64_t k, const uint8_t* codes, const uint16_t* scales, const uint16_t* zeros,
                                      int64_t n, uint16_t* t, hipStream_t stream);
sq_status sq_verify_gemm_f16_acc(const uint16_t* x, int64_t m, int64_t k, const uint16_t* w16, int64_t n, float* y,
                                 hipStream_t stream);

/* SiLU-gated product of the fused gate|up projection output:
 *   t[i][c] = f16(g / (1 + exp(-g)) * u),  g = gu[i][c], u = gu[i][inter + c]  (fp32).
 * gu [m][2 inter] f32; t [m][inter] fp16 out; 1 <= m, 1 <= inter,
 * m * inter < 2^40. */
sq_status sq_silu_mul_f16(const float* gu, int64_t m, int64_t inter, uint16_t* t, hipStream_t stream);

/* Commit of a round (SS III-D.4: the accepted drafts and the corrected or bonus
 * token are emitted; the rest of the block is removed and decoding restarts
 * from the emitted token).  Per sequence s with n = n_accepted[s] (0 <= n <= kd):
 *   out_tokens[s][out_len[s] + i] = draft_tokens[i][s] (i < n), then next_token[s]
 *     (entries at or past out_capacity are not stored: SQ_DEV_OVERFLOW);
 *   out_len[s] += n + 1;  prev[s] = n > 0 ? draft_tokens[n - 1][s] : pending[s];
 *   pending[s] = next_token[s];  pos_base[s] += n + 1.
 * A sequence with n outside [0, kd] keeps its state (SQ_DEV_NO_DIST).
 * draft_tokens [kd][b] (NULL when kd == 0); pending, prev, pos_base, out_len [b]
 * in/out; out_tokens [b][out_capacity] out, NULL to keep no history (then
 * out_len may be NULL). 1 <= b < 2^24, 0 <= kd <= 64. */
sq_status sq_spec_commit(const int32_t* n_accepted, const int32_t* next_token, const int32_t* draft_tokens,
                         int32_t b, int32_t kd, int32_t* pending, int32_t* prev, int32_t* pos_base,
                         int32_t* out_tokens, int64_t out_capacity, int32_t* out_len, int32_t* status,
                         hipStream_t stream);

/* ------------------------------------------------------------------------
 * Several draft chains per sequence (multi-candidate drafting; SS III-D.2
 * lets a draft variant produce many candidate tokens in one step, and the
 * paper gives no verification rule for them).  Each sequence s drafts c
 * chains of kd tokens; chain j samples its own tokens from the quantized
 * parent (the rows of s are the c chains, as b * c rows of every draft step),
 * so the candidates at any node of the chains' common prefix tree are
 * independent draws from the draft distribution there.  The FP16 parent
 * verifies every chain in one pass (b * c * (kd + 1) rows).  Acceptance walks
 * the tree by recursive rejection sampling, which keeps the parent's
 * distribution exact and is the rule of sq_spec_accept when c = 1. */

/* Multi-candidate acceptance or correction (SS III-D.4 over c chains):
 * at the node reached by the accepted prefix, with q and p the draft's and
 * the parent's distributions there (the lowest alive chain's rows), the alive
 * chains' tokens x are tested in ascending chain order against a residual r
 * (r = p at first): x is accepted iff u * q(x) < r(x); after a rejection
 * r <- max(0, r - q), renormalised.  An accepted token continues with the
 * chains that drafted it; when every alive chain is rejected the emitted
 * token is drawn from r; after kd accepted tokens, the bonus token from p of
 * the last node.  Arithmetic: q, p as in sq_spec_accept (fp64 softmax held in
 * fp32); the first test u q(x) < p(x) in fp64; its residual
 * R = rint(max(0, p - q) 2^60) with Z = sum R (or R = rint(p 2^60) when Z = 0);
 * later tests u q(x) Z < R(x) and later residuals R <- max(0, R - floor(q Z))
 * in exact integer arithmetic (same fallback); the draw takes the smallest y
 * whose running sum of R exceeds floor(u24 Z / 2^24).
 * T = 0 (greedy): the argmax of the node's parent row (smallest index on
 * ties) is accepted when an alive chain drafted it; else it is emitted.
 * draft_logits  [kd][b][c][v] f32 (draft step d for every chain)
 * target_logits [b][c][kd+1][v] f32 (chain j's verification rows)
 * draft_tokens  [kd][b][c] int32
 * u24           [b][c kd + 1] uint32: u24[s][d c + j] tests chain j at depth d,
 *               u24[s][c kd] drives the final draw (NULL allowed at T = 0)
 * n_accepted, next_token [b] out; chain [b] out: the lowest chain whose first
 *   n tokens are the accepted ones (its draft_tokens[0..n)[s] and next_token
 *   are the emitted tokens).  A sequence with a row without a distribution
 *   (T > 0: any of its rows; T = 0: any target row) gets -1 in all three.
 * q_out [kd][b][c][v], p_out [b][c][kd+1][v]: optional fp32 copies, T > 0 only.
 * Limits: 1 <= b <= 65535, 1 <= c <= 64, 0 <= kd <= 64, 1 <= v <= 2^26,
 *   b c (2 kd + 1) ceil(v / 1024) < 2^24; T finite and >= 0.  Uses the library
 *   workspace (row statistics, the fp32 rows unless q_out / p_out are given,
 *   and one int64 row per sequence). */
sq_status sq_spec_accept_multi(const float* draft_logits, const float* target_logits, const int32_t* draft_tokens,
                               const uint32_t* u24, int32_t b, int32_t c, int32_t kd, int32_t v, float temperature,
                               int32_t* n_accepted, int32_t* next_token, int32_t* chain, float* q_out, float* p_out,
                               hipStream_t stream);

/* The accepted chain's cache entries to the other chains of its sequence
 * (before sq_spec_commit_multi moves the positions): for every layer, kv head
 * and sequence s with 0 <= chain[s] < c and n_accepted[s] >= 0, the entries of
 * row s c + chain[s] at positions pos + lo_offset .. pos + n_accepted[s] +
 * hi_offset (pos = pos_base[s c + chain[s]]; clipped to [0, capacity)) are
 * copied to rows s c + j, j != chain[s].  The parent's
 * cache takes lo_offset = hi_offset = 0 (the pending token and the accepted
 * drafts), the draft's lo_offset = hi_offset = -1.
 * k_cache [layers][b c][hkv][capacity][128] fp16, v_cache
 * [layers][b c][hkv][128][capacity] fp16 (the layout of sq_rope_kv_f16, layers
 * contiguous); chain, n_accepted [b]; pos_base [b c].  1 <= layers, b c,
 * hkv <= 65535; c <= 64; capacity as for sq_rope_kv_f16; |offsets| <= 64. */
sq_status sq_kv_adopt_f16(uint16_t* k_cache, uint16_t* v_cache, int32_t layers, int32_t b, int32_t c, int32_t hkv,
                          int64_t capacity, const int32_t* chain, const int32_t* n_accepted, const int32_t* pos_base,
                          int32_t lo_offset, int32_t hi_offset, hipStream_t stream);

/* The commit of sq_spec_commit for c chains per sequence: with n =
 * n_accepted[s] and a = chain[s], the emitted tokens draft_tokens[i][s][a]
 * (i < n) and next_token[s] are appended to out_tokens[s]; every chain j of s
 * gets pending[s c + j] = next_token[s], prev[s c + j] = the last emitted
 * draft (pending[s c + a] when n = 0) and pos_base[s c + j] = pos_base[s c + a]
 * + n + 1.  A sequence with n outside [0, kd] or a outside [0, c) keeps its
 * state (SQ_DEV_NO_DIST).  pending, prev, pos_base [b c]; other arrays as in
 * sq_spec_commit.  1 <= b < 2^24, 1 <= c <= 64, 0 <= kd <= 64. */
sq_status sq_spec_commit_multi(const int32_t* n_accepted, const int32_t* next_token, const int32_t* chain,
                               const int32_t* draft_tokens, int32_t b, int32_t c, int32_t kd, int32_t* pending,
                               int32_t* prev, int32_t* pos_base, int32_t* out_tokens, int64_t out_capacity,
                               int32_t* out_len, int32_t* status, hipStream_t stream);

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

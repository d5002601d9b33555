// Host-side launchers of the SpecQuant kernels; argument validation happens
// in the C-ABI layer before any of these is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sq {

// Library-owned device workspace of at least `bytes` bytes on the current
// device, in *out.  It only grows; a buffer it outgrows stays allocated until
// the process ends (graphs captured earlier may still use it).  Growing is
// refused while `stream` is being captured (hipErrorStreamCaptureUnsupported);
// hipErrorOutOfMemory when the allocation fails.
hipError_t workspace(size_t bytes, hipStream_t stream, void** out);

// At least `count` int32 counters on the current device that are zero
// between launches, in *out: zeroed on `stream` when allocated (same growth
// rules as the workspace); every kernel that counts on them returns them to
// zero before it ends.
hipError_t zeroed_counters(size_t count, hipStream_t stream, int32_t** out);

// Compute units of the current device (cached per device).
int cu_count();

// Resident workgroups per CU of `kernel` with `threads` threads and `lds`
// bytes of dynamic LDS (cached; at least 1).
int resident_blocks(const void* kernel, int threads, size_t lds);

hipError_t launch_quantize_int4(const uint16_t* w, int64_t n, int64_t k, uint8_t* codes, uint16_t* scales,
                                uint16_t* zeros, int32_t* flag, hipStream_t stream);
hipError_t launch_quantize_fp8(const uint16_t* w, int64_t n, int64_t k, uint8_t* codes, float* scales,
                               int32_t* flag, hipStream_t stream);

// Input rows of a projection taken as f16(rmsnorm(h row)) with weights w:
// staged row m is h row m * group + group - 1 ([m * group][k] fp32), normalised
// inside the projection's activation staging with the arithmetic of
// launch_add_rmsnorm (the same bits).
struct NormSrc {
  const float* h;
  const uint16_t* w;
  float eps;
  int group;
};

// nrm: activations from normalised rows instead of x (x unused); accum: y is
// fp32 and the projection is added into it (y += x . W'^T); silu: rows
// [0, n / 2) are gates and [n / 2, n) ups, and y is t [m][n / 2] fp16 =
// f16(silu(gate) * up).  Each returns hipErrorNotSupported, enqueuing nothing,
// for shapes whose kernel lacks it.
hipError_t launch_gemv_w4(const uint16_t* x, int m, int64_t k, const uint8_t* codes, const uint16_t* scales,
                          const uint16_t* zeros, int64_t n, void* y, bool f16_out, hipStream_t stream,
                          const NormSrc* nrm = nullptr, bool accum = false, bool silu = false);
hipError_t launch_gemv_w8(const uint16_t* x, int m, int64_t k, const uint8_t* codes, const float* scales,
                          int64_t n, void* y, bool f16_out, hipStream_t stream);
hipError_t launch_gemm_f16(const uint16_t* x, int m, int64_t k, const uint16_t* w, int64_t n, void* y,
                           bool f16_out, hipStream_t stream);
// Verification over row blocks on the vector ALUs, 1 <= m <= 8; returns
// hipErrorNotSupported (nothing enqueued) for shapes it does not take.
hipError_t launch_gemm_rows_f16(const uint16_t* x, int m, int64_t k, const uint16_t* w, int64_t n, void* y,
                                bool f16_out, hipStream_t stream, const NormSrc* nrm = nullptr, bool accum = false);

// The matrix-core streaming kernels (one implementation for the three weight
// kinds; m <= 8 for INT4 / FP8, m <= 64 for FP16).
hipError_t launch_linear_w4(const uint16_t* x, int m, int64_t k, const uint8_t* codes, const uint16_t* scales,
                            const uint16_t* zeros, int64_t n, void* y, bool f16_out, hipStream_t stream);
hipError_t launch_linear_w8(const uint16_t* x, int m, int64_t k, const uint8_t* codes, const float* scales,
                            int64_t n, void* y, bool f16_out, hipStream_t stream);
hipError_t launch_linear_f16(const uint16_t* x, int m, int64_t k, const uint16_t* w, int64_t n, void* y,
                             bool f16_out, hipStream_t stream);

// Sum of S split-K partials [S][mn] fp32 into y[mn] (fixed order s = 0..S-1).
hipError_t launch_splitk_reduce(const float* partial, int splits, int64_t mn, void* y, bool f16_out,
                                hipStream_t stream);

// The streaming-read probe: `blocks` workgroups read bytes / 16 cells of src
// and write one XOR word each to sink[0 .. blocks).
hipError_t launch_stream_read(const void* src, int64_t bytes, uint32_t* sink, int blocks, hipStream_t stream);

hipError_t launch_spec_accept(const float* draft, const float* target, const int32_t* tokens, const uint32_t* u24,
                              int b, int kd, int v, float temperature, int32_t* n_accepted, int32_t* next_token,
                              float* q_out, float* p_out, hipStream_t stream);

// Logits per chunk of a vocabulary row in the accept kernels (the chunk
// partials of the softmax statistics and of the draw weights).
constexpr int kAcceptChunk = 1024;

// Bytes of scratch one accept call needs (workspace or static array).
size_t spec_accept_scratch_bytes(int b, int kd, int v, float temperature);

// Size of the static scratch array of the allocation-free accept call.
constexpr size_t kNoAllocScratchBytes = size_t(4) << 20;

// The accept call on the static scratch array of the current device (no
// allocation); hipErrorInvalidValue when the call needs more than
// kNoAllocScratchBytes (the C ABI checks that first).
hipError_t launch_spec_accept_noalloc(const float* draft, const float* target, const int32_t* tokens,
                                      const uint32_t* u24, int b, int kd, int v, float temperature,
                                      int32_t* n_accepted, int32_t* next_token, float* q_out, float* p_out,
                                      hipStream_t stream);

// The decoder layer around the projections (decoder.hip).
hipError_t launch_embed_block(const uint16_t* table, int64_t vocab, int hidden, const int32_t* first,
                              const int32_t* rest, int b, int kd, float* h, int32_t* status, hipStream_t stream);
hipError_t launch_add_rmsnorm(float* h, const float* delta, int64_t m, int hidden, const uint16_t* w, float eps,
                              int group, uint16_t* x, hipStream_t stream);
hipError_t launch_rope_kv(const float* qkv, const uint16_t* bias, int m, int hq, int hkv, int rps,
                          const int32_t* pos_base, int pos_offset, int64_t len_bound, int64_t capacity, double theta,
                          uint16_t* q_out, uint16_t* kc, uint16_t* vc, int32_t* status, hipStream_t stream);
// Workspace bytes of one attention call (chunk partials).
size_t attention_workspace_bytes(int b, int hq, int hkv, int rps, int64_t len_bound);
hipError_t launch_attention(const uint16_t* q, const uint16_t* kc, const uint16_t* vc, int b, int rps, int hq,
                            int hkv, int64_t capacity, const int32_t* pos_base, int pos_offset, int64_t len_bound,
                            uint16_t* out, hipStream_t stream);
// launch_rope_kv (without q_out) + launch_attention in one chunk kernel and the
// merge, the same bits; hipErrorNotSupported (nothing enqueued) for blocks of
// more than 16 rows per sequence or 64 query rows per kv head.
hipError_t launch_rope_attention(const float* qkv, const uint16_t* bias, int b, int rps, int hq, int hkv,
                                 int64_t capacity, const int32_t* pos_base, int pos_offset, int64_t len_bound,
                                 double theta, uint16_t* kc, uint16_t* vc, uint16_t* out, int32_t* status,
                                 hipStream_t stream);
hipError_t launch_silu_mul(const float* gu, int64_t m, int64_t inter, uint16_t* t, hipStream_t stream);
hipError_t launch_spec_commit(const int32_t* n_accepted, const int32_t* next_token, const int32_t* drafts, int b,
                              int kd, int32_t* pending, int32_t* prev, int32_t* pos_base, int32_t* out_tokens,
                              int64_t out_capacity, int32_t* out_len, int32_t* status, hipStream_t stream);

// Multi-candidate acceptance over c draft chains per sequence (accept.hip).
size_t spec_accept_multi_scratch_bytes(int b, int c, int kd, int v, float temperature, bool have_q, bool have_p);
hipError_t launch_spec_accept_multi(const float* draft, const float* target, const int32_t* tokens,
                                    const uint32_t* u24, int b, int c, int kd, int v, float temperature,
                                    int32_t* n_accepted, int32_t* next_token, int32_t* chain, float* q_out,
                                    float* p_out, hipStream_t stream);
// Copy the accepted chain's cache entries to the other chains of its sequence;
// the commit of a round with several chains (decoder.hip).
hipError_t launch_kv_adopt(uint16_t* kc, uint16_t* vc, int layers, int b, int c, int hkv, int64_t capacity,
                           const int32_t* chain, const int32_t* n_accepted, const int32_t* pos_base, int lo_offset,
                           int hi_offset, hipStream_t stream);
hipError_t launch_spec_commit_multi(const int32_t* n_accepted, const int32_t* next_token, const int32_t* chain,
                                    const int32_t* drafts, int b, int c, int kd, int32_t* pending, int32_t* prev,
                                    int32_t* pos_base, int32_t* out_tokens, int64_t out_capacity, int32_t* out_len,
                                    int32_t* status, hipStream_t stream);

}  // namespace sq

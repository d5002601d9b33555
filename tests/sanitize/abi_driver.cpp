// Drives the C-ABI validation of every entry point (csrc/abi.cpp, linked with
// abi_stubs.cpp) through invalid and valid arguments, including sizes at the
// limits, under AddressSanitizer and UndefinedBehaviorSanitizer.  Addresses
// are fake and never dereferenced (the stub launchers only record calls).
#include <stdint.h>
#include <stdio.h>

#include <cmath>

#include "specquant.h"

namespace stub {
extern int calls;
}

static int failures = 0;
#define EXPECT(expr, want)                                                          \
  do {                                                                              \
    const int got_ = (int)(expr);                                                   \
    if (got_ != (int)(want)) {                                                      \
      printf("FAIL line %d: %s = %d, want %d\n", __LINE__, #expr, got_, (int)(want)); \
      ++failures;                                                                   \
    }                                                                               \
  } while (0)

template <class T>
static T* at(uint64_t a) {
  return reinterpret_cast<T*>(a);
}

int main() {
  const uint64_t A = 0x7F0000000000ull, B = A + (1ull << 32), C = A + (2ull << 32), D = A + (3ull << 32),
                 E = A + (4ull << 32);
  // far-apart fake addresses for limit-sized buffers (up to 2^42 bytes each)
  const uint64_t FA = 0x100000000000ull, FB = FA + (1ull << 42), FC = FA + (2ull << 42), FD = FA + (3ull << 42),
                 FE = FA + (4ull << 42);
  hipStream_t s = nullptr;
  // quantizers
  EXPECT(sq_quantize_int4_g128(nullptr, 4, 128, at<uint8_t>(B), at<uint16_t>(C), at<uint16_t>(D), nullptr, s),
         SQ_ERR_NULL);
  EXPECT(sq_quantize_int4_g128(at<uint16_t>(A), 4, 100, at<uint8_t>(B), at<uint16_t>(C), at<uint16_t>(D), nullptr, s),
         SQ_ERR_SHAPE);
  EXPECT(sq_quantize_int4_g128(at<uint16_t>(A), 0x7FFFFFFF, 1 << 20, at<uint8_t>(B), at<uint16_t>(C), at<uint16_t>(D),
                               nullptr, s),
         SQ_ERR_ALIAS);  // 2^31 x 2^20 weights: the ranges overlap, the size arithmetic must not overflow
  EXPECT(sq_quantize_int4_g128(at<uint16_t>(A), 4, 128, at<uint8_t>(B), at<uint16_t>(C), at<uint16_t>(D), nullptr, s),
         SQ_OK);
  EXPECT(sq_quantize_fp8_e4m3(at<uint16_t>(A), 4, 24, at<uint8_t>(B), at<float>(C), nullptr, s), SQ_ERR_SHAPE);
  EXPECT(sq_quantize_fp8_e4m3(at<uint16_t>(A), 4, 32, at<uint8_t>(B), at<float>(C + 2), nullptr, s), SQ_ERR_ALIGN);
  EXPECT(sq_quantize_fp8_e4m3(at<uint16_t>(A), 4, 32, at<uint8_t>(B), at<float>(C), nullptr, s), SQ_OK);
  // GEMVs and the verify GEMM
  EXPECT(sq_qgemv_w4a16(at<uint16_t>(A), 65, 256, at<uint8_t>(B), at<uint16_t>(C), at<uint16_t>(D), 10, at<void>(E),
                        SQ_F32, s),
         SQ_ERR_SHAPE);
  EXPECT(sq_qgemv_w4a16(at<uint16_t>(A), 1, 256, at<uint8_t>(B), at<uint16_t>(C), at<uint16_t>(D), 10, at<void>(E),
                        (sq_dtype)7, s),
         SQ_ERR_UNSUPPORTED);
  EXPECT(sq_qgemv_w4a16(at<uint16_t>(A), 8, 1 << 20, at<uint8_t>(B), at<uint16_t>(C), at<uint16_t>(D), 0x7FFFFFFF,
                        at<void>(E), SQ_F32, s),
         SQ_ERR_ALIAS);
  EXPECT(sq_qgemv_w4a16(at<uint16_t>(A), 1, 256, at<uint8_t>(B), at<uint16_t>(C), at<uint16_t>(D), 10, at<void>(E),
                        SQ_F16, s),
         SQ_OK);
  EXPECT(sq_qgemv_w8a16(at<uint16_t>(A), 4, 4096, at<uint8_t>(B), at<float>(C), 16384, at<void>(E), SQ_F16, s),
         SQ_OK);
  EXPECT(sq_verify_gemm_f16(at<uint16_t>(A), 65, 64, at<uint16_t>(B), 10, at<void>(E), SQ_F32, s), SQ_ERR_SHAPE);
  EXPECT(sq_verify_gemm_f16(at<uint16_t>(A), 5, 3584, at<uint16_t>(B), 4608, at<void>(E), SQ_F16, s), SQ_OK);
  EXPECT(sq_verify_gemm_f16(at<uint16_t>(A), 36, 3584, at<uint16_t>(B), 151936, at<void>(E), SQ_F32, s), SQ_OK);
  // the decoder's fused projections
  EXPECT(sq_qgemv_w4a16_rmsnorm(at<float>(A), 1, at<uint16_t>(C), 1e-6f, 1, 3584, at<uint8_t>(B), at<uint16_t>(D),
                                at<uint16_t>(D + (1ull << 24)), 4608, at<void>(E), SQ_F32, s),
         SQ_OK);
  EXPECT(sq_qgemv_w4a16_rmsnorm(at<float>(A), 2, at<uint16_t>(C), std::nanf(""), 1, 3584, at<uint8_t>(B), at<uint16_t>(D),
                                at<uint16_t>(D + (1ull << 24)), 4608, at<void>(E), SQ_F32, s),
         SQ_ERR_NONFINITE);
  EXPECT(sq_verify_gemm_f16_rmsnorm(at<float>(A), 1, at<uint16_t>(C), 1e-6f, 5, 3584, at<uint16_t>(B), 4608,
                                    at<void>(E), SQ_F32, s),
         SQ_OK);
  EXPECT(sq_verify_gemm_f16_rmsnorm(at<float>(A), 1, at<uint16_t>(C), 1e-6f, 5, 3584, at<uint16_t>(B), 37888,
                                    at<void>(E), SQ_F32, s),
         SQ_ERR_UNSUPPORTED);
  EXPECT(sq_qgemv_w4a16_rmsnorm_silu(at<float>(A), 1, at<uint16_t>(C), 1e-6f, 1, 3584, at<uint8_t>(B),
                                     at<uint16_t>(D), at<uint16_t>(D + (1ull << 24)), 37888, at<uint16_t>(E), s),
         SQ_OK);
  EXPECT(sq_qgemv_w4a16_rmsnorm_silu(at<float>(A), 1, at<uint16_t>(C), 1e-6f, 1, 3584, at<uint8_t>(B),
                                     at<uint16_t>(D), at<uint16_t>(D + (1ull << 24)), 37887, at<uint16_t>(E), s),
         SQ_ERR_SHAPE);
  EXPECT(sq_qgemv_w4a16_rmsnorm_silu(at<float>(A), 1, at<uint16_t>(C), 1e-6f, 3, 3584, at<uint8_t>(B),
                                     at<uint16_t>(D), at<uint16_t>(D + (1ull << 24)), 37888, at<uint16_t>(E), s),
         SQ_ERR_UNSUPPORTED);
  EXPECT(sq_qgemv_w4a16_acc(at<uint16_t>(A), 1, 18944, at<uint8_t>(B), at<uint16_t>(C), at<uint16_t>(D), 3584,
                            at<float>(E), s),
         SQ_OK);
  EXPECT(sq_verify_gemm_f16_acc(at<uint16_t>(A), 5, 18944, at<uint16_t>(B), 3584, at<float>(E), s), SQ_OK);
  EXPECT(sq_verify_gemm_f16_acc(at<uint16_t>(A), 5, 18944, at<uint16_t>(B), 3584, at<float>(E + 2), s),
         SQ_ERR_ALIGN);
  // bias + rotation + attention in one call
  EXPECT(sq_rope_attention_f16(at<float>(A), at<uint16_t>(B), 1, 5, 28, 4, at<int32_t>(C), 0, 2048, 2048, 1e6,
                               at<uint16_t>(D), at<uint16_t>(D + (1ull << 24)), at<uint16_t>(E), nullptr, s),
         SQ_OK);
  EXPECT(sq_rope_attention_f16(at<float>(A), at<uint16_t>(B), 1, 10, 28, 4, at<int32_t>(C), 0, 2048, 2048, 1e6,
                               at<uint16_t>(D), at<uint16_t>(D + (1ull << 24)), at<uint16_t>(E), nullptr, s),
         SQ_ERR_UNSUPPORTED);
  EXPECT(sq_rope_attention_f16(at<float>(A), at<uint16_t>(B), 1, 5, 28, 4, at<int32_t>(C), 0, 2048, 2048, 1e6,
                               at<uint16_t>(D), at<uint16_t>(D + 4096), at<uint16_t>(E), nullptr, s),
         SQ_ERR_ALIAS);
  // accept, and its allocation-free twin
  float nan = std::nanf("");
  EXPECT(sq_spec_accept(at<float>(A), at<float>(B), at<int32_t>(C), at<uint32_t>(D), 1, 4, 100, nan, at<int32_t>(E),
                        at<int32_t>(E + 64), nullptr, nullptr, s),
         SQ_ERR_NONFINITE);
  EXPECT(sq_spec_accept(nullptr, at<float>(B), nullptr, at<uint32_t>(D), (1 << 24) - 1, 0, 1, 1.0f, at<int32_t>(E),
                        at<int32_t>(E + (1 << 26)), nullptr, nullptr, s),
         SQ_OK);
  EXPECT(sq_spec_accept(at<float>(A), at<float>(B), at<int32_t>(C), at<uint32_t>(D), 1, 64, 1 << 26, 1.0f,
                        at<int32_t>(E), at<int32_t>(E + 64), nullptr, nullptr, s),
         SQ_ERR_ALIAS);  // 65 rows of 2^26 logits reach past the next fake buffer
  EXPECT(sq_spec_accept(at<float>(FA), at<float>(FB), at<int32_t>(FC), at<uint32_t>(FD), 1, 64, 1 << 26, 1.0f,
                        at<int32_t>(FE), at<int32_t>(FE + 64), at<float>(FE + (1ull << 40)),
                        at<float>(FE + (2ull << 40)), s),
         SQ_OK);
  EXPECT(sq_spec_accept_noalloc(at<float>(A), at<float>(B), at<int32_t>(C), at<uint32_t>(D), 100, 8, 151936, 1.0f,
                                at<int32_t>(E), at<int32_t>(E + 4096), nullptr, nullptr, s),
         SQ_ERR_SHAPE);
  EXPECT(sq_spec_accept_noalloc(at<float>(A), at<float>(B), at<int32_t>(C), at<uint32_t>(D), 4, 8, 151936, 1.0f,
                                at<int32_t>(E), at<int32_t>(E + 4096), nullptr, nullptr, s),
         SQ_OK);
  EXPECT(sq_probe_stream_read(at<void>(A), 1ll << 40, at<uint32_t>(E), s), SQ_ERR_ALIAS);
  EXPECT(sq_probe_stream_read(at<void>(FA), 1ll << 40, at<uint32_t>(FB), s), SQ_OK);
  EXPECT(sq_qgemv_w4a16(at<uint16_t>(FA), 8, 1 << 20, at<uint8_t>(FB), at<uint16_t>(FC), at<uint16_t>(FD), 1 << 22,
                        at<void>(FE), SQ_F32, s),
         SQ_OK);  // 2^22 rows of 2^20 k: 2 TiB of codes, sizes past 32 bits
  for (int st = 0; st <= 9; ++st) (void)sq_status_str((sq_status)st);
  EXPECT(sq_abi_version(), SQ_ABI_VERSION);
  if (stub::calls < 10) {
    printf("FAIL: only %d launcher calls\n", stub::calls);
    ++failures;
  }
  printf(failures ? "FAILED %d\n" : "ABI OK\n", failures);
  return failures ? 1 : 0;
}

// Host-only stand-ins for the HIP runtime calls and the kernel launchers that
// the C-ABI layer (csrc/abi.cpp) calls, so that its validation and dispatch
// code can be built with AddressSanitizer and UndefinedBehaviorSanitizer and
// run without a GPU.  Every launcher records its call and returns success;
// nothing touches the pointers it is given.
#include <stdint.h>
#include <string.h>

#include "sq_internal.hpp"

namespace stub {
int calls = 0;
char last[64] = "";
void record(const char* what) {
  ++calls;
  strncpy(last, what, sizeof(last) - 1);
}
}  // namespace stub

extern "C" {
hipError_t hipGetLastError(void) { return hipSuccess; }
hipError_t hipGetDevice(int* d) {
  *d = 0;
  return hipSuccess;
}
hipError_t hipDeviceGetAttribute(int* v, hipDeviceAttribute_t, int) {
  *v = 256;
  return hipSuccess;
}
hipError_t hipStreamIsCapturing(hipStream_t, hipStreamCaptureStatus* s) {
  *s = hipStreamCaptureStatusNone;
  return hipSuccess;
}
static char g_pool[1 << 20];
hipError_t hipMalloc(void** p, size_t bytes) {
  *p = bytes <= sizeof(g_pool) ? g_pool : nullptr;
  return *p ? hipSuccess : hipErrorOutOfMemory;
}
hipError_t hipMemsetAsync(void* p, int v, size_t bytes, hipStream_t) {
  memset(p, v, bytes);
  return hipSuccess;
}
hipError_t hipFree(void*) { return hipSuccess; }
hipError_t hipOccupancyMaxActiveBlocksPerMultiprocessor(int* b, const void*, int, size_t) {
  *b = 1;
  return hipSuccess;
}
}

namespace sq {
#define STUB(name, ...)                 \
  hipError_t name(__VA_ARGS__) {        \
    stub::record(#name);                \
    return hipSuccess;                  \
  }
STUB(launch_quantize_int4, const uint16_t*, int64_t, int64_t, uint8_t*, uint16_t*, uint16_t*, int32_t*, hipStream_t)
STUB(launch_quantize_fp8, const uint16_t*, int64_t, int64_t, uint8_t*, float*, int32_t*, hipStream_t)
STUB(launch_gemv_w4, const uint16_t*, int, int64_t, const uint8_t*, const uint16_t*, const uint16_t*, int64_t, void*,
     bool, hipStream_t, const NormSrc*, bool, bool)
STUB(launch_gemv_w8, const uint16_t*, int, int64_t, const uint8_t*, const float*, int64_t, void*, bool, hipStream_t)
STUB(launch_gemm_f16, const uint16_t*, int, int64_t, const uint16_t*, int64_t, void*, bool, hipStream_t)
STUB(launch_gemm_rows_f16, const uint16_t*, int, int64_t, const uint16_t*, int64_t, void*, bool, hipStream_t,
     const NormSrc*, bool)
STUB(launch_linear_w4, const uint16_t*, int, int64_t, const uint8_t*, const uint16_t*, const uint16_t*, int64_t, void*,
     bool, hipStream_t)
STUB(launch_linear_w8, const uint16_t*, int, int64_t, const uint8_t*, const float*, int64_t, void*, bool, hipStream_t)
STUB(launch_linear_f16, const uint16_t*, int, int64_t, const uint16_t*, int64_t, void*, bool, hipStream_t)
STUB(launch_splitk_reduce, const float*, int, int64_t, void*, bool, hipStream_t)
STUB(launch_stream_read, const void*, int64_t, uint32_t*, int, hipStream_t)
STUB(launch_spec_accept, const float*, const float*, const int32_t*, const uint32_t*, int, int, int, float, int32_t*,
     int32_t*, float*, float*, hipStream_t)
STUB(launch_spec_accept_noalloc, const float*, const float*, const int32_t*, const uint32_t*, int, int, int, float,
     int32_t*, int32_t*, float*, float*, hipStream_t)
STUB(launch_embed_block, const uint16_t*, int64_t, int, const int32_t*, const int32_t*, int, int, float*, int32_t*,
     hipStream_t)
STUB(launch_add_rmsnorm, float*, const float*, int64_t, int, const uint16_t*, float, int, uint16_t*, hipStream_t)
STUB(launch_rope_kv, const float*, const uint16_t*, int, int, int, int, const int32_t*, int, int64_t, int64_t, double,
     uint16_t*, uint16_t*, uint16_t*, int32_t*, hipStream_t)
STUB(launch_attention, const uint16_t*, const uint16_t*, const uint16_t*, int, int, int, int, int64_t, const int32_t*,
     int, int64_t, uint16_t*, hipStream_t)
STUB(launch_rope_attention, const float*, const uint16_t*, int, int, int, int, int64_t, const int32_t*, int, int64_t,
     double, uint16_t*, uint16_t*, uint16_t*, int32_t*, hipStream_t)
STUB(launch_silu_mul, const float*, int64_t, int64_t, uint16_t*, hipStream_t)
STUB(launch_spec_commit, const int32_t*, const int32_t*, const int32_t*, int, int, int32_t*, int32_t*, int32_t*,
     int32_t*, int64_t, int32_t*, int32_t*, hipStream_t)
STUB(launch_spec_accept_multi, const float*, const float*, const int32_t*, const uint32_t*, int, int, int, int, float,
     int32_t*, int32_t*, int32_t*, float*, float*, hipStream_t)
STUB(launch_kv_adopt, uint16_t*, uint16_t*, int, int, int, int, int64_t, const int32_t*, const int32_t*, const int32_t*,
     int, int, hipStream_t)
STUB(launch_spec_commit_multi, const int32_t*, const int32_t*, const int32_t*, const int32_t*, int, int, int, int32_t*,
     int32_t*, int32_t*, int32_t*, int64_t, int32_t*, int32_t*, hipStream_t)
size_t spec_accept_scratch_bytes(int b, int kd, int v, float) {
  const size_t c = (size_t)(v + kAcceptChunk - 1) / kAcceptChunk;
  return 16 * (size_t)b * (2 * kd + 1) * c + 16 * (size_t)b * c + 40 * (size_t)b;
}
}  // namespace sq

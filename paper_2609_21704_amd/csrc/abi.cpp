// C ABI of the SpecQuant hot path: host-side argument validation, the
// library-owned device workspace, and dispatch to the HIP kernels.
#include <math.h>
#include <stddef.h>
#include <stdint.h>

#include <map>
#include <mutex>
#include <tuple>
#include <vector>

#include "sq_internal.hpp"
#include "specquant.h"

static_assert(sq::kNoAllocScratchBytes == SQ_NOALLOC_SCRATCH_BYTES, "one size for the static scratch array");

// Large matrices stream through the matrix-core kernel; small ones (where
// its fixed cost of staging activations and combining chunks, about 4 us more
// than the others', dominates) and m > 16 use the vector-ALU GEMV and the
// tile-per-workgroup GEMM, which measured faster there.  Thresholds in weight
// bytes.
constexpr int64_t kLinearMinBytesF16 = int64_t(28) << 20;  // between 3584^2 and 4608 x 3584 (7B o, q|k|v)
constexpr int64_t kLinearMinBytesF16Wide = int64_t(4) << 20;  // m > 16: between 1152 x 896 and 896 x 4864
constexpr int64_t kLinearMinBytesW8 = int64_t(64) << 20;
constexpr int64_t kRowsMinBytesF16 = int64_t(4) << 20;  // 0.5B gate|up 896 x 4864 takes it, 896 x 896 not
constexpr int64_t kRowsMaxRowsF16 = 32768;              // 14B gate|up 27648 x 5120 takes it, 7B 37888 x 3584 not

namespace sq {
namespace {

constexpr int kMaxDevices = 64;

// A device buffer that only grows.  A buffer it outgrows is retired, never
// freed: a graph captured while that buffer was current keeps its address and
// may be replayed at any later time, and kernels enqueued earlier may still be
// using it.  Retired buffers live until the process ends (at most as many
// bytes again as the current one, since each growth at least doubles).
struct Pool {
  void* ptr = nullptr;
  size_t bytes = 0;
  std::vector<void*> retired;
};

std::mutex g_ws_mutex;
Pool g_ws[kMaxDevices];
Pool g_cnt[kMaxDevices];
int g_cus[kMaxDevices];

// Current buffer of `pool` with at least `bytes` bytes.  A new buffer is
// allocated only outside stream capture (allocating would invalidate the
// capture); it is zeroed on `stream` when `zero` is set.
hipError_t pool_get(Pool& pool, size_t bytes, size_t grain, bool zero, hipStream_t stream, void** out) {
  *out = nullptr;
  if (pool.ptr && pool.bytes >= bytes) {
    *out = pool.ptr;
    return hipSuccess;
  }
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &cs) != hipSuccess) {
    (void)hipGetLastError();
    return hipErrorInvalidValue;
  }
  if (cs != hipStreamCaptureStatusNone) return hipErrorStreamCaptureUnsupported;
  size_t want = bytes > 2 * pool.bytes ? bytes : 2 * pool.bytes;
  want = (want + grain - 1) / grain * grain;
  void* p = nullptr;
  if (hipMalloc(&p, want) != hipSuccess) {
    (void)hipGetLastError();
    return hipErrorOutOfMemory;
  }
  if (zero && hipMemsetAsync(p, 0, want, stream) != hipSuccess) {
    (void)hipGetLastError();
    (void)hipFree(p);  // never handed out
    return hipErrorOutOfMemory;
  }
  if (pool.ptr) pool.retired.push_back(pool.ptr);
  pool.ptr = p;
  pool.bytes = want;
  *out = p;
  return hipSuccess;
}

}  // namespace

int resident_blocks(const void* kernel, int threads, size_t lds) {
  static std::mutex mu;
  static std::map<std::tuple<const void*, int, size_t>, int> cache;
  const auto key = std::make_tuple(kernel, threads, lds);
  std::lock_guard<std::mutex> lock(mu);
  auto it = cache.find(key);
  if (it != cache.end()) return it->second;
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, kernel, threads, lds) != hipSuccess || blocks < 1) {
    (void)hipGetLastError();
    blocks = 1;
  }
  cache[key] = blocks;
  return blocks;
}

int cu_count() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
  std::lock_guard<std::mutex> lock(g_ws_mutex);
  if (g_cus[dev] <= 0) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) cus = 256;
    g_cus[dev] = cus;
  }
  return g_cus[dev];
}

hipError_t workspace(size_t bytes, hipStream_t stream, void** out) {
  *out = nullptr;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_ws_mutex);
  return pool_get(g_ws[dev], bytes, size_t(2) << 20, false, stream, out);
}

hipError_t zeroed_counters(size_t count, hipStream_t stream, int32_t** out) {
  *out = nullptr;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_ws_mutex);
  void* p = nullptr;
  const hipError_t e = pool_get(g_cnt[dev], count * sizeof(int32_t), size_t(64) << 10, true, stream, &p);
  *out = static_cast<int32_t*>(p);
  return e;
}

}  // namespace sq

namespace {

inline bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Byte ranges [a, a + na) and [b, b + nb) intersect.
inline bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  if (!a || !b || na == 0 || nb == 0) return false;
  const uintptr_t pa = reinterpret_cast<uintptr_t>(a), pb = reinterpret_cast<uintptr_t>(b);
  return pa < pb + nb && pb < pa + na;
}

struct Range {
  const void* p;
  size_t n;
};

// Every output range against every input range and every other output range.
template <size_t NO, size_t NI>
bool any_alias(const Range (&outs)[NO], const Range (&ins)[NI]) {
  for (size_t i = 0; i < NO; ++i) {
    for (size_t j = 0; j < NI; ++j)
      if (overlap(outs[i].p, outs[i].n, ins[j].p, ins[j].n)) return true;
    for (size_t j = i + 1; j < NO; ++j)
      if (overlap(outs[i].p, outs[i].n, outs[j].p, outs[j].n)) return true;
  }
  return false;
}

inline sq_status device_status(hipError_t e) {
  if (e == hipSuccess) return SQ_OK;
  if (e == hipErrorStreamCaptureUnsupported) return SQ_ERR_CAPTURE;  // the workspace would have to grow
  return SQ_ERR_DEVICE;
}

// The fused projections: a kernel without the fused form returns
// hipErrorNotSupported before it enqueues anything.
inline sq_status fused_status(hipError_t e) {
  return e == hipErrorNotSupported ? SQ_ERR_UNSUPPORTED : device_status(e);
}

constexpr int64_t kMaxK = int64_t(1) << 20;
constexpr int64_t kMaxN = 0x7FFFFFFF;
constexpr int64_t kMaxHidden = 16384;

// Shared limits of the block layout of the rope / attention calls.
sq_status check_block(int32_t b, int32_t rows_per_seq, int32_t hq, int32_t hkv, int64_t len_bound,
                      int64_t capacity) {
  if (b < 1 || rows_per_seq < 1 || rows_per_seq > 64 || hkv < 1 || hq < hkv || hq > 128 || hq % hkv != 0)
    return SQ_ERR_SHAPE;
  if (capacity < 64 || capacity > kMaxN || capacity % 64 != 0 || len_bound < 1 || len_bound > capacity)
    return SQ_ERR_SHAPE;
  if ((int64_t)b * rows_per_seq > kMaxN || (int64_t)b * hkv > 65535) return SQ_ERR_SHAPE;
  return SQ_OK;
}

// Shared checks of a normalised input (h rows m * group + group - 1, norm weights).
sq_status check_norm_src(const float* h, int32_t group, const uint16_t* norm_w, float eps, int64_t m, int64_t k) {
  if (!h || !norm_w) return SQ_ERR_NULL;
  if (group < 1 || m * group > kMaxN || k > kMaxHidden) return SQ_ERR_SHAPE;
  if (!isfinite(eps)) return SQ_ERR_NONFINITE;
  if (eps < 0.f) return SQ_ERR_SHAPE;
  if (!aligned(h, 16) || !aligned(norm_w, 16)) return SQ_ERR_ALIGN;
  return SQ_OK;
}

}  // namespace

extern "C" {

int32_t sq_abi_version(void) { return SQ_ABI_VERSION; }

const char* sq_status_str(sq_status s) {
  switch (s) {
    case SQ_OK: return "SQ_OK";
    case SQ_ERR_NULL: return "SQ_ERR_NULL: a required pointer is NULL";
    case SQ_ERR_SHAPE: return "SQ_ERR_SHAPE: a size is outside the supported range";
    case SQ_ERR_ALIGN: return "SQ_ERR_ALIGN: a pointer is misaligned";
    case SQ_ERR_ALIAS: return "SQ_ERR_ALIAS: an output overlaps an input or another output";
    case SQ_ERR_NONFINITE: return "SQ_ERR_NONFINITE: a scalar argument is NaN or infinite";
    case SQ_ERR_UNSUPPORTED: return "SQ_ERR_UNSUPPORTED: a dtype or mode outside what the call supports";
    case SQ_ERR_DEVICE: return "SQ_ERR_DEVICE: the HIP runtime reported an error";
    case SQ_ERR_CAPTURE:
      return "SQ_ERR_CAPTURE: the library workspace would have to grow while the stream is captured";
  }
  return "unknown sq_status";
}

sq_status sq_quantize_int4_g128(const uint16_t* w16, int64_t n, int64_t k, uint8_t* codes, uint16_t* scales,
                                uint16_t* zeros, int32_t* nonfinite_flag, hipStream_t stream) {
  if (!w16 || !codes || !scales || !zeros) return SQ_ERR_NULL;
  if (n < 1 || n > kMaxN || k < 128 || k > kMaxK || k % 128 != 0) return SQ_ERR_SHAPE;
  if (!aligned(w16, 16) || !aligned(codes, 16) || !aligned(scales, 2) || !aligned(zeros, 2) ||
      !aligned(nonfinite_flag, 4))
    return SQ_ERR_ALIGN;
  const size_t nk = (size_t)n * (size_t)k, ng = nk / 128;
  const Range outs[] = {{codes, nk / 2}, {scales, ng * 2}, {zeros, ng * 2}, {nonfinite_flag, 4}};
  const Range ins[] = {{w16, nk * 2}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  (void)hipGetLastError();
  return device_status(sq::launch_quantize_int4(w16, n, k, codes, scales, zeros, nonfinite_flag, stream));
}

sq_status sq_quantize_fp8_e4m3(const uint16_t* w16, int64_t n, int64_t k, uint8_t* codes, float* scales,
                               int32_t* nonfinite_flag, hipStream_t stream) {
  if (!w16 || !codes || !scales) return SQ_ERR_NULL;
  if (n < 1 || n > kMaxN || k < 16 || k > kMaxK || k % 16 != 0) return SQ_ERR_SHAPE;
  if (!aligned(w16, 16) || !aligned(codes, 16) || !aligned(scales, 4) || !aligned(nonfinite_flag, 4))
    return SQ_ERR_ALIGN;
  const size_t nk = (size_t)n * (size_t)k;
  const Range outs[] = {{codes, nk}, {scales, (size_t)n * 4}, {nonfinite_flag, 4}};
  const Range ins[] = {{w16, nk * 2}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  (void)hipGetLastError();
  return device_status(sq::launch_quantize_fp8(w16, n, k, codes, scales, nonfinite_flag, stream));
}

sq_status sq_qgemv_w4a16(const uint16_t* x, int64_t m, int64_t k, const uint8_t* codes, const uint16_t* scales,
                         const uint16_t* zeros, int64_t n, void* y, sq_dtype y_dtype, hipStream_t stream) {
  if (!x || !codes || !scales || !zeros || !y) return SQ_ERR_NULL;
  if (m < 1 || m > 64 || n < 1 || n > kMaxN || k < 128 || k > kMaxK || k % 128 != 0) return SQ_ERR_SHAPE;
  if (y_dtype != SQ_F16 && y_dtype != SQ_F32) return SQ_ERR_UNSUPPORTED;
  const size_t ysz = y_dtype == SQ_F16 ? 2 : 4;
  if (!aligned(x, 16) || !aligned(codes, 16) || !aligned(scales, 2) || !aligned(zeros, 2) || !aligned(y, ysz))
    return SQ_ERR_ALIGN;
  const size_t nk = (size_t)n * (size_t)k;
  const Range outs[] = {{y, (size_t)m * n * ysz}};
  const Range ins[] = {{x, (size_t)m * k * 2}, {codes, nk / 2}, {scales, nk / 64}, {zeros, nk / 64}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  (void)hipGetLastError();
  // the GEMVs up to m = 8, the matrix-core kernel (activation tiles of 16 rows) beyond
  if (m > 8)
    return device_status(sq::launch_linear_w4(x, (int)m, k, codes, scales, zeros, n, y, y_dtype == SQ_F16, stream));
  return device_status(sq::launch_gemv_w4(x, (int)m, k, codes, scales, zeros, n, y, y_dtype == SQ_F16, stream));
}

sq_status sq_qgemv_w8a16(const uint16_t* x, int64_t m, int64_t k, const uint8_t* codes, const float* scales,
                         int64_t n, void* y, sq_dtype y_dtype, hipStream_t stream) {
  if (!x || !codes || !scales || !y) return SQ_ERR_NULL;
  if (m < 1 || m > 64 || n < 1 || n > kMaxN || k < 16 || k > kMaxK || k % 16 != 0) return SQ_ERR_SHAPE;
  if (y_dtype != SQ_F16 && y_dtype != SQ_F32) return SQ_ERR_UNSUPPORTED;
  const size_t ysz = y_dtype == SQ_F16 ? 2 : 4;
  if (!aligned(x, 16) || !aligned(codes, 16) || !aligned(scales, 4) || !aligned(y, ysz)) return SQ_ERR_ALIGN;
  const size_t nk = (size_t)n * (size_t)k;
  const Range outs[] = {{y, (size_t)m * n * ysz}};
  const Range ins[] = {{x, (size_t)m * k * 2}, {codes, nk}, {scales, (size_t)n * 4}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  (void)hipGetLastError();
  // the matrix-core kernel from its size on at m >= 3, where its chunk
  // bookkeeping fits (it enqueues nothing when it returns hipErrorNotSupported);
  // at m <= 2 the GEMVs stream faster at every size (measured)
  // (above m = 8 only the matrix-core kernel)
  hipError_t e = hipErrorNotSupported;
  if (m > 8 || (m >= 3 && n * k >= kLinearMinBytesW8))
    e = sq::launch_linear_w8(x, (int)m, k, codes, scales, n, y, y_dtype == SQ_F16, stream);
  if (m > 8) return device_status(e);
  if (e == hipErrorNotSupported) e = sq::launch_gemv_w8(x, (int)m, k, codes, scales, n, y, y_dtype == SQ_F16, stream);
  return device_status(e);
}

sq_status sq_verify_gemm_f16(const uint16_t* x, int64_t m, int64_t k, const uint16_t* w16, int64_t n, void* y,
                             sq_dtype y_dtype, hipStream_t stream) {
  if (!x || !w16 || !y) return SQ_ERR_NULL;
  if (m < 1 || m > 64 || n < 1 || n > kMaxN || k < 8 || k > kMaxK || k % 8 != 0) return SQ_ERR_SHAPE;
  if (y_dtype != SQ_F16 && y_dtype != SQ_F32) return SQ_ERR_UNSUPPORTED;
  const size_t ysz = y_dtype == SQ_F16 ? 2 : 4;
  if (!aligned(x, 16) || !aligned(w16, 16) || !aligned(y, ysz)) return SQ_ERR_ALIGN;
  const Range outs[] = {{y, (size_t)m * n * ysz}};
  const Range ins[] = {{x, (size_t)m * k * 2}, {w16, (size_t)n * k * 2}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  (void)hipGetLastError();
  // row blocks on the vector ALUs for m <= 8 from 4 MiB of weights up to
  // 32768 rows (their activations and row slots must fit in LDS), the
  // matrix-core streaming kernel for larger matrices (m > 16: from 4 MiB),
  // else the tiled GEMM
  // (measured crossovers; each returns hipErrorNotSupported, enqueuing
  // nothing, for a shape it does not take)
  hipError_t e = hipErrorNotSupported;
  if (m <= 8 && n * k * 2 >= kRowsMinBytesF16 && n <= kRowsMaxRowsF16)
    e = sq::launch_gemm_rows_f16(x, (int)m, k, w16, n, y, y_dtype == SQ_F16, stream);
  if (e == hipErrorNotSupported && n * k * 2 >= (m > 16 ? kLinearMinBytesF16Wide : kLinearMinBytesF16))
    e = sq::launch_linear_f16(x, (int)m, k, w16, n, y, y_dtype == SQ_F16, stream);
  if (e == hipErrorNotSupported) e = sq::launch_gemm_f16(x, (int)m, k, w16, n, y, y_dtype == SQ_F16, stream);
  return device_status(e);
}

sq_status sq_qgemv_w4a16_rmsnorm(const float* h, int32_t group, const uint16_t* norm_w, float eps, int64_t m,
                                 int64_t k, const uint8_t* codes, const uint16_t* scales, const uint16_t* zeros,
                                 int64_t n, void* y, sq_dtype y_dtype, hipStream_t stream) {
  if (!codes || !scales || !zeros || !y) return SQ_ERR_NULL;
  if (m < 1 || m > 64 || n < 1 || n > kMaxN || k < 128 || k > kMaxK || k % 128 != 0) return SQ_ERR_SHAPE;
  const sq_status ns = check_norm_src(h, group, norm_w, eps, m, k);
  if (ns != SQ_OK) return ns;
  if (y_dtype != SQ_F16 && y_dtype != SQ_F32) return SQ_ERR_UNSUPPORTED;
  const size_t ysz = y_dtype == SQ_F16 ? 2 : 4;
  if (!aligned(codes, 16) || !aligned(scales, 2) || !aligned(zeros, 2) || !aligned(y, ysz)) return SQ_ERR_ALIGN;
  const size_t nk = (size_t)n * (size_t)k;
  const Range outs[] = {{y, (size_t)m * n * ysz}};
  const Range ins[] = {{h, (size_t)m * group * k * 4}, {norm_w, (size_t)k * 2}, {codes, nk / 2}, {scales, nk / 64},
                       {zeros, nk / 64}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  if (m > 8) return SQ_ERR_UNSUPPORTED;
  (void)hipGetLastError();
  const sq::NormSrc nrm{h, norm_w, eps, group};
  return fused_status(sq::launch_gemv_w4(nullptr, (int)m, k, codes, scales, zeros, n, y, y_dtype == SQ_F16, stream,
                                         &nrm, false));
}

sq_status sq_qgemv_w4a16_rmsnorm_silu(const float* h, int32_t group, const uint16_t* norm_w, float eps, int64_t m,
                                      int64_t k, const uint8_t* codes, const uint16_t* scales, const uint16_t* zeros,
                                      int64_t n, uint16_t* t, hipStream_t stream) {
  if (!codes || !scales || !zeros || !t) return SQ_ERR_NULL;
  if (m < 1 || m > 64 || n < 2 || n > kMaxN || n % 2 != 0 || k < 128 || k > kMaxK || k % 128 != 0)
    return SQ_ERR_SHAPE;
  const sq_status ns = check_norm_src(h, group, norm_w, eps, m, k);
  if (ns != SQ_OK) return ns;
  if (!aligned(codes, 16) || !aligned(scales, 2) || !aligned(zeros, 2) || !aligned(t, 2)) return SQ_ERR_ALIGN;
  const size_t nk = (size_t)n * (size_t)k;
  const Range outs[] = {{t, (size_t)m * (n / 2) * 2}};
  const Range ins[] = {{h, (size_t)m * group * k * 4}, {norm_w, (size_t)k * 2}, {codes, nk / 2}, {scales, nk / 64},
                       {zeros, nk / 64}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  if (m > 2) return SQ_ERR_UNSUPPORTED;
  (void)hipGetLastError();
  const sq::NormSrc nrm{h, norm_w, eps, group};
  return fused_status(
      sq::launch_gemv_w4(nullptr, (int)m, k, codes, scales, zeros, n, t, true, stream, &nrm, false, true));
}

sq_status sq_qgemv_w4a16_acc(const uint16_t* x, int64_t m, int64_t k, const uint8_t* codes, const uint16_t* scales,
                             const uint16_t* zeros, int64_t n, float* y, hipStream_t stream) {
  if (!x || !codes || !scales || !zeros || !y) return SQ_ERR_NULL;
  if (m < 1 || m > 64 || n < 1 || n > kMaxN || k < 128 || k > kMaxK || k % 128 != 0) return SQ_ERR_SHAPE;
  if (!aligned(x, 16) || !aligned(codes, 16) || !aligned(scales, 2) || !aligned(zeros, 2) || !aligned(y, 4))
    return SQ_ERR_ALIGN;
  const size_t nk = (size_t)n * (size_t)k;
  const Range outs[] = {{y, (size_t)m * n * 4}};
  const Range ins[] = {{x, (size_t)m * k * 2}, {codes, nk / 2}, {scales, nk / 64}, {zeros, nk / 64}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  if (m > 8) return SQ_ERR_UNSUPPORTED;
  (void)hipGetLastError();
  return fused_status(sq::launch_gemv_w4(x, (int)m, k, codes, scales, zeros, n, y, false, stream, nullptr, true));
}

sq_status sq_verify_gemm_f16_rmsnorm(const float* h, int32_t group, const uint16_t* norm_w, float eps, int64_t m,
                                     int64_t k, const uint16_t* w16, int64_t n, void* y, sq_dtype y_dtype,
                                     hipStream_t stream) {
  if (!w16 || !y) return SQ_ERR_NULL;
  if (m < 1 || m > 64 || n < 1 || n > kMaxN || k < 8 || k > kMaxK || k % 8 != 0) return SQ_ERR_SHAPE;
  const sq_status ns = check_norm_src(h, group, norm_w, eps, m, k);
  if (ns != SQ_OK) return ns;
  if (y_dtype != SQ_F16 && y_dtype != SQ_F32) return SQ_ERR_UNSUPPORTED;
  const size_t ysz = y_dtype == SQ_F16 ? 2 : 4;
  if (!aligned(w16, 16) || !aligned(y, ysz)) return SQ_ERR_ALIGN;
  const Range outs[] = {{y, (size_t)m * n * ysz}};
  const Range ins[] = {{h, (size_t)m * group * k * 4}, {norm_w, (size_t)k * 2}, {w16, (size_t)n * k * 2}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  // the row blocks, where sq_verify_gemm_f16 takes them
  if (!(m <= 8 && n * k * 2 >= kRowsMinBytesF16 && n <= kRowsMaxRowsF16)) return SQ_ERR_UNSUPPORTED;
  (void)hipGetLastError();
  const sq::NormSrc nrm{h, norm_w, eps, group};
  return fused_status(
      sq::launch_gemm_rows_f16(nullptr, (int)m, k, w16, n, y, y_dtype == SQ_F16, stream, &nrm, false));
}

sq_status sq_verify_gemm_f16_acc(const uint16_t* x, int64_t m, int64_t k, const uint16_t* w16, int64_t n, float* y,
                                 hipStream_t stream) {
  if (!x || !w16 || !y) return SQ_ERR_NULL;
  if (m < 1 || m > 64 || n < 1 || n > kMaxN || k < 8 || k > kMaxK || k % 8 != 0) return SQ_ERR_SHAPE;
  if (!aligned(x, 16) || !aligned(w16, 16) || !aligned(y, 4)) return SQ_ERR_ALIGN;
  const Range outs[] = {{y, (size_t)m * n * 4}};
  const Range ins[] = {{x, (size_t)m * k * 2}, {w16, (size_t)n * k * 2}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  if (!(m <= 8 && n * k * 2 >= kRowsMinBytesF16 && n <= kRowsMaxRowsF16)) return SQ_ERR_UNSUPPORTED;
  (void)hipGetLastError();
  return fused_status(sq::launch_gemm_rows_f16(x, (int)m, k, w16, n, y, false, stream, nullptr, true));
}

sq_status sq_probe_stream_read(const void* src, int64_t bytes, uint32_t* sink, hipStream_t stream) {
  if (!src || !sink) return SQ_ERR_NULL;
  if (bytes < 16 || bytes > (int64_t(1) << 40) || bytes % 16 != 0) return SQ_ERR_SHAPE;
  if (!aligned(src, 16) || !aligned(sink, 4)) return SQ_ERR_ALIGN;
  const Range outs[] = {{sink, (size_t)SQ_PROBE_SINK_WORDS * 4}};
  const Range ins[] = {{src, (size_t)bytes}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  (void)hipGetLastError();
  return device_status(sq::launch_stream_read(src, bytes, sink, SQ_PROBE_SINK_WORDS, stream));
}

// ------------------------------------------------------------ decoder layer
sq_status sq_embed_block_f16(const uint16_t* table, int64_t vocab, int64_t hidden, const int32_t* first,
                             const int32_t* rest, int32_t b, int32_t kd, float* h, int32_t* status,
                             hipStream_t stream) {
  if (!table || !first || !h || (kd > 0 && !rest)) return SQ_ERR_NULL;
  if (vocab < 1 || vocab > kMaxN || hidden < 8 || hidden > kMaxHidden || hidden % 8 != 0 || b < 1 || kd < 0 ||
      kd > 63 || (int64_t)b * (kd + 1) > kMaxN)
    return SQ_ERR_SHAPE;
  if (!aligned(table, 16) || !aligned(first, 4) || !aligned(rest, 4) || !aligned(h, 16) || !aligned(status, 4))
    return SQ_ERR_ALIGN;
  const size_t rows = (size_t)b * (kd + 1);
  const Range outs[] = {{h, rows * hidden * 4}, {status, 4}};
  const Range ins[] = {{table, (size_t)vocab * hidden * 2}, {first, (size_t)b * 4}, {rest, (size_t)kd * b * 4}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  (void)hipGetLastError();
  return device_status(sq::launch_embed_block(table, vocab, (int)hidden, first, rest, b, kd, h, status, stream));
}

sq_status sq_add_rmsnorm_f16(float* h, const float* delta, int64_t m, int64_t hidden, const uint16_t* w,
                             float eps, int32_t group, uint16_t* x, hipStream_t stream) {
  if (!h || !w || !x) return SQ_ERR_NULL;
  if (m < 1 || m > kMaxN || hidden < 8 || hidden > kMaxHidden || hidden % 8 != 0 || group < 1 || m % group != 0)
    return SQ_ERR_SHAPE;
  if (!isfinite(eps)) return SQ_ERR_NONFINITE;
  if (eps < 0.f) return SQ_ERR_SHAPE;
  if (!aligned(h, 16) || !aligned(delta, 16) || !aligned(w, 16) || !aligned(x, 16)) return SQ_ERR_ALIGN;
  const size_t mh = (size_t)m * hidden;
  const Range outs[] = {{h, mh * 4}, {x, mh / group * 2}};
  const Range ins[] = {{delta, mh * 4}, {w, (size_t)hidden * 2}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  (void)hipGetLastError();
  return device_status(sq::launch_add_rmsnorm(h, delta, m, (int)hidden, w, eps, group, x, stream));
}

sq_status sq_rope_kv_f16(const float* qkv, const uint16_t* bias, int32_t b, int32_t rows_per_seq, int32_t hq,
                         int32_t hkv, const int32_t* pos_base, int32_t pos_offset, int64_t len_bound,
                         int64_t capacity, double theta, uint16_t* q_out, uint16_t* k_cache, uint16_t* v_cache,
                         int32_t* status, hipStream_t stream) {
  if (!qkv || !pos_base || !q_out || !k_cache || !v_cache) return SQ_ERR_NULL;
  const sq_status bs = check_block(b, rows_per_seq, hq, hkv, len_bound, capacity);
  if (bs != SQ_OK) return bs;
  if (!isfinite(theta)) return SQ_ERR_NONFINITE;
  if (!(theta > 1.0)) return SQ_ERR_SHAPE;
  if (!aligned(qkv, 16) || !aligned(bias, 16) || !aligned(pos_base, 4) || !aligned(q_out, 16) ||
      !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(status, 4))
    return SQ_ERR_ALIGN;
  const size_t m = (size_t)b * rows_per_seq, nh = (size_t)hq + 2 * (size_t)hkv;
  const size_t cache = (size_t)b * hkv * capacity * 128 * 2;
  const Range outs[] = {{q_out, m * hq * 128 * 2}, {k_cache, cache}, {v_cache, cache}, {status, 4}};
  const Range ins[] = {{qkv, m * nh * 128 * 4}, {bias, nh * 128 * 2}, {pos_base, (size_t)b * 4}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  (void)hipGetLastError();
  return device_status(sq::launch_rope_kv(qkv, bias, (int)m, hq, hkv, rows_per_seq, pos_base, pos_offset, len_bound,
                                          capacity, theta, q_out, k_cache, v_cache, status, stream));
}

sq_status sq_attention_f16(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, int32_t b,
                           int32_t rows_per_seq, int32_t hq, int32_t hkv, const int32_t* pos_base,
                           int32_t pos_offset, int64_t len_bound, int64_t capacity, uint16_t* out,
                           hipStream_t stream) {
  if (!q || !k_cache || !v_cache || !pos_base || !out) return SQ_ERR_NULL;
  const sq_status bs = check_block(b, rows_per_seq, hq, hkv, len_bound, capacity);
  if (bs != SQ_OK) return bs;
  if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(pos_base, 4) ||
      !aligned(out, 16))
    return SQ_ERR_ALIGN;
  const size_t m = (size_t)b * rows_per_seq;
  const size_t cache = (size_t)b * hkv * capacity * 128 * 2;
  const Range outs[] = {{out, m * hq * 128 * 2}};
  const Range ins[] = {{q, m * hq * 128 * 2}, {k_cache, cache}, {v_cache, cache}, {pos_base, (size_t)b * 4}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  (void)hipGetLastError();
  return device_status(sq::launch_attention(q, k_cache, v_cache, b, rows_per_seq, hq, hkv, capacity, pos_base,
                                            pos_offset, len_bound, out, stream));
}

sq_status sq_rope_attention_f16(const float* qkv, const uint16_t* bias, int32_t b, int32_t rows_per_seq, int32_t hq,
                                int32_t hkv, const int32_t* pos_base, int32_t pos_offset, int64_t len_bound,
                                int64_t capacity, double theta, uint16_t* k_cache, uint16_t* v_cache, uint16_t* out,
                                int32_t* status, hipStream_t stream) {
  if (!qkv || !pos_base || !k_cache || !v_cache || !out) return SQ_ERR_NULL;
  const sq_status bs = check_block(b, rows_per_seq, hq, hkv, len_bound, capacity);
  if (bs != SQ_OK) return bs;
  if (!isfinite(theta)) return SQ_ERR_NONFINITE;
  if (!(theta > 1.0)) return SQ_ERR_SHAPE;
  if (!aligned(qkv, 16) || !aligned(bias, 16) || !aligned(pos_base, 4) || !aligned(k_cache, 16) ||
      !aligned(v_cache, 16) || !aligned(out, 16) || !aligned(status, 4))
    return SQ_ERR_ALIGN;
  const size_t m = (size_t)b * rows_per_seq, nh = (size_t)hq + 2 * (size_t)hkv;
  const size_t cache = (size_t)b * hkv * capacity * 128 * 2;
  const Range outs[] = {{out, m * hq * 128 * 2}, {k_cache, cache}, {v_cache, cache}, {status, 4}};
  const Range ins[] = {{qkv, m * nh * 128 * 4}, {bias, nh * 128 * 2}, {pos_base, (size_t)b * 4}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  if (rows_per_seq > 16 || rows_per_seq * (hq / hkv) > 64) return SQ_ERR_UNSUPPORTED;
  (void)hipGetLastError();
  return fused_status(sq::launch_rope_attention(qkv, bias, b, rows_per_seq, hq, hkv, capacity, pos_base, pos_offset,
                                                len_bound, theta, k_cache, v_cache, out, status, stream));
}

sq_status sq_silu_mul_f16(const float* gu, int64_t m, int64_t inter, uint16_t* t, hipStream_t stream) {
  if (!gu || !t) return SQ_ERR_NULL;
  if (m < 1 || inter < 1 || m > kMaxN || inter > kMaxN || m * inter >= (int64_t(1) << 40)) return SQ_ERR_SHAPE;
  if (!aligned(gu, 4) || !aligned(t, 2)) return SQ_ERR_ALIGN;
  const Range outs[] = {{t, (size_t)(m * inter) * 2}};
  const Range ins[] = {{gu, (size_t)(m * inter) * 8}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  (void)hipGetLastError();
  return device_status(sq::launch_silu_mul(gu, m, inter, t, stream));
}

sq_status sq_spec_commit(const int32_t* n_accepted, const int32_t* next_token, const int32_t* draft_tokens,
                         int32_t b, int32_t kd, int32_t* pending, int32_t* prev, int32_t* pos_base,
                         int32_t* out_tokens, int64_t out_capacity, int32_t* out_len, int32_t* status,
                         hipStream_t stream) {
  if (!n_accepted || !next_token || !pending || !prev || !pos_base || (kd > 0 && !draft_tokens) ||
      (out_tokens && !out_len))
    return SQ_ERR_NULL;
  if (b < 1 || b >= (1 << 24) || kd < 0 || kd > 64 || (out_tokens && (out_capacity < 1 || out_capacity > kMaxN)))
    return SQ_ERR_SHAPE;
  if (!aligned(n_accepted, 4) || !aligned(next_token, 4) || !aligned(draft_tokens, 4) || !aligned(pending, 4) ||
      !aligned(prev, 4) || !aligned(pos_base, 4) || !aligned(out_tokens, 4) || !aligned(out_len, 4) ||
      !aligned(status, 4))
    return SQ_ERR_ALIGN;
  const size_t b4 = (size_t)b * 4;
  const size_t hist = out_tokens ? (size_t)b * (size_t)out_capacity * 4 : 0;
  const Range outs[] = {{pending, b4}, {prev, b4}, {pos_base, b4}, {out_tokens, hist},
                        {out_tokens ? out_len : nullptr, b4}, {status, 4}};
  const Range ins[] = {{n_accepted, b4}, {next_token, b4}, {draft_tokens, (size_t)kd * b4}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  (void)hipGetLastError();
  return device_status(sq::launch_spec_commit(n_accepted, next_token, draft_tokens, b, kd, pending, prev, pos_base,
                                              out_tokens, out_capacity, out_tokens ? out_len : nullptr, status,
                                              stream));
}

// ------------------------------------------------------ several draft chains
sq_status sq_spec_accept_multi(const float* draft_logits, const float* target_logits, const int32_t* draft_tokens,
                               const uint32_t* u24, int32_t b, int32_t c, int32_t kd, int32_t v, float temperature,
                               int32_t* n_accepted, int32_t* next_token, int32_t* chain, float* q_out, float* p_out,
                               hipStream_t stream) {
  if (!target_logits || !n_accepted || !next_token || !chain) return SQ_ERR_NULL;
  if (kd > 0 && (!draft_logits || !draft_tokens)) return SQ_ERR_NULL;
  if (b < 1 || b > 65535 || c < 1 || c > 64 || kd < 0 || kd > 64 || v < 1 || v > (1 << 26)) return SQ_ERR_SHAPE;
  const int64_t nchunk = (v + sq::kAcceptChunk - 1) / sq::kAcceptChunk;
  if ((int64_t)b * c * (2 * kd + 1) * nchunk >= (int64_t(1) << 24)) return SQ_ERR_SHAPE;
  if (!isfinite(temperature)) return SQ_ERR_NONFINITE;
  if (temperature < 0.0f) return SQ_ERR_UNSUPPORTED;
  if (temperature == 0.0f && (q_out || p_out)) return SQ_ERR_UNSUPPORTED;
  if (temperature > 0.0f && !u24) return SQ_ERR_NULL;
  if (!aligned(draft_logits, 4) || !aligned(target_logits, 4) || !aligned(draft_tokens, 4) || !aligned(u24, 4) ||
      !aligned(n_accepted, 4) || !aligned(next_token, 4) || !aligned(chain, 4) || !aligned(q_out, 4) ||
      !aligned(p_out, 4))
    return SQ_ERR_ALIGN;
  const size_t bc = (size_t)b * c, bcv = bc * v;
  const Range outs[] = {{n_accepted, (size_t)b * 4}, {next_token, (size_t)b * 4}, {chain, (size_t)b * 4},
                        {q_out, (size_t)kd * bcv * 4}, {p_out, (size_t)(kd + 1) * bcv * 4}};
  const Range ins[] = {{draft_logits, (size_t)kd * bcv * 4},
                       {target_logits, (size_t)(kd + 1) * bcv * 4},
                       {draft_tokens, (size_t)kd * bc * 4},
                       {u24, temperature > 0.0f ? (size_t)b * (c * kd + 1) * 4 : 0}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  (void)hipGetLastError();
  return device_status(sq::launch_spec_accept_multi(draft_logits, target_logits, draft_tokens, u24, b, c, kd, v,
                                                    temperature, n_accepted, next_token, chain, q_out, p_out,
                                                    stream));
}

sq_status sq_kv_adopt_f16(uint16_t* k_cache, uint16_t* v_cache, int32_t layers, int32_t b, int32_t c, int32_t hkv,
                          int64_t capacity, const int32_t* chain, const int32_t* n_accepted, const int32_t* pos_base,
                          int32_t lo_offset, int32_t hi_offset, hipStream_t stream) {
  if (!k_cache || !v_cache || !chain || !n_accepted || !pos_base) return SQ_ERR_NULL;
  if (layers < 1 || layers > 65535 || b < 1 || c < 1 || c > 64 || (int64_t)b * c > 65535 || hkv < 1 ||
      hkv > 65535 || capacity < 64 || capacity > kMaxN || capacity % 64 != 0 || lo_offset < -64 || lo_offset > 64 ||
      hi_offset < -64 || hi_offset > 64)
    return SQ_ERR_SHAPE;
  if (!aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(chain, 4) || !aligned(n_accepted, 4) ||
      !aligned(pos_base, 4))
    return SQ_ERR_ALIGN;
  const size_t cache = (size_t)layers * b * c * hkv * capacity * 128 * 2;
  const Range outs[] = {{k_cache, cache}, {v_cache, cache}};
  const Range ins[] = {{chain, (size_t)b * 4}, {n_accepted, (size_t)b * 4}, {pos_base, (size_t)b * c * 4}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  (void)hipGetLastError();
  return device_status(sq::launch_kv_adopt(k_cache, v_cache, layers, b, c, hkv, capacity, chain, n_accepted, pos_base,
                                           lo_offset, hi_offset, stream));
}

sq_status sq_spec_commit_multi(const int32_t* n_accepted, const int32_t* next_token, const int32_t* chain,
                               const int32_t* draft_tokens, int32_t b, int32_t c, int32_t kd, int32_t* pending,
                               int32_t* prev, int32_t* pos_base, int32_t* out_tokens, int64_t out_capacity,
                               int32_t* out_len, int32_t* status, hipStream_t stream) {
  if (!n_accepted || !next_token || !chain || !pending || !prev || !pos_base || (kd > 0 && !draft_tokens) ||
      (out_tokens && !out_len))
    return SQ_ERR_NULL;
  if (b < 1 || b >= (1 << 24) || c < 1 || c > 64 || kd < 0 || kd > 64 ||
      (out_tokens && (out_capacity < 1 || out_capacity > kMaxN)))
    return SQ_ERR_SHAPE;
  if (!aligned(n_accepted, 4) || !aligned(next_token, 4) || !aligned(chain, 4) || !aligned(draft_tokens, 4) ||
      !aligned(pending, 4) || !aligned(prev, 4) || !aligned(pos_base, 4) || !aligned(out_tokens, 4) ||
      !aligned(out_len, 4) || !aligned(status, 4))
    return SQ_ERR_ALIGN;
  const size_t b4 = (size_t)b * 4, bc4 = b4 * c;
  const size_t hist = out_tokens ? (size_t)b * (size_t)out_capacity * 4 : 0;
  const Range outs[] = {{pending, bc4}, {prev, bc4}, {pos_base, bc4}, {out_tokens, hist},
                        {out_tokens ? out_len : nullptr, b4}, {status, 4}};
  const Range ins[] = {{n_accepted, b4}, {next_token, b4}, {chain, b4}, {draft_tokens, (size_t)kd * bc4}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  (void)hipGetLastError();
  return device_status(sq::launch_spec_commit_multi(n_accepted, next_token, chain, draft_tokens, b, c, kd, pending,
                                                    prev, pos_base, out_tokens, out_capacity,
                                                    out_tokens ? out_len : nullptr, status, stream));
}

}  // extern "C"

namespace {

// Host-side validation shared by the two accept entry points.
sq_status validate_accept(const float* draft_logits, const float* target_logits, const int32_t* draft_tokens,
                          const uint32_t* u24, int32_t b, int32_t kd, int32_t v, float temperature,
                          int32_t* n_accepted, int32_t* next_token, float* q_out, float* p_out) {
  if (!target_logits || !n_accepted || !next_token) return SQ_ERR_NULL;
  if (kd > 0 && (!draft_logits || !draft_tokens)) return SQ_ERR_NULL;
  if (b < 1 || b >= (1 << 24) || kd < 0 || kd > 64 || v < 1 || v > (1 << 26)) return SQ_ERR_SHAPE;
  const int64_t nchunk = (v + sq::kAcceptChunk - 1) / sq::kAcceptChunk;
  // every kernel grid stays below 2^24 workgroups of 256 threads (2^32 work-items)
  if ((int64_t)b * (2 * kd + 1) * nchunk >= (int64_t(1) << 24)) return SQ_ERR_SHAPE;
  if (!isfinite(temperature)) return SQ_ERR_NONFINITE;
  if (temperature < 0.0f) return SQ_ERR_UNSUPPORTED;
  if (temperature == 0.0f && (q_out || p_out)) return SQ_ERR_UNSUPPORTED;
  if (temperature > 0.0f && !u24) return SQ_ERR_NULL;
  if (!aligned(draft_logits, 4) || !aligned(target_logits, 4) || !aligned(draft_tokens, 4) || !aligned(u24, 4) ||
      !aligned(n_accepted, 4) || !aligned(next_token, 4) || !aligned(q_out, 4) || !aligned(p_out, 4))
    return SQ_ERR_ALIGN;
  const size_t bk = (size_t)b * kd, bv = (size_t)b * v;
  const Range outs[] = {{n_accepted, (size_t)b * 4},
                        {next_token, (size_t)b * 4},
                        {q_out, (size_t)kd * bv * 4},
                        {p_out, (size_t)(kd + 1) * bv * 4}};
  const Range ins[] = {{draft_logits, (size_t)kd * bv * 4},
                       {target_logits, (size_t)(kd + 1) * bv * 4},
                       {draft_tokens, bk * 4},
                       {u24, (size_t)b * (kd + 1) * 4}};
  if (any_alias(outs, ins)) return SQ_ERR_ALIAS;
  return SQ_OK;
}

}  // namespace

extern "C" {

sq_status sq_spec_accept(const float* draft_logits, const float* target_logits, const int32_t* draft_tokens,
                         const uint32_t* u24, int32_t b, int32_t kd, int32_t v, float temperature,
                         int32_t* n_accepted, int32_t* next_token, float* q_out, float* p_out, hipStream_t stream) {
  const sq_status st = validate_accept(draft_logits, target_logits, draft_tokens, u24, b, kd, v, temperature,
                                       n_accepted, next_token, q_out, p_out);
  if (st != SQ_OK) return st;
  (void)hipGetLastError();
  return device_status(sq::launch_spec_accept(draft_logits, target_logits, draft_tokens, u24, b, kd, v, temperature,
                                              n_accepted, next_token, q_out, p_out, stream));
}

sq_status sq_spec_accept_noalloc(const float* draft_logits, const float* target_logits, const int32_t* draft_tokens,
                                 const uint32_t* u24, int32_t b, int32_t kd, int32_t v, float temperature,
                                 int32_t* n_accepted, int32_t* next_token, float* q_out, float* p_out,
                                 hipStream_t stream) {
  const sq_status st = validate_accept(draft_logits, target_logits, draft_tokens, u24, b, kd, v, temperature,
                                       n_accepted, next_token, q_out, p_out);
  if (st != SQ_OK) return st;
  if (sq::spec_accept_scratch_bytes(b, kd, v, temperature) > SQ_NOALLOC_SCRATCH_BYTES) return SQ_ERR_SHAPE;
  (void)hipGetLastError();
  return device_status(sq::launch_spec_accept_noalloc(draft_logits, target_logits, draft_tokens, u24, b, kd, v,
                                                      temperature, n_accepted, next_token, q_out, p_out, stream));
}

}  // extern "C"

// Diagnostic kernels used by the measurement harness: a plain streaming copy,
// the reference point for HBM bandwidth and for hardware byte counters.
#include "common.h"

namespace cofie {
namespace {

__global__ __launch_bounds__(256) void stream_copy_kernel(const uint4* __restrict__ src,
                                                          uint4* __restrict__ dst, int64_t n16) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n16;
       i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

// Streaming read: every 16-byte word is loaded once; a per-thread XOR is
// written so the loads cannot be elided.
__global__ __launch_bounds__(256) void stream_read_kernel(const uint4* __restrict__ src, int64_t n16,
                                                          uint32_t* __restrict__ sink) {
  uint32_t x = 0;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n16;
       i += (int64_t)gridDim.x * blockDim.x) {
    const uint4 v = src[i];
    x ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  sink[blockIdx.x * (int64_t)blockDim.x + threadIdx.x] = x;
}

}  // namespace
}  // namespace cofie

extern "C" int cofie_diag_stream_copy(const void* src, void* dst, size_t bytes, void* stream) {
  using namespace cofie;
  clear_error();
  if (bytes == 0) return COFIE_OK;
  if (!src || !dst) return set_error(COFIE_EINVAL, "null pointer");
  if ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst) | bytes) % 16 != 0)
    return set_error(COFIE_EINVAL, "pointers and size must be multiples of 16 bytes");
  const int64_t n16 = (int64_t)(bytes / 16);
  const int64_t grid = std::min<int64_t>((n16 + 255) / 256, 16LL * device_cu_count());
  return launch("diag_stream_copy", stream_copy_kernel, dim3((unsigned)grid), dim3(256), 0,
                static_cast<hipStream_t>(stream), static_cast<const uint4*>(src),
                static_cast<uint4*>(dst), n16);
}

extern "C" int cofie_diag_stream_read(const void* src, size_t bytes, uint32_t* sink,
                                      size_t sink_words, void* stream) {
  using namespace cofie;
  clear_error();
  if (bytes == 0) return COFIE_OK;
  if (!src || !sink) return set_error(COFIE_EINVAL, "null pointer");
  if ((reinterpret_cast<uintptr_t>(src) | bytes) % 16 != 0)
    return set_error(COFIE_EINVAL, "pointer and size must be multiples of 16 bytes");
  const int64_t n16 = (int64_t)(bytes / 16);
  int64_t grid = std::min<int64_t>((n16 + 255) / 256, 16LL * device_cu_count());
  grid = std::min<int64_t>(grid, (int64_t)(sink_words / 256));
  if (grid < 1) return set_error(COFIE_EINVAL, "sink needs at least 256 words");
  return launch("diag_stream_read", stream_read_kernel, dim3((unsigned)grid), dim3(256), 0,
                static_cast<hipStream_t>(stream), static_cast<const uint4*>(src), n16, sink);
}

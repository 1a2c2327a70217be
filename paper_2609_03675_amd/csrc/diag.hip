// Diagnostic kernels used by the measurement harness: a plain streaming copy,
// the reference point for HBM bandwidth and for hardware byte counters.
#include "common.h"

namespace cofie {
namespace {

typedef unsigned int u32x4v __attribute__((ext_vector_type(4)));

// Both probes use non-temporal accesses, as the streaming kernels they are
// compared with do, one 16-byte access per thread and iteration over a grid
// of 8 workgroups per CU: the fastest plain streaming read measured on the
// MI355X (7.1 TB/s for 1 GiB; unrolling 4 grid-strided loads per thread read
// at 5.6 TB/s, plain loads at 6.4 TB/s).
__global__ __launch_bounds__(256) void stream_copy_kernel(const u32x4v* __restrict__ src,
                                                          u32x4v* __restrict__ dst, int64_t n16) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n16;
       i += (int64_t)gridDim.x * blockDim.x)
    __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

// Streaming read: every 16-byte word is loaded once; a per-thread XOR is
// written so the loads cannot be elided.
__global__ __launch_bounds__(256) void stream_read_kernel(const u32x4v* __restrict__ src, int64_t n16,
                                                          uint32_t* __restrict__ sink) {
  u32x4v x = {0u, 0u, 0u, 0u};
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n16;
       i += (int64_t)gridDim.x * blockDim.x)
    x ^= __builtin_nontemporal_load(src + i);
  sink[blockIdx.x * (int64_t)blockDim.x + threadIdx.x] = x.x ^ x.y ^ x.z ^ x.w;
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
  const int64_t grid = std::min<int64_t>((n16 + 255) / 256, 8LL * device_cu_count());
  return launch("diag_stream_copy", stream_copy_kernel, dim3((unsigned)grid), dim3(256), 0,
                static_cast<hipStream_t>(stream), static_cast<const u32x4v*>(src),
                static_cast<u32x4v*>(dst), n16);
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
  int64_t grid = std::min<int64_t>((n16 + 255) / 256, 8LL * device_cu_count());
  grid = std::min<int64_t>(grid, (int64_t)(sink_words / 256));
  if (grid < 1) return set_error(COFIE_EINVAL, "sink needs at least 256 words");
  return launch("diag_stream_read", stream_read_kernel, dim3((unsigned)grid), dim3(256), 0,
                static_cast<hipStream_t>(stream), static_cast<const u32x4v*>(src), n16, sink);
}

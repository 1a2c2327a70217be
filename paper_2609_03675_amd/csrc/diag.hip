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

// Internal plumbing shared by the libcofie sources: error reporting, kernel
// launch with optional event timing, and a stream-ordered scratch arena.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <cstdio>
#include <string>

#include "cofie.h"

namespace cofie {

// ---- errors -----------------------------------------------------------------
int set_error(int code, const char* fmt, ...);
void clear_error();

#define COFIE_CHECK_HIP(expr)                                                        \
  do {                                                                               \
    hipError_t _e = (expr);                                                          \
    if (_e != hipSuccess)                                                            \
      return ::cofie::set_error(COFIE_EHIP, "%s failed: %s", #expr, hipGetErrorString(_e)); \
  } while (0)

// ---- kernel timing ------------------------------------------------------------
// When the profiler is enabled, prof_slot hands out a start/stop event pair for
// one launch (and returns false otherwise).  The launch carries the pair in its
// own dispatch (hipExtLaunchKernel), so the elapsed time is the kernel's alone,
// without the latency of separate event packets on the stream.
bool prof_slot(const char* name, hipEvent_t* start, hipEvent_t* stop);

// Launch `kernel` on `s` (timed when profiling is on) and turn a launch failure
// into COFIE_EHIP.
template <typename... KArgs, typename... Args>
int launch(const char* name, void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t lds,
           hipStream_t s, Args... args) {
  if (grid.x == 0 || grid.y == 0 || grid.z == 0) return COFIE_OK;
  (void)hipGetLastError();
  hipEvent_t start = nullptr, stop = nullptr;
  if (prof_slot(name, &start, &stop))
    hipExtLaunchKernelGGL(kernel, grid, block, (uint32_t)lds, s, start, stop, 0u, static_cast<KArgs>(args)...);
  else
    hipLaunchKernelGGL(kernel, grid, block, lds, s, static_cast<KArgs>(args)...);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    return set_error(COFIE_EHIP, "launch of %s failed: %s", name, hipGetErrorString(e));
  return COFIE_OK;
}

// Allow a kernel more than the default dynamic LDS (gfx950 has 160 KiB per CU).
// The attribute is set once per kernel and size, so later calls (including
// ones made while a stream is being captured into a graph) make no runtime call.
bool lds_attr_done(const void* kernel, size_t bytes);
void lds_attr_mark(const void* kernel, size_t bytes);

template <typename... KArgs>
int allow_lds(void (*kernel)(KArgs...), size_t bytes) {
  if (bytes <= 65536) return COFIE_OK;
  const void* k = reinterpret_cast<const void*>(kernel);
  if (lds_attr_done(k, bytes)) return COFIE_OK;
  hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  if (e != hipSuccess)
    return set_error(COFIE_EHIP, "hipFuncSetAttribute(LDS=%zu) failed: %s", bytes,
                     hipGetErrorString(e));
  lds_attr_mark(k, bytes);
  return COFIE_OK;
}

// ---- scratch arena ------------------------------------------------------------
// A planner and allocator in one: the same sequence of take() calls first sizes
// the arena (base == nullptr) and then carves it.  Every block is 256-byte
// aligned.
struct Arena {
  char* base = nullptr;
  size_t used = 0;
  template <typename T>
  T* take(size_t count) {
    size_t off = (used + 255) & ~size_t(255);
    used = off + count * sizeof(T);
    return base ? reinterpret_cast<T*>(base + off) : nullptr;
  }
  size_t bytes() const { return (used + 255) & ~size_t(255); }
};

// Owns library-allocated scratch (hipMallocAsync) or wraps the caller's.
class Scratch {
 public:
  Scratch() = default;
  Scratch(const Scratch&) = delete;
  Scratch& operator=(const Scratch&) = delete;
  ~Scratch();
  // Make `need` bytes available: the caller's workspace if given (ENOMEM if too
  // small), else a stream-ordered allocation freed when this object dies.
  int acquire(void* ws, size_t ws_bytes, size_t need, hipStream_t s);
  char* ptr() const { return base_; }

 private:
  char* base_ = nullptr;
  bool owned_ = false;
  hipStream_t stream_ = nullptr;
};

inline int ceil_div(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

// Number of compute units of the current device (cached).
int device_cu_count();

}  // namespace cofie

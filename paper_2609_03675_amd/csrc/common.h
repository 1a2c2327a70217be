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

// ---- host-side address check (dry run) ------------------------------------------
// With the dry run on (cofie_debug_dry_run, for tests on the host: no GPU is
// touched), the entry points validate and plan as usual but launch nothing and
// make no HIP call; the kernels that have an address model walk instead every
// global and LDS address their threads would touch, computed by the same
// index functions the kernels use, and check each against the buffers the
// caller registered (fake device addresses with their sizes) or the launch's
// LDS size.  A violation records the first offending access.
bool dry_run();
// [base + off, base + off + bytes) must lie in the registered buffer that
// holds `base` (the kernel's base pointer for this access)
void dry_access(const void* base, int64_t off, int64_t bytes, const char* what);
void dry_lds(int64_t off, int64_t bytes, int64_t lds_bytes, const char* what);
// lo <= v < hi (an index that stays inside its buffer but would read or write
// another row's or slot's data)
void dry_range(int64_t v, int64_t lo, int64_t hi, const char* what);
// Host-to-device copy of a plan table: in a dry run the bytes are kept on the
// host as the shadow of `dst`, where the address models read them back with
// dry_shadow (null for an address that no copy wrote).
int copy_to_device(void* dst, const void* src, size_t bytes, hipStream_t s, const char* what);
const void* dry_shadow(const void* dst);

// Launch `kernel` on `s` (timed when profiling is on) and turn a launch failure
// into COFIE_EHIP.  In a dry run nothing is launched.
template <typename... KArgs, typename... Args>
int launch(const char* name, void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t lds,
           hipStream_t s, Args... args) {
  if (grid.x == 0 || grid.y == 0 || grid.z == 0) return COFIE_OK;
  if (dry_run()) return COFIE_OK;
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
  if (bytes <= 65536 || dry_run()) return COFIE_OK;
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

// ---- last workgroup to arrive -------------------------------------------------
// Lets the workgroups of one launch finish a reduction without a second
// launch: the one workgroup that arrives last continues with everything the
// others published.  Measured on gfx950, a device-scope fence costs a whole
// L2 writeback and invalidate (tens of microseconds when every workgroup of a
// grid does it), and atomics on one address serialise at ~20-30 ns each, so:
//  * published data is written with device-coherent stores (st_agent: relaxed
//    agent-scope atomic stores, which write through to the coherence point),
//    so no contributor has to write its L2 back or invalidate it;
//  * each wave waits for its own stores to complete (s_waitcnt vmcnt(0))
//    before the workgroup barrier, and one thread then adds to the counter
//    (an agent-scope release RMW);
//  * only the last arriver acquires (one L2/L1 invalidate, completed before
//    the workgroup barrier), after which plain loads of every wave see the
//    published data;
//  * up to kArriveFlat contributors count on one counter; more go through a
//    two-level tree: workgroup b of nb counts at sub-counter b % G
//    (G = kArriveFan), the last of each sub-counter at the root, so no
//    counter sees more than max(ceil(nb / G), G) arrivals.  Counters sit
//    `stride` ints apart.
// A tree is (G + 1) * stride ints, zero on entry (an earlier kernel on the
// stream clears it).  Nobody waits for anybody, so this cannot deadlock.
constexpr int kArriveFan = 8;
constexpr int kArriveFlat = 32;

template <typename T>
__device__ __forceinline__ void st_agent(T* p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// This wave's vector-memory operations have completed (gfx9 s_waitcnt
// encoding: vmcnt = 0, expcnt and lgkmcnt not waited for).
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// One counter: true in every thread of the workgroup whose addition completes
// `total` arrivals.
__device__ inline bool arrive_counter(int32_t* counter, int32_t total, int32_t* flag_sh) {
  wait_vmem();
  __syncthreads();
  if (threadIdx.x == 0) {
    const int32_t old = __hip_atomic_fetch_add(counter, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    const bool last = old + 1 == total;
    if (last) {
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
      wait_vmem();  // the invalidate has completed before the other waves load
    }
    *flag_sh = last;
  }
  __syncthreads();
  return *flag_sh != 0;
}

// Sub-counters of a tree for nb contributors (0: one flat counter).
inline __host__ __device__ int32_t arrive_fan(int32_t nb) { return nb <= kArriveFlat ? 0 : kArriveFan; }

// Workgroup b (0 <= b < nb) of the contributors to `tree` arrives; true in the
// last one.  Every thread of the workgroup calls it, after its st_agent stores.
__device__ inline bool arrive_last(int32_t* tree, int32_t stride, int32_t b, int32_t nb, int32_t* flag_sh) {
  if (nb <= 1) {  // the only contributor: its own waves' stores are complete
    wait_vmem();
    __syncthreads();
    return true;
  }
  if (nb <= kArriveFlat) return arrive_counter(tree, nb, flag_sh);
  const int32_t G = arrive_fan(nb);
  const int32_t j = b % G;
  const int32_t expect = (nb - 1 - j) / G + 1;  // contributors b' < nb with b' % G == j
  if (!arrive_counter(tree + (1 + j) * stride, expect, flag_sh)) return false;
  return arrive_counter(tree, G, flag_sh);
}

}  // namespace cofie

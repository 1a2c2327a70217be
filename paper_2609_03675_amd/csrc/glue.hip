// Coarse-to-fine glue on gfx950.
//
// cofie_mask_compact: the NGFF candidate set S_c as frame indices (Sec. 3.1 -
//   3.2: the candidates are what the visual encoder runs on).  One workgroup
//   walks the mask in chunks of 1024 x 16 frames: per-thread counts, a block
//   exclusive scan, a running total across chunks.  One launch and no scratch
//   for any n; the whole stream of even a C5-sized batch is a few chunks.
// cofie_gather_frames: frame refinement (Sec. 3.3): the rows of the frames in
//   S_e, in the order given (chronological for a top-k), appended to a compact
//   buffer -- the hidden states / cached keys and values / positions of the
//   kept frames.  A one-workgroup scan turns the clamped frame lengths into
//   the output CSR; a copy kernel then streams every selected frame's
//   contiguous byte range with 16-byte lanes (4-byte or byte lanes when the
//   pointers or the row size are not aligned), bounded by the capacity.
#include <climits>
#include <type_traits>

#include "common.h"

namespace cofie {
namespace {

constexpr int kGlueThreads = 1024;
constexpr int kMaskPerThread = 16;

// Exclusive prefix sum over the block (1024 threads); total in *total.
__device__ int64_t block_exscan64(int64_t v, int64_t* total, int64_t* wsum) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int64_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  int64_t before = 0, all = 0;
  for (int i = 0; i < nw; ++i) {
    if (i < wave) before += wsum[i];
    all += wsum[i];
  }
  __syncthreads();
  *total = all;
  return before + x - v;
}

__global__ __launch_bounds__(kGlueThreads) void mask_compact_kernel(const uint8_t* mask, int64_t n,
                                                                    int64_t seg_len, int64_t nseg,
                                                                    int32_t* out_idx,
                                                                    int32_t* out_seg_start) {
  __shared__ int64_t wsum[16];
  const int tid = threadIdx.x;
  const int64_t per_chunk = (int64_t)kGlueThreads * kMaskPerThread;
  int64_t base_count = 0;
  for (int64_t c0 = 0; c0 < n; c0 += per_chunk) {
    const int64_t f0 = c0 + (int64_t)tid * kMaskPerThread;
    uint8_t m[kMaskPerThread];
#pragma unroll
    for (int j = 0; j < kMaskPerThread; ++j) m[j] = f0 + j < n ? mask[f0 + j] : 0;
    int64_t cnt = 0;
#pragma unroll
    for (int j = 0; j < kMaskPerThread; ++j) cnt += m[j] != 0 ? 1 : 0;
    int64_t total;
    int64_t pos = base_count + block_exscan64(cnt, &total, wsum);
#pragma unroll
    for (int j = 0; j < kMaskPerThread; ++j) {
      const int64_t f = f0 + j;
      if (f < n) {
        // this frame opens a stream segment: candidates before it
        if (seg_len > 0 ? f % seg_len == 0 : f == 0) out_seg_start[seg_len > 0 ? f / seg_len : 0] = (int32_t)pos;
        if (m[j] != 0) out_idx[pos++] = (int32_t)f;
      }
    }
    base_count += total;
  }
  if (tid == 0) {
    if (n == 0 && nseg > 0) out_seg_start[0] = 0;
    out_seg_start[nseg] = (int32_t)base_count;
  }
}

// Rows [lo, hi) of frame f: its CSR range clamped to [0, n_rows) (empty for
// a frame index outside [0, n_frames) or a decreasing range).
__host__ __device__ __forceinline__ void frame_rows(const int32_t* offs, int32_t n_frames, int64_t n_rows,
                                                    int32_t f, int64_t* lo, int64_t* hi) {
  if (f < 0 || f >= n_frames) {
    *lo = *hi = 0;
    return;
  }
  int64_t a = offs[f], b = offs[f + 1];
  a = a < 0 ? 0 : (a > n_rows ? n_rows : a);
  b = b < 0 ? 0 : (b > n_rows ? n_rows : b);
  *lo = a;
  *hi = b < a ? a : b;
}

// An output offset as stored: a running row count saturated at 2^31 - 1, so
// that a total past the int32 range never wraps to a negative offset (the
// capacity is below 2^31, so every frame placed past it is skipped).
__host__ __device__ __forceinline__ int32_t out_offset(int64_t rows) {
  return (int32_t)(rows < INT32_MAX ? rows : INT32_MAX);
}

// out_offs[0..k]: exclusive scan of the selected frames' clamped row counts
__global__ __launch_bounds__(kGlueThreads) void gather_offsets_kernel(const int32_t* offs, int32_t n_frames,
                                                                      int64_t n_rows, const int32_t* sel,
                                                                      int32_t k, int32_t* out_offs) {
  __shared__ int64_t wsum[16];
  const int tid = threadIdx.x;
  int64_t base = 0;
  for (int32_t i0 = 0; i0 < k; i0 += kGlueThreads) {
    const int32_t i = i0 + tid;
    int64_t len = 0;
    if (i < k) {
      int64_t lo, hi;
      frame_rows(offs, n_frames, n_rows, sel[i], &lo, &hi);
      len = hi - lo;
    }
    int64_t total;
    const int64_t ex = block_exscan64(len, &total, wsum);
    if (i < k) out_offs[i + 1] = out_offset(base + ex + len);
    base += total;
  }
  if (tid == 0) out_offs[0] = 0;
}

// Copy of the selected frames' rows: blockIdx.y (strided) picks the frame,
// blockIdx.x (strided) a slice of its bytes.  V = bytes per lane access (16:
// non-temporal, both sides are touched once).  With out_offs null each
// workgroup sums the row counts of the frames before its own, and workgroup
// (0, 0) writes the output offsets to offs_out, so no offsets kernel runs
// first.
typedef unsigned u32x4v __attribute__((ext_vector_type(4)));

template <int V>
__global__ __launch_bounds__(256) void gather_copy_kernel(const uint8_t* src, int64_t n_rows, int64_t row_bytes,
                                                          const int32_t* offs, int32_t n_frames,
                                                          const int32_t* sel, int32_t k, uint8_t* dst,
                                                          int64_t capacity, const int32_t* out_offs,
                                                          int32_t* offs_out, int32_t* out_rows) {
  using T = typename std::conditional<V == 16, u32x4v, typename std::conditional<V == 4, uint32_t, uint8_t>::type>::type;
  constexpr int U = 4;  // accesses in flight per lane
  __shared__ int64_t wsum[4];
  for (int32_t i = blockIdx.y; i < k; i += gridDim.y) {
    int64_t lo, hi;
    frame_rows(offs, n_frames, n_rows, sel[i], &lo, &hi);
    int64_t o;
    if (out_offs) {
      o = out_offs[i];
    } else {
      int64_t part = 0;
      for (int32_t j = threadIdx.x; j < i; j += blockDim.x) {
        int64_t a, b;
        frame_rows(offs, n_frames, n_rows, sel[j], &a, &b);
        part += b - a;
      }
      (void)block_exscan64(part, &o, wsum);
    }
    int64_t rows = hi - lo;
    const int64_t room = capacity - o;
    rows = rows < room ? rows : (room > 0 ? room : 0);
    if (rows <= 0) continue;
    const int64_t nv = rows * row_bytes / V;  // row_bytes % V == 0 on this path
    const T* s = reinterpret_cast<const T*>(src + lo * row_bytes);
    T* d = reinterpret_cast<T*>(dst + o * row_bytes);
    const int64_t step = (int64_t)gridDim.x * blockDim.x;
    for (int64_t e0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e0 < nv; e0 += step * U) {
      T v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t e = e0 + u * step;
        if constexpr (V == 16) v[u] = __builtin_nontemporal_load(s + (e < nv ? e : 0));
        else v[u] = s[e < nv ? e : 0];
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t e = e0 + u * step;
        if (e < nv) {
          if constexpr (V == 16) __builtin_nontemporal_store(v[u], d + e);
          else d[e] = v[u];
        }
      }
    }
    if (out_rows) {
      for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < rows; r += step)
        out_rows[o + r] = (int32_t)(lo + r);
    }
  }
  if (!out_offs && blockIdx.x == 0 && blockIdx.y == 0) {
    int64_t base = 0;
    for (int32_t i0 = 0; i0 < k; i0 += blockDim.x) {
      const int32_t i = i0 + threadIdx.x;
      int64_t len = 0;
      if (i < k) {
        int64_t lo, hi;
        frame_rows(offs, n_frames, n_rows, sel[i], &lo, &hi);
        len = hi - lo;
      }
      int64_t total;
      const int64_t ex = block_exscan64(len, &total, wsum);
      if (i < k) offs_out[i + 1] = out_offset(base + ex + len);
      base += total;
    }
    if (threadIdx.x == 0) offs_out[0] = 0;
  }
}

// at most this many frames take the one-kernel gather (each workgroup sums
// the row counts before its frame)
constexpr int32_t kGatherFused = 4096;

// Address model of gather_copy_kernel<V> (dry run): the frames' row ranges
// through frame_rows on the host copies of sel and the frame offsets (given
// with cofie_debug_buffer_data), each frame's output position as the kernel
// takes it (the saturated offsets, or the exact prefix when it scans itself),
// the source and destination bytes, the source-row output.
void model_gather(int V, const uint8_t* src, int64_t n_rows, int64_t row_bytes, const int32_t* offs, int32_t n_frames,
                  const int32_t* sel, int32_t k, const uint8_t* dst, int64_t capacity, bool scanned,
                  const int32_t* offs_out, const int32_t* out_rows) {
  const int32_t* sel_h = static_cast<const int32_t*>(dry_shadow(sel));
  const int32_t* offs_h = static_cast<const int32_t*>(dry_shadow(offs));
  if (!sel_h || !offs_h) {
    dry_range(0, 0, 0, "gather: sel or the frame offsets without host contents");
    return;
  }
  dry_range(row_bytes % V, 0, 1, "gather: row size not a multiple of the access");
  dry_access(offs_out, 0, 4 * ((int64_t)k + 1), "gather: output offsets");
  int64_t pre = 0;  // the exact prefix of the clamped row counts
  for (int32_t i = 0; i < k; ++i) {
    dry_access(sel, 4 * (int64_t)i, 4, "gather: sel");
    const int32_t f = sel_h[i];
    if (f >= 0 && f < n_frames) dry_access(offs, 4 * (int64_t)f, 8, "gather: frame offsets");
    int64_t lo, hi;
    frame_rows(offs_h, n_frames, n_rows, f, &lo, &hi);
    const int64_t o = scanned ? out_offset(pre) : pre;
    pre += hi - lo;
    int64_t rows = hi - lo;
    const int64_t room = capacity - o;
    rows = rows < room ? rows : (room > 0 ? room : 0);
    if (rows <= 0) continue;
    dry_access(src, lo * row_bytes, rows * row_bytes, "gather: source rows");
    dry_access(dst, o * row_bytes, rows * row_bytes, "gather: destination rows");
    if (out_rows) dry_access(out_rows, 4 * o, 4 * rows, "gather: source row indices");
  }
}

}  // namespace
}  // namespace cofie

using namespace cofie;

extern "C" {

int cofie_mask_compact(const uint8_t* mask, int64_t n, int64_t segment_len, int32_t* out_idx,
                       int32_t* out_seg_start, void* stream) {
  clear_error();
  if (n < 0 || n >= (int64_t(1) << 31)) return set_error(COFIE_EINVAL, "n = %lld out of range", (long long)n);
  if (segment_len < 0) return set_error(COFIE_EINVAL, "segment_len is negative");
  if (!out_seg_start) return set_error(COFIE_EINVAL, "out_seg_start is NULL");
  if (n > 0 && (!mask || !out_idx)) return set_error(COFIE_EINVAL, "mask or out_idx is NULL");
  const int64_t nseg = segment_len > 0 ? ceil_div(n, segment_len) : 1;
  return launch("glue_mask_compact", mask_compact_kernel, dim3(1), dim3(kGlueThreads), 0,
                static_cast<hipStream_t>(stream), mask, n, segment_len, nseg, out_idx, out_seg_start);
}

int cofie_gather_frames(const void* src, int64_t n_rows, int64_t row_bytes, const int32_t* frame_offsets,
                        int32_t n_frames, const int32_t* sel, int32_t k, void* dst,
                        int64_t dst_capacity_rows, int32_t* out_offsets, int32_t* out_rows, void* stream) {
  clear_error();
  if (n_rows < 0 || n_rows >= (int64_t(1) << 31)) return set_error(COFIE_EINVAL, "n_rows out of range");
  if (row_bytes <= 0) return set_error(COFIE_EINVAL, "row_bytes must be positive");
  if (n_frames < 0 || k < 0 || dst_capacity_rows < 0)
    return set_error(COFIE_EINVAL, "negative n_frames, k or capacity");
  if (dst_capacity_rows >= (int64_t(1) << 31))
    return set_error(COFIE_EINVAL, "dst_capacity_rows = %lld: the output rows are int32 offsets, below 2^31",
                     (long long)dst_capacity_rows);
  if (!out_offsets) return set_error(COFIE_EINVAL, "out_offsets is NULL");
  if (k > 0 && (!sel || !frame_offsets)) return set_error(COFIE_EINVAL, "sel or frame_offsets is NULL");
  if (k > 0 && n_rows > 0 && (!src || (dst_capacity_rows > 0 && !dst)))
    return set_error(COFIE_EINVAL, "src or dst is NULL");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool fused = k > 0 && k <= kGatherFused && n_rows > 0 && dst_capacity_rows > 0;
  if (!fused) {
    int rc = launch("glue_gather_offsets", gather_offsets_kernel, dim3(1), dim3(kGlueThreads), 0, s,
                    frame_offsets, n_frames, n_rows, sel, k, out_offsets);
    if (rc || k == 0 || n_rows == 0 || dst_capacity_rows == 0) return rc;
  }
  const int32_t* offs_in = fused ? nullptr : out_offsets;
  const int cus = device_cu_count();
  const unsigned gy = (unsigned)std::min<int64_t>(k, 65535);
  const unsigned gx = (unsigned)std::max<int64_t>(1, std::min<int64_t>(64, ceil_div(4 * cus, k)));
  const uintptr_t al = reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst) | (uintptr_t)row_bytes;
  const uint8_t* sp = static_cast<const uint8_t*>(src);
  uint8_t* dp = static_cast<uint8_t*>(dst);
  if (dry_run()) {
    model_gather(al % 16 == 0 ? 16 : (al % 4 == 0 ? 4 : 1), sp, n_rows, row_bytes, frame_offsets, n_frames, sel, k, dp,
                 dst_capacity_rows, !fused, out_offsets, out_rows);
    return COFIE_OK;
  }
  if (al % 16 == 0)
    return launch("glue_gather_copy", gather_copy_kernel<16>, dim3(gx, gy), dim3(256), 0, s, sp, n_rows, row_bytes,
                  frame_offsets, n_frames, sel, k, dp, dst_capacity_rows, offs_in, out_offsets, out_rows);
  if (al % 4 == 0)
    return launch("glue_gather_copy", gather_copy_kernel<4>, dim3(gx, gy), dim3(256), 0, s, sp, n_rows, row_bytes,
                  frame_offsets, n_frames, sel, k, dp, dst_capacity_rows, offs_in, out_offsets, out_rows);
  return launch("glue_gather_copy", gather_copy_kernel<1>, dim3(gx, gy), dim3(256), 0, s, sp, n_rows, row_bytes,
                frame_offsets, n_frames, sel, k, dp, dst_capacity_rows, offs_in, out_offsets, out_rows);
}

}  // extern "C"

// NGFF -- Novelty-Guided Frame Filtering (Sec. 3.2) on gfx950.
//
// Pipeline of one cofie_ngff_filter call (all on the caller's stream):
//   [fill]     zero the histogram when several workgroups share a frame
//   hist       streaming histogram: 12-byte coalesced loads (64 lanes x 12 B =
//              768 contiguous bytes per wave instruction), byte -> bin in
//              registers, increments into 64 lane-private LDS copies laid out
//              bin-major ([bin][lane]) so that the lanes of one instruction
//              always hit 64 distinct banks; one merge per workgroup
//   band_keep  exact integer L1 distances D(t, t-k), 1 <= k <= L_max, from
//              histogram rows staged in LDS (each row computed once), and per
//              frame t one word whose bit k says whether t would be kept by
//              novelty if t-k were the last kept frame (that depends only on
//              the band and theta)
//   select     one workgroup per stream: next[r] (the frame kept after r)
//              from those words, the keep chain from frame 0 by pointer
//              doubling inside 64-frame windows and a walk across windows,
//              the M_min top-up, scores, mask and counts
// With L_max > 31 or histogram rows too wide for LDS, the band, next[] and
// the selection run as separate kernels (band from global memory).
// Without the gap rule (L_max <= 0) a sequential kernel per stream measures
// D(t, r(t)) directly.
// Novelty comparisons run on integers: s >= tau  <=>  max(D) >= theta with
// theta = min{D : score(D) >= tau}, exact because the score, D / 2M rounded
// once to fp32, never decreases in D.  Scores are that correctly rounded
// quotient (one IEEE division of exact operands for 2M < 2^24; an fp64
// quotient and an exact midpoint test beyond), so they are bit-identical to
// any correct implementation.
#include <cstring>
#include <vector>
#include "common.h"

namespace cofie {
namespace {

constexpr int kUnitBytes = 768;  // one wave-wide load: 64 lanes x 12 bytes
constexpr int kUnroll = 3;       // units per batch and wave (two batches in flight)

enum HistKind { K_PC = 0, K_GRAY1 = 1, K_GRAY3 = 2, K_JOINT = 3 };

struct HistArgs {
  const uint8_t* frames;
  int64_t frame_bytes;
  int64_t npix;
  uint32_t* hist;
  int32_t nbins;
  int32_t B;
  int32_t shift;  // 8 - log2(B): bin = v >> shift
  int32_t logB;
  int32_t splits; // workgroups per frame
  int32_t units;  // whole 768-byte units covered by the vector path
  int32_t atomic; // 1: several workgroups per frame add into a zeroed histogram
  // frame t of the launch reads frame (t / group) * in_stride + in_off + t % group
  // and writes histogram row (t / group) * out_stride + out_off + t % group;
  // group = 0: frame t, row t
  int64_t group, in_stride, in_off, out_stride, out_off;
};

struct __attribute__((packed, aligned(4))) U3 {
  uint32_t x, y, z;
};

__device__ __forceinline__ uint32_t luma_bt601(uint32_t r, uint32_t g, uint32_t b) {
  return (299u * r + 587u * g + 114u * b + 500u) / 1000u;
}

// Bin of one pixel for the pixel-wise kinds (GRAY of RGB, JOINT3D).
template <int KIND, int BC>
__device__ __forceinline__ uint32_t pixel_bin(uint32_t r, uint32_t g, uint32_t b, const HistArgs& a) {
  const int shift = BC ? (8 - __builtin_ctz(BC)) : a.shift;
  const int logB = BC ? __builtin_ctz(BC) : a.logB;
  if constexpr (KIND == K_GRAY3) {
    return luma_bt601(r, g, b) >> shift;
  } else {
    return ((r >> shift) << (2 * logB)) | ((g >> shift) << logB) | (b >> shift);
  }
}

// Count the 12 bytes one lane loaded (4 RGB pixels, or 12 gray pixels).
template <int KIND, int P, int BC>
__device__ __forceinline__ void count12(uint32_t* cnt, const U3& v, uint32_t lane, const HistArgs& a) {
  const uint32_t w[3] = {v.x, v.y, v.z};
  const uint32_t copy = lane & (P - 1);
  if constexpr (KIND == K_PC || KIND == K_GRAY1) {
    if constexpr (P == 64 && BC != 0) {
      // bins of 4 bytes at once, then byte-permute each bin into bits 8..15 of
      // an LDS byte address whose low byte is lane*4: bin*256 + lane*4.  The
      // channel (byte position mod 3, fixed because lanes read 12-byte pixel-
      // aligned chunks) becomes a constant offset of c*B rows.
      constexpr int shift = 8 - __builtin_ctz(BC);
      constexpr uint32_t m4 = (uint32_t)(BC - 1) * 0x01010101u;
      const uint32_t lane4 = lane * 4u;
#pragma unroll
      for (int j = 0; j < 3; ++j) {
        const uint32_t tb = (w[j] >> shift) & m4;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int c = (KIND == K_PC) ? ((4 * j + i) % 3) : 0;
          const uint32_t addr = __builtin_amdgcn_perm(tb, lane4, 0x0C0C0000u | ((4u + i) << 8));
          atomicAdd(reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(cnt) + addr) + c * BC * 64, 1u);
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < 3; ++j) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int c = (KIND == K_PC) ? ((4 * j + i) % 3) : 0;
          const uint32_t bin = ((w[j] >> (8 * i)) & 0xFFu) >> a.shift;
          atomicAdd(cnt + (bin + (uint32_t)(c * a.B)) * P + copy, 1u);
        }
      }
    }
  } else {
    uint32_t byte[12];
#pragma unroll
    for (int k = 0; k < 12; ++k) byte[k] = (w[k >> 2] >> (8 * (k & 3))) & 0xFFu;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const uint32_t bin = pixel_bin<KIND, BC>(byte[3 * p], byte[3 * p + 1], byte[3 * p + 2], a);
      atomicAdd(cnt + bin * P + copy, 1u);
    }
  }
}

// One pixel read byte by byte (ragged tails and unaligned frames).
template <int KIND, int P, int BC>
__device__ __forceinline__ void count_pixel(uint32_t* cnt, const uint8_t* px, uint32_t lane,
                                            const HistArgs& a) {
  const uint32_t copy = lane & (P - 1);
  if constexpr (KIND == K_GRAY1) {
    atomicAdd(cnt + (uint32_t)(px[0] >> a.shift) * P + copy, 1u);
  } else if constexpr (KIND == K_PC) {
#pragma unroll
    for (int c = 0; c < 3; ++c)
      atomicAdd(cnt + ((uint32_t)(px[c] >> a.shift) + (uint32_t)(c * a.B)) * P + copy, 1u);
  } else {
    atomicAdd(cnt + pixel_bin<KIND, BC>(px[0], px[1], px[2], a) * P + copy, 1u);
  }
}

// Frame (or histogram row) of launch frame t under the map of HistArgs.
__host__ __device__ __forceinline__ int64_t hist_map(int64_t t, int64_t group, int64_t stride, int64_t off) {
  return group ? (t / group) * stride + off + t % group : t;
}
// Unit that wave g (of G sharing a frame) loads as the i-th of its batches'
// units: g + i G, clamped to the last whole unit.
__host__ __device__ __forceinline__ int hist_unit(int g, int i, int G, int units) {
  const int u = g + i * G;
  return u < units ? u : units - 1;
}

// grid: n * splits workgroups; workgroup (t, s) counts its share of frame t.
template <int KIND, int P, int BC>
__global__ __launch_bounds__(512) void ngff_hist_kernel(HistArgs a) {
  extern __shared__ uint32_t cnt[];  // [nbins][P]
  const int tid = threadIdx.x, nthr = blockDim.x;
  const uint32_t lane = tid & 63;
  const int wave = tid >> 6, nw = nthr >> 6;
  const int64_t t = blockIdx.x / a.splits;
  const int s = (int)(blockIdx.x - t * a.splits);
  const int64_t src_frame = hist_map(t, a.group, a.in_stride, a.in_off);
  const int64_t dst_row = hist_map(t, a.group, a.out_stride, a.out_off);
  const uint8_t* f = a.frames + src_frame * a.frame_bytes;
  const int G = a.splits * nw;  // waves sharing this frame
  const int g = s * nw + wave;
  // batches of kUnroll units per wave (unit u0 + j G), software pipelined: the
  // next batch is in flight while this one is counted.  Loads are
  // unconditional from clamped units (a repeated unit is in cache and is not
  // counted); the two register sets alternate without copies.
  const int nbatch = g < a.units ? (a.units - g + G * kUnroll - 1) / (G * kUnroll) : 0;
  auto load_batch = [&](U3 (&v)[kUnroll], int b) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < kUnroll; ++j) {
      const int u = hist_unit(g, b * kUnroll + j, G, a.units);
      // frames are read once: non-temporal loads (1 fps stream 28.0 -> 26.4 us,
      // high-res 1031 -> 938 us)
      const uint32_t* src = reinterpret_cast<const uint32_t*>(f + (int64_t)u * kUnitBytes + lane * 12);
      v[j].x = __builtin_nontemporal_load(src);
      v[j].y = __builtin_nontemporal_load(src + 1);
      v[j].z = __builtin_nontemporal_load(src + 2);
    }
  };
  auto count_batch = [&](const U3 (&v)[kUnroll], int b) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < kUnroll; ++j)
      if (g + (b * kUnroll + j) * G < a.units) count12<KIND, P, BC>(cnt, v[j], lane, a);
  };
  // the first batch is issued before the counters are cleared; the barrier
  // orders LDS only, so it does not wait for those loads
  U3 va[kUnroll], vb[kUnroll];
  if (nbatch > 0) load_batch(va, 0);
  const int ncnt = a.nbins * P;
  for (int i = tid; i < ncnt; i += nthr) cnt[i] = 0;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
  if (nbatch > 0) {
    int b = 0;
    for (; b + 2 <= nbatch; b += 2) {
      load_batch(vb, b + 1);
      count_batch(va, b);
      load_batch(va, b + 2);
      count_batch(vb, b + 1);
    }
    if (b < nbatch) count_batch(va, b);
  }
  // pixels after the whole units (or every pixel of an unaligned frame)
  const int C = (KIND == K_GRAY1) ? 1 : 3;
  const int64_t p0 = (int64_t)a.units * (kUnitBytes / C);
  for (int64_t p = p0 + (int64_t)g * 64 + lane; p < a.npix; p += (int64_t)G * 64)
    count_pixel<KIND, P, BC>(cnt, f + p * C, lane, a);
  __syncthreads();

  // merge the P lane copies: J threads per bin each add P/J copies (rotated by
  // the bin so that the lanes of a wave hit distinct banks), then combine
  constexpr int J = P >= 8 ? 8 : P;
  constexpr int PER = P / J;
  uint32_t* out = a.hist + dst_row * a.nbins;
  const int bins_per_pass = nthr / J;
  const int j = tid % J;
  for (int b0 = 0; b0 < a.nbins; b0 += bins_per_pass) {
    const int b = b0 + tid / J;
    uint32_t sum = 0;
    if (b < a.nbins) {
#pragma unroll
      for (int i = 0; i < PER; ++i) sum += cnt[b * P + ((j * PER + i + b) & (P - 1))];
    }
#pragma unroll
    for (int o = J / 2; o > 0; o >>= 1) sum += __shfl_xor(sum, o, J);
    if (j == 0 && b < a.nbins) {
      if (a.atomic) {
        if (sum) atomicAdd(out + b, sum);
      } else {
        out[b] = sum;
      }
    }
  }
}

__global__ void fill_u32_kernel(uint32_t* p, uint32_t v, int64_t count) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// ---- alternative signals (Table 5): low-res frame difference, dHash -----------------
// The luma image box-averaged on a gh x gw grid (row y in grid row
// (y gh) div H, column x in (x gw) div W), each cell's mean rounded half up;
// the frame difference emits the gh gw means, dHash the 64 bits "cell
// (r, c+1) brighter than cell (r, c)" of an 8 x 9 grid.  The rows' L1 distance
// over 255 gh gw (or 64) is the signal's distance, so the keep rule runs on
// them like on histogram rows.  One workgroup per frame: each wave takes whole
// image rows, each lane 4 consecutive pixels per load (12 contiguous bytes:
// 768 per wave instruction when the frame allows it), sums a run of pixels of
// one cell in registers and adds it to the cell's LDS counter.
struct SigArgs {
  const uint8_t* frames;
  int64_t frame_bytes;
  int32_t H, W, C;
  int32_t gh, gw;
  int32_t dhash;  // 1: the 64 hash bits, 0: the gh gw cell means
  int32_t nsig;
  int32_t vec;    // 1: 4-pixel loads (4-byte aligned frames, W a multiple of 4)
  uint32_t* out;  // [n][nsig]
};

constexpr int kSigThreads = 256;
constexpr int kSigMaxW = 16384;  // the column -> grid column table (uint16, LDS)

__global__ __launch_bounds__(kSigThreads) void ngff_sig_kernel(SigArgs a) {
  __shared__ uint32_t cell[4096];
  __shared__ uint16_t gcol[kSigMaxW];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nw = kSigThreads / 64;
  const int ncell = a.gh * a.gw;
  for (int i = tid; i < ncell; i += kSigThreads) cell[i] = 0;
  for (int x = tid; x < a.W; x += kSigThreads) gcol[x] = (uint16_t)(((int64_t)x * a.gw) / a.W);
  __syncthreads();
  const uint8_t* f = a.frames + (int64_t)blockIdx.x * a.frame_bytes;
  auto luma = [&](uint32_t r, uint32_t g, uint32_t b) __attribute__((always_inline)) {
    return a.C == 3 ? luma_bt601(r, g, b) : r;
  };
  for (int y = wave; y < a.H; y += nw) {
    const int cy = (int)(((int64_t)y * a.gh) / a.H) * a.gw;
    const uint8_t* row = f + (int64_t)y * a.W * a.C;
    if (a.vec) {
      // lane: pixels x0 .. x0 + 3 (12 bytes of RGB or 4 bytes of gray)
      for (int x0 = 4 * lane; x0 < a.W; x0 += 256) {
        uint32_t v[4];
        if (a.C == 3) {
          const U3 w = *reinterpret_cast<const U3*>(row + 3 * x0);
          v[0] = luma(w.x & 255u, (w.x >> 8) & 255u, (w.x >> 16) & 255u);
          v[1] = luma(w.x >> 24, w.y & 255u, (w.y >> 8) & 255u);
          v[2] = luma((w.y >> 16) & 255u, w.y >> 24, w.z & 255u);
          v[3] = luma((w.z >> 8) & 255u, (w.z >> 16) & 255u, w.z >> 24);
        } else {
          const uint32_t w = *reinterpret_cast<const uint32_t*>(row + x0);
#pragma unroll
          for (int i = 0; i < 4; ++i) v[i] = (w >> (8 * i)) & 255u;
        }
        // runs of one cell: one LDS add per run
        int c = gcol[x0];
        uint32_t run = v[0];
#pragma unroll
        for (int i = 1; i < 4; ++i) {
          const int ci = gcol[x0 + i];
          if (ci != c) {
            atomicAdd(&cell[cy + c], run);
            c = ci;
            run = 0;
          }
          run += v[i];
        }
        atomicAdd(&cell[cy + c], run);
      }
    } else {
      for (int x = lane; x < a.W; x += 64) {
        const uint8_t* px = row + (int64_t)x * a.C;
        const uint32_t v = a.C == 3 ? luma_bt601(px[0], px[1], px[2]) : px[0];
        atomicAdd(&cell[cy + gcol[x]], v);
      }
    }
  }
  __syncthreads();
  // cell means, rounded half up: grid row i spans rows [ceil(i H / gh),
  // ceil((i + 1) H / gh)), grid column j likewise
  auto first = [](int64_t i, int64_t len, int64_t g) __attribute__((always_inline)) { return (i * len + g - 1) / g; };
  for (int i = tid; i < ncell; i += kSigThreads) {
    const int r = i / a.gw, c = i - r * a.gw;
    const uint32_t area = (uint32_t)((first(r + 1, a.H, a.gh) - first(r, a.H, a.gh)) *
                                     (first(c + 1, a.W, a.gw) - first(c, a.W, a.gw)));
    cell[i] = (cell[i] + area / 2) / area;
  }
  __syncthreads();
  uint32_t* o = a.out + (int64_t)blockIdx.x * a.nsig;
  if (a.dhash) {
    if (tid < 64) {
      const int r = tid >> 3, c = tid & 7;
      o[tid] = cell[r * 9 + c + 1] > cell[r * 9 + c] ? 1u : 0u;
    }
  } else {
    for (int i = tid; i < ncell; i += kSigThreads) o[i] = cell[i];
  }
}

// ---- band of distances ----------------------------------------------------------
struct BandArgs {
  const uint32_t* hist;
  int64_t n;
  int32_t nbins;
  int32_t L;       // band width (>= 1)
  int64_t seg_len; // frames per stream
  int32_t TB;      // frames per workgroup
  int32_t stride;  // LDS row stride in words (nbins + 1), 0 = read global memory
  int32_t* band;   // [n][L]: band[t*L + k-1] = D(t, t-k), 0 if t-k precedes the stream
  // when window != null, the first wrows rows of every stream are read from
  // window[stream][row] ([n / seg_len][wrows][nbins]) instead of hist
  const uint32_t* window;
  int32_t wrows;
};

__device__ __forceinline__ const uint32_t* band_row(const BandArgs& a, int64_t r) {
  if (a.window) {
    const int64_t sg = r / a.seg_len, q = r - sg * a.seg_len;
    if (q < a.wrows) return a.window + (sg * a.wrows + q) * a.nbins;
  }
  return a.hist + r * a.nbins;
}

__global__ __launch_bounds__(256) void ngff_band_kernel(BandArgs a) {
  extern __shared__ uint32_t rows[];
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int64_t t0 = (int64_t)blockIdx.x * a.TB;
  const int64_t r0 = t0 - a.L > 0 ? t0 - a.L : 0;
  const int64_t r1 = t0 + a.TB < a.n ? t0 + a.TB : a.n;
  if (a.stride) {
    // all loads of a batch are issued before their stores (clamped indices)
    const int64_t total = (r1 - r0) * a.nbins;
    constexpr int V = 8;
    for (int64_t i0 = tid; i0 < total; i0 += (int64_t)V * nthr) {
      uint32_t v[V];
      int64_t idx[V];
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const int64_t i = i0 + (int64_t)j * nthr;
        idx[j] = i < total ? i : 0;
        const int64_t r = idx[j] / a.nbins;
        v[j] = band_row(a, r0 + r)[idx[j] - r * a.nbins];
      }
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const int64_t r = idx[j] / a.nbins;
        rows[r * a.stride + (idx[j] - r * a.nbins)] = v[j];
      }
    }
    __syncthreads();
  }
  // (row, lag) pairs, LPP lanes per pair (a power of two <= 64: a group never
  // straddles a wave), bins strided over the group, combined with shuffles
  const int npairs = (int)(r1 - t0) * a.L;
  int LPP = 1;
  while (LPP < 64 && 2 * LPP * npairs <= nthr) LPP <<= 1;
  const int sub = tid & (LPP - 1), groups = nthr / LPP;
  const int passes = (npairs + groups - 1) / groups;  // whole passes: every lane runs the shuffles
  for (int ps = 0; ps < passes; ++ps) {
    const int pi = ps * groups + tid / LPP;
    const bool ok = pi < npairs;
    const int64_t t = t0 + (ok ? pi / a.L : 0);
    const int k = ok ? pi % a.L + 1 : 1;
    const int64_t seg0 = (t / a.seg_len) * a.seg_len;
    uint32_t D = 0;
    if (ok && t - k >= seg0) {
      const uint32_t* x;
      const uint32_t* y;
      if (a.stride) {
        x = rows + (t - r0) * a.stride;
        y = rows + (t - k - r0) * a.stride;
      } else {
        x = band_row(a, t);
        y = band_row(a, t - k);
      }
      for (int b = sub; b < a.nbins; b += LPP) {
        const uint32_t u = x[b], v = y[b];
        D += u > v ? u - v : v - u;
      }
    }
    for (int o = 1; o < LPP; o <<= 1) D += __shfl_xor(D, o, LPP);
    if (ok && sub == 0) a.band[t * a.L + (k - 1)] = (int32_t)D;
  }
}

// The score of an integer distance D: D / 2M rounded once to the nearest
// fp32 (ties to even).  For 2M < 2^24 both operands are exact in fp32 and one
// IEEE division gives it.  Beyond (frames above ~2.8 MP per channel, up to
// 2M < 2^31): q = D / 2M in fp64 (exact operands, one rounding) rounded to
// fp32 is within one fp32 ulp of the answer; the answer is decided by the
// exact sign of (midpoint * 2M - D) for the midpoints between q's fp32 value
// and its neighbours (one FMA each: the product of a 25-bit midpoint and a
// 31-bit integer is exact before FMA's single rounding, which keeps the sign).
__device__ __forceinline__ float score_of(int64_t D, int64_t twoM) {
  if (twoM < (int64_t(1) << 24)) return (float)(int32_t)D / (float)(int32_t)twoM;
  if (D <= 0) return 0.f;
  const double N = (double)twoM, x = (double)D;
  const float f = (float)(x / N);
  const uint32_t b = __float_as_uint(f);
  const float lo = __uint_as_float(b - 1), hi = __uint_as_float(b + 1);
  const double s_hi = fma(0.5 * ((double)f + (double)hi), N, -x);  // > 0: D/2M below the upper midpoint
  if (s_hi < 0) return hi;
  if (s_hi == 0) return (b & 1u) ? hi : f;
  const double s_lo = fma(0.5 * ((double)lo + (double)f), N, -x);
  if (s_lo > 0) return lo;
  if (s_lo == 0) return (b & 1u) ? lo : f;
  return f;
}

// Smallest integer D in [0, 2M+1] with score_of(D) >= tau, or 2M+2 if none
// (NaN tau, or tau above the score of 2M+1).  For 2M < 2^24: with y = tau * 2M
// (exact in fp64: a 24-bit mantissa times an integer below 2^24) every D >= y
// passes and, because 1/2M exceeds half an fp32 ulp of tau, every D <= y - 1
// fails; so the answer is ceil(y) or ceil(y) - 1 and one exact IEEE test
// decides (straight-line code).  Beyond, a binary search: score_of never
// decreases in D.
__device__ int64_t theta_of(float tau, int64_t twoM) {
  const float den = (float)twoM;
  if (!(tau == tau)) return twoM + 2;
  if (tau <= 0.f) return 0;
  if (twoM >= (int64_t(1) << 24)) {
    int64_t lo = 0, hi = twoM + 2;  // answer in [lo, hi]; hi = none
    while (lo < hi) {
      const int64_t mid = lo + (hi - lo) / 2;
      if (score_of(mid, twoM) >= tau) hi = mid;
      else lo = mid + 1;
    }
    return lo;
  }
  const double y = (double)tau * (double)twoM;
  if (y > (double)(twoM + 1))
    return ((float)(int32_t)(twoM + 1) / den >= tau) ? twoM + 1 : twoM + 2;
  const int64_t x = (int64_t)ceil(y);
  if (x >= 1 && (float)(int32_t)(x - 1) / den >= tau) return x - 1;
  return x;
}

struct RuleArgs {
  const int32_t* band;
  int64_t n;
  int64_t seg_len;
  int32_t L;
  int32_t M_min;
  int64_t twoM;
  float tau;
  const float* tau_seg;  // device, may be null
};

__device__ __forceinline__ float tau_of_segment(const RuleArgs& a, int64_t seg) {
  return a.tau_seg ? a.tau_seg[seg] : a.tau;
}

// next[r] (segment-relative): first u in (r, r+L] that the rule keeps when r is
// the last kept frame: u is the stream's last frame, or u - r >= L, or
// max(D(u,u-1), D(u,r)) >= theta.  The stream's last frame gets T.
__global__ void ngff_next_kernel(RuleArgs a, int32_t* next) {
  const int64_t r = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (r >= a.n) return;
  const int64_t seg = r / a.seg_len, s0 = seg * a.seg_len;
  const int64_t T = a.n - s0 < a.seg_len ? a.n - s0 : a.seg_len;
  const int64_t rr = r - s0;
  if (rr == T - 1) {
    next[r] = (int32_t)T;
    return;
  }
  const int64_t theta = theta_of(tau_of_segment(a, seg), a.twoM);
  int64_t u = rr + 1;
  for (int k = 1;; ++k, ++u) {
    if (u == T - 1 || k >= a.L) break;
    const int32_t* row = a.band + (s0 + u) * a.L;
    const int32_t Dadj = row[0], Dref = row[k - 1];
    if ((Dadj > Dref ? Dadj : Dref) >= theta) break;
  }
  next[r] = (int32_t)u;
}

// Block-wide sum of v (blockDim.x a multiple of 64, <= 1024).
__device__ int64_t block_sum(int64_t v, int64_t* red) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  int64_t s = 0;
  for (int i = 0; i < nw; ++i) s += red[i];
  __syncthreads();
  return s;
}

// Block-wide inclusive prefix maximum (blockDim a multiple of 64, <= 1024).
__device__ int block_inclusive_max(int v, int* wtmp) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x = x > y ? x : y;
  }
  if (lane == 63) wtmp[wave] = x;
  __syncthreads();
  int before = -1;
  for (int i = 0; i < wave; ++i) before = before > wtmp[i] ? before : wtmp[i];
  __syncthreads();
  return x > before ? x : before;
}

// Selection of one stream by one workgroup (1024 threads), in chunks of C
// frames (a multiple of 64; the whole stream when it fits):
//  1. stage(c0, c1, nx) writes next[r] (stream-relative) for r in [c0, c1)
//     into LDS;
//  2. windows of 64 frames, one wave each: lane l starts at frame w + l, and
//     six rounds of pointer doubling over the lanes (shuffles) give, for every
//     lane, the mask of the chain frames inside the window reached from it and
//     the first chain frame past the window (its exit);
//  3. one thread follows the chain across windows: the entry of window i is
//     the exit of window i-1's entry, so its kept frames are the entry's mask;
//  4. every thread finishes the chunk's frames: r(t) = the highest kept frame
//     below t in its window's mask, else the last kept frame before the
//     window; score = max(D(t,t-1), D(t,r(t))) / 2M from the band; mask bit.
// Then, if fewer than M_min frames were kept, the top-up frames are added
// (they never become r, so scores stay as they are).  LDS: next [C] ints,
// marks [C] u64, window masks [C/64] u64, last kept before window [C/64].
template <typename StageFn>
__device__ void select_walk(const RuleArgs& a, int64_t seg, int C, StageFn stage, int32_t* nx, uint64_t* mk,
                            uint64_t* kmask, int32_t* lastb, const int32_t* adj_g, float* scores, uint8_t* mask,
                            int32_t* count) {
  __shared__ int64_t red[16];
  __shared__ int32_t walk_sh[3];  // carried entry frame, last kept frame, kept count
  constexpr int U = 4;            // frames per thread and batch of the finishing pass
  const int64_t s0 = seg * a.seg_len;
  const int T = (int)(a.n - s0 < a.seg_len ? a.n - s0 : a.seg_len);
  const int tid = threadIdx.x, nthr = blockDim.x, lane = tid & 63, wave = tid >> 6, nw = nthr >> 6;
  const int32_t* band = a.band + s0 * a.L;
  const int32_t* adj = adj_g ? adj_g + s0 : nullptr;  // D(t, t-1), contiguous
  if (tid == 0) {
    walk_sh[0] = 0;
    walk_sh[1] = -1;
    walk_sh[2] = 0;
  }
  for (int c0 = 0; c0 < T; c0 += C) {
    const int c1 = c0 + C < T ? c0 + C : T;
    const int nwin = (c1 - c0 + 63) >> 6;
    stage(c0, c1, nx);
    __syncthreads();
    for (int wi = wave; wi < nwin; wi += nw) {
      const int w = c0 + (wi << 6), f = w + lane;
      int J = f < c1 ? nx[f - c0] - w : 64;  // >= 64: past the window
      uint64_t M = f < c1 ? 1ull << lane : 0ull;
#pragma unroll
      for (int rnd = 0; rnd < 6; ++rnd) {
        const bool in = J < 64;
        const int src = in ? J : lane;
        const uint32_t lo = (uint32_t)__shfl((int)(uint32_t)M, src), hi = (uint32_t)__shfl((int)(uint32_t)(M >> 32), src);
        const int Jo = __shfl(J, src);
        if (in) {
          M |= ((uint64_t)hi << 32) | lo;
          J = Jo;
        }
      }
      if (f < c1) {
        mk[f - c0] = M;
        nx[f - c0] = w + J;  // exit frame
      }
    }
    __syncthreads();
    if (tid == 0) {
      // the chain across windows: the entry of window i is the exit of window
      // i-1's entry (one thread; a few windows per stream)
      int e = walk_sh[0], last = walk_sh[1], kept = walk_sh[2];
      for (int wi = 0; wi < nwin; ++wi) {
        const int w = c0 + (wi << 6);
        lastb[wi] = last;
        uint64_t m = 0;
        if (e < w + 64 && e < T) {
          m = mk[e - c0];
          last = w + 63 - __builtin_clzll(m);
          kept += __builtin_popcountll(m);
          e = nx[e - c0];
        }
        kmask[wi] = m;
      }
      walk_sh[0] = e;
      walk_sh[1] = last;
      walk_sh[2] = kept;
    }
    __syncthreads();
    for (int base = c0; base < c1; base += U * nthr) {
      int32_t Da[U], Dr[U];
      bool kp[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        int t = base + u * nthr + tid;
        t = t < c1 ? t : c1 - 1;
        const int wi = (t - c0) >> 6, bit = (t - c0) & 63;
        const uint64_t m = kmask[wi];
        const uint64_t below = m & ((1ull << bit) - 1);
        const int r = below ? c0 + (wi << 6) + 63 - __builtin_clzll(below) : lastb[wi];
        kp[u] = (m >> bit) & 1;
        const int32_t* row = band + (int64_t)t * a.L;
        Da[u] = adj ? adj[t] : row[0];
        Dr[u] = row[t > 0 ? t - r - 1 : 0];  // t - r <= L: the gap rule bounds every jump
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int t = base + u * nthr + tid;
        if (t < c1) {
          mask[s0 + t] = kp[u];
          scores[s0 + t] = t > 0 ? score_of(Da[u] > Dr[u] ? Da[u] : Dr[u], a.twoM) : 1.0f;
        }
      }
    }
    __syncthreads();  // the next chunk reuses the LDS arrays
  }
  const int K = walk_sh[2];
  int64_t added = 0;
  if (a.M_min >= 2 && K < a.M_min) {
    // top-up: the frames floor(i (T-1) / (M_min-1)), i < M_min (non-decreasing
    // in i; each distinct frame not kept yet is added once)
    wait_vmem();  // this wave's mask stores have completed
    __syncthreads();
    for (int64_t i = tid; i < a.M_min; i += nthr) {
      const int64_t u = (i * (T - 1)) / (a.M_min - 1);
      const bool first = i == 0 || ((i - 1) * (T - 1)) / (a.M_min - 1) != u;
      added += first && mask[s0 + u] == 0;
    }
    __syncthreads();
    for (int64_t i = tid; i < a.M_min; i += nthr) mask[s0 + (i * (T - 1)) / (a.M_min - 1)] = 1;
  }
  const int64_t total = K + block_sum(added, red);
  if (count && tid == 0) count[seg] = (int32_t)total;
}

// LDS bytes of select_walk's arrays for chunks of C frames (plus the
// keep-test words of [c0, c1 + 32) when next[] is formed from them).
__host__ __device__ constexpr size_t select_lds(int C, bool from_words) {
  return (size_t)C * 12 + (size_t)(C / 64) * 12 + (from_words ? (size_t)(C + 32) * 4 : 0) + 64;
}

// One workgroup per stream.  FROM_WORDS: next[r] is the first k <
// min(L, T-1-r) with bit k of the keep-test word G[r+k] set, else that bound
// (the gap rule or the last frame); otherwise next[] is read from next_g.
template <bool FROM_WORDS>
__global__ __launch_bounds__(1024) void ngff_select_kernel(RuleArgs a, const uint32_t* G, const int32_t* next_g,
                                                           const int32_t* adj, int32_t C, float* scores,
                                                           uint8_t* mask, int32_t* count) {
  extern __shared__ __align__(16) int32_t lds_i[];
  const int64_t seg = blockIdx.x, s0 = seg * a.seg_len;
  const int T = (int)(a.n - s0 < a.seg_len ? a.n - s0 : a.seg_len);
  uint64_t* mk = reinterpret_cast<uint64_t*>(lds_i);
  uint64_t* kmask = mk + C;
  int32_t* nx = reinterpret_cast<int32_t*>(kmask + C / 64);
  int32_t* lastb = nx + C;
  uint32_t* gs = reinterpret_cast<uint32_t*>(lastb + C / 64);  // FROM_WORDS: G of [c0, c1 + 32)
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int L = a.L;
  auto stage = [&](int c0, int c1, int32_t* dst) __attribute__((always_inline)) {
    if constexpr (FROM_WORDS) {
      const int ce = c1 + 32 < T ? c1 + 32 : T;
      constexpr int V = 4;  // loads in flight per thread
      for (int t0 = c0 + tid; t0 < ce; t0 += V * nthr) {
        uint32_t v[V];
#pragma unroll
        for (int j = 0; j < V; ++j) {
          const int t = t0 + j * nthr;
          v[j] = G[s0 + (t < ce ? t : c0)];
        }
#pragma unroll
        for (int j = 0; j < V; ++j) {
          const int t = t0 + j * nthr;
          if (t < ce) gs[t - c0] = v[j];
        }
      }
      __syncthreads();
      for (int r = c0 + tid; r < c1; r += nthr) {
        const int kmax = L < T - 1 - r ? L : T - 1 - r;  // keep at r + kmax at the latest
        int found = kmax;
        // words read 8 at a time (entries past the staged ones are never
        // used: k < kmax keeps r + k < T - 1)
        for (int k0 = 1; k0 < kmax && found == kmax; k0 += 8) {
          uint32_t hit = 0;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int k = k0 + j;
            hit |= (uint32_t)(k < kmax && ((gs[r + k - c0] >> k) & 1u)) << j;
          }
          if (hit) found = k0 + __builtin_ctz(hit);
        }
        dst[r - c0] = r == T - 1 ? T : r + found;
      }
    } else {
      for (int t = c0 + tid; t < c1; t += nthr) dst[t - c0] = next_g[s0 + t];
    }
  };
  select_walk(a, seg, C, stage, nx, mk, kmask, lastb, adj, scores, mask, count);
}

// Band rows and keep-test words (L_max <= 31).  Workgroup b owns frames
// [t0, t0+TB): it stages histogram rows [t0-L, t0+TB) transposed in LDS
// ([bin][row]), computes the band rows D(t, t-k) of its frames (lanes split
// the (row, lag) pairs and the bins), and packs the keep tests each row
// decides into one word: bit k of G[t] is set when, with r = t-k the last
// kept frame, the rule keeps t by novelty (max(D(t,t-1), D(t,r)) >= theta,
// t-k in t's stream).
struct BandKeepArgs {
  const uint32_t* hist;
  int64_t n;
  int32_t nbins;
  int32_t TB;       // frames per workgroup
  int32_t RS;       // LDS row stride (words) of the staged rows, >= TB + L
  RuleArgs rule;
  int32_t* band;    // [n][L]
  int32_t* adj;     // [n] D(t, t-1) (the band's first column, contiguous)
  uint32_t* G;      // [n] keep-test words
};

__global__ __launch_bounds__(1024) void ngff_band_keep_kernel(BandKeepArgs a) {
  extern __shared__ __align__(16) uint32_t sm[];
  const RuleArgs& ru = a.rule;
  const int L = ru.L;
  const int64_t n = a.n, seg_len = ru.seg_len;
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int64_t t0 = (int64_t)blockIdx.x * a.TB;
  const int64_t t1 = t0 + a.TB < n ? t0 + a.TB : n;
  const int64_t r0 = t0 - L > 0 ? t0 - L : 0;  // histogram rows [r0, t1)
  const int RS = a.RS;
  uint32_t* rows = sm;                                                  // [nbins][RS]
  int32_t* bl = reinterpret_cast<int32_t*>(sm + (size_t)a.nbins * RS);  // [TB][L]
  {
    // rows [r0, t1) are contiguous in global memory; all loads are issued
    // before any store (indices past the end are clamped to 0 and rewrite
    // element 0 with its own value)
    const int total = (int)(t1 - r0) * a.nbins;
    const uint32_t* src = a.hist + r0 * a.nbins;
    constexpr int V = 8;
    for (int i0 = tid; i0 < total; i0 += V * nthr) {
      uint32_t v[V];
      int idx[V];
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const int i = i0 + j * nthr;
        idx[j] = i < total ? i : 0;
        v[j] = src[idx[j]];
      }
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const int r = idx[j] / a.nbins, b = idx[j] - r * a.nbins;
        rows[b * RS + r] = v[j];
      }
    }
  }
  __syncthreads();
  // band: (row, lag) pairs, LPP lanes per pair (a power of two <= 64, so a
  // group never straddles a wave), bins strided over the group
  const int npairs = (int)(t1 - t0) * L;
  int LPP = 1;
  while (LPP < 64 && 2 * LPP * npairs <= nthr) LPP <<= 1;
  const int sub = tid & (LPP - 1);
  const int groups = nthr / LPP;
  const int passes = (npairs + groups - 1) / groups;  // whole passes: every lane runs the shuffles
  for (int ps = 0; ps < passes; ++ps) {
    const int pi = ps * groups + tid / LPP;
    const bool ok = pi < npairs;
    const int64_t t = t0 + (ok ? pi / L : 0);
    const int k = ok ? pi % L + 1 : 1;
    const int64_t seg0 = (t / seg_len) * seg_len;
    uint32_t D = 0;
    if (ok && t - k >= seg0) {
      const uint32_t* x = rows + (t - r0);
      const uint32_t* y = rows + (t - k - r0);
      for (int b = sub; b < a.nbins; b += LPP) {
        const uint32_t u = x[b * RS], v = y[b * RS];
        D += u > v ? u - v : v - u;
      }
    }
    for (int o = 1; o < LPP; o <<= 1) D += __shfl_xor(D, o, LPP);
    if (ok && sub == 0) {
      bl[pi] = (int32_t)D;
      a.band[t * L + (k - 1)] = (int32_t)D;
    }
  }
  __syncthreads();
  // keep-test words of these rows
  for (int64_t t = t0 + tid; t < t1; t += nthr) {
    const int64_t seg = t / seg_len;
    const int kmax = (int)(t - seg * seg_len) < L ? (int)(t - seg * seg_len) : L;  // t - k stays in the stream
    const int64_t theta = theta_of(tau_of_segment(ru, seg), ru.twoM);
    const int32_t* row = bl + (t - t0) * L;
    const int32_t Dadj = row[0];
    a.adj[t] = Dadj;
    uint32_t g = 0;
    for (int k = 1; k <= kmax; ++k) {
      const int32_t Dref = row[k - 1];
      g |= (uint32_t)((Dadj > Dref ? Dadj : Dref) >= theta) << k;
    }
    a.G[t] = g;
  }
}

// L_max <= 0: no gap rule, so r(t) can lie arbitrarily far back.  One
// workgroup per stream walks t sequentially and measures D(t, r) from the
// histograms with a block reduction.
__global__ __launch_bounds__(256) void ngff_select_seq_kernel(RuleArgs a, const uint32_t* hist,
                                                              int32_t nbins, uint8_t* flag_g,
                                                              float* scores, uint8_t* mask,
                                                              int32_t* count) {
  __shared__ int64_t red[16];
  const int64_t seg = blockIdx.x, s0 = seg * a.seg_len;
  const int64_t T = a.n - s0 < a.seg_len ? a.n - s0 : a.seg_len;
  const int tid = threadIdx.x, nthr = blockDim.x;
  uint8_t* fl = flag_g + s0;
  for (int64_t i = tid; i < T; i += nthr) fl[i] = 0;
  const int64_t theta = theta_of(tau_of_segment(a, seg), a.twoM);
  __syncthreads();
  if (tid == 0) {
    fl[0] = 1;
    scores[s0] = 1.0f;
  }
  int64_t r = 0, kept = 1;
  for (int64_t t = 1; t < T; ++t) {
    const uint32_t* x = hist + (s0 + t) * nbins;
    const uint32_t* y = hist + (s0 + r) * nbins;
    int64_t part = 0;
    for (int b = tid; b < nbins; b += nthr) {
      const uint32_t u = x[b], v = y[b];
      part += u > v ? u - v : v - u;
    }
    const int64_t Dref = block_sum(part, red);
    const int32_t Dadj = a.band[(s0 + t) * a.L];  // band of width 1
    const int64_t D = Dadj > Dref ? Dadj : Dref;
    const bool keep = (t == T - 1) || D >= theta;
    if (tid == 0) {
      scores[s0 + t] = score_of(D, a.twoM);
      fl[t] = keep ? 1 : 0;
    }
    if (keep) {
      r = t;
      ++kept;
    }
  }
  __syncthreads();
  if (a.M_min >= 2 && kept < a.M_min) {
    for (int64_t i = tid; i < a.M_min; i += nthr) {
      const int64_t u = (i * (T - 1)) / (a.M_min - 1);
      if (fl[u] == 0) fl[u] = 2;
    }
  }
  __syncthreads();
  int64_t local = 0;
  for (int64_t t = tid; t < T; t += nthr) {
    local += fl[t] != 0;
    mask[s0 + t] = fl[t] != 0;
  }
  const int64_t total = block_sum(local, red);
  if (count && tid == 0) count[seg] = (int32_t)total;
}

// ---- threshold calibration ---------------------------------------------------------
__global__ void calib_init_kernel(int32_t* best, int64_t nseg, int64_t twoM) {
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i < nseg) best[i] = (int32_t)(twoM + 1);
}

// Kept count (top-up included) of one stream under integer threshold theta.
__device__ int64_t kept_count(const RuleArgs& a, int64_t s0, int64_t T, int64_t theta) {
  int64_t r = 0, kept = 1;
  while (r < T - 1) {
    int64_t u = r + 1;
    for (int k = 1;; ++k, ++u) {
      if (u == T - 1 || k >= a.L) break;
      const int32_t* row = a.band + (s0 + u) * a.L;
      const int32_t Dadj = row[0], Dref = row[k - 1];
      if ((Dadj > Dref ? Dadj : Dref) >= theta) break;
    }
    r = u;
    ++kept;
  }
  if (a.M_min >= 2 && kept < a.M_min) {
    // add the distinct uniform frames missing from the (short) kept chain
    int64_t prev = -1;
    for (int64_t i = 0; i < a.M_min; ++i) {
      const int64_t u = (i * (T - 1)) / (a.M_min - 1);
      if (u == prev) continue;
      prev = u;
      bool in_chain = false;
      int64_t c = 0;
      while (true) {  // walk the chain again: it has fewer than M_min frames
        if (c == u) {
          in_chain = true;
          break;
        }
        if (c > u || c >= T - 1) break;
        int64_t v = c + 1;
        for (int k = 1;; ++k, ++v) {
          if (v == T - 1 || k >= a.L) break;
          const int32_t* row = a.band + (s0 + v) * a.L;
          const int32_t Dadj = row[0], Dref = row[k - 1];
          if ((Dadj > Dref ? Dadj : Dref) >= theta) break;
        }
        c = v;
      }
      if (!in_chain) ++kept;
    }
  }
  return kept;
}

// One thread per candidate threshold: every band entry of a stream, plus 0 and
// 2M+1 per stream.  Satisfying candidates race with atomicMin.
__global__ void calib_kernel(RuleArgs a, int64_t nseg, int64_t target, int32_t* best) {
  const int64_t c = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  const int64_t nband = a.n * a.L;
  int64_t seg, theta;
  if (c < nband) {
    const int64_t t = c / a.L;
    const int k = (int)(c - t * a.L) + 1;
    seg = t / a.seg_len;
    if (t - k < seg * a.seg_len) return;
    theta = a.band[c];
  } else if (c < nband + 2 * nseg) {
    const int64_t e = c - nband;
    seg = e >> 1;
    theta = (e & 1) ? a.twoM + 1 : 0;
  } else {
    return;
  }
  if (theta >= __hip_atomic_load(best + seg, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return;
  const int64_t s0 = seg * a.seg_len;
  const int64_t T = a.n - s0 < a.seg_len ? a.n - s0 : a.seg_len;
  if (kept_count(a, s0, T, theta) <= target) atomicMin(best + seg, (int32_t)theta);
}

__global__ void calib_final_kernel(const int32_t* best, int64_t nseg, int64_t twoM, float* tau) {
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (i < nseg) tau[i] = score_of(best[i], twoM);
}

// ---- host side ------------------------------------------------------------------------

bool is_pow2(int v) { return v > 0 && (v & (v - 1)) == 0; }

struct NgffShape {
  int64_t n;
  int32_t H, W, C, B, mode;
  int64_t nbins, npix, frame_bytes, mass;
};

int validate_frames(const uint8_t* frames, int64_t n, int32_t H, int32_t W, int32_t C, int32_t bins,
                    int32_t mode, NgffShape* sh) {
  if (n < 0) return set_error(COFIE_EINVAL, "n = %lld is negative", (long long)n);
  if (n > 0 && !frames) return set_error(COFIE_EINVAL, "frames is NULL");
  if (H <= 0 || W <= 0) return set_error(COFIE_EINVAL, "H = %d, W = %d must be positive", H, W);
  if (C != 1 && C != 3) return set_error(COFIE_EINVAL, "C = %d must be 1 or 3", C);
  if (mode == COFIE_SIGNAL_FRAMEDIFF || mode == COFIE_SIGNAL_DHASH) {
    // the alternative signals: rows of G^2 cell means or 64 hash bits, 2M =
    // 255 G^2 or 64 (G a power of two, so that M is an integer)
    if (W > kSigMaxW) return set_error(COFIE_EUNSUPPORTED, "W = %d exceeds %d for this signal", W, kSigMaxW);
    if ((int64_t)H * W * 255 >= (int64_t(1) << 32))  // 32-bit cell sums
      return set_error(COFIE_EUNSUPPORTED, "%d x %d frames exceed the signal's 32-bit cell sums", H, W);
    if (mode == COFIE_SIGNAL_FRAMEDIFF) {
      if (bins < 2 || bins > 64 || !is_pow2(bins))
        return set_error(COFIE_EUNSUPPORTED, "frame-difference grid %d is not a power of two in [2, 64]", bins);
      if (bins > H || bins > W) return set_error(COFIE_EINVAL, "grid %d finer than the %d x %d image", bins, H, W);
    } else if (H < 8 || W < 9) {
      return set_error(COFIE_EINVAL, "dHash needs H >= 8 and W >= 9 (got %d x %d)", H, W);
    }
    sh->n = n;
    sh->H = H;
    sh->W = W;
    sh->C = C;
    sh->B = bins;
    sh->mode = mode;
    sh->nbins = cofie_ngff_nbins(mode, bins);
    sh->npix = (int64_t)H * W;
    sh->frame_bytes = sh->npix * C;
    sh->mass = mode == COFIE_SIGNAL_FRAMEDIFF ? 255 * (int64_t)bins * bins / 2 : 32;
    return COFIE_OK;
  }
  if (mode != COFIE_HIST_GRAY && mode != COFIE_HIST_PER_CHANNEL && mode != COFIE_HIST_JOINT3D)
    return set_error(COFIE_EINVAL, "unknown hist_mode %d", mode);
  if (C == 1 && mode != COFIE_HIST_GRAY)
    return set_error(COFIE_EINVAL, "C = 1 frames support only the GRAY histogram");
  if (bins < 2 || bins > 256) return set_error(COFIE_EINVAL, "bins = %d outside [2, 256]", bins);
  if (!is_pow2(bins))
    return set_error(COFIE_EUNSUPPORTED, "bins = %d is not a power of two", bins);
  const int64_t nbins = cofie_ngff_nbins(mode, bins);
  if (nbins > 4096)
    return set_error(COFIE_EUNSUPPORTED, "%lld bins exceed 4096", (long long)nbins);
  const int64_t npix = (int64_t)H * W;
  const int64_t mass = mode == COFIE_HIST_PER_CHANNEL ? 3 * npix : npix;
  if (2 * mass >= (int64_t(1) << 31))
    return set_error(COFIE_EUNSUPPORTED, "2M = %lld >= 2^31: distances would not fit the int32 band",
                     (long long)(2 * mass));
  sh->n = n;
  sh->H = H;
  sh->W = W;
  sh->C = C;
  sh->B = bins;
  sh->mode = mode;
  sh->nbins = nbins;
  sh->npix = npix;
  sh->frame_bytes = npix * C;
  sh->mass = mass;
  return COFIE_OK;
}

// Histogram launch geometry.
struct HistPlan {
  int kind, P, threads, splits, units;
  size_t lds;
};

HistPlan plan_hist(const NgffShape& sh, const uint8_t* frames) {
  HistPlan p;
  if (sh.mode == COFIE_HIST_PER_CHANNEL)
    p.kind = K_PC;
  else if (sh.mode == COFIE_HIST_JOINT3D)
    p.kind = K_JOINT;
  else
    p.kind = sh.C == 1 ? K_GRAY1 : K_GRAY3;
  p.P = 64;
  while ((size_t)sh.nbins * p.P * 4 > 160 * 1024) p.P >>= 1;
  p.lds = (size_t)sh.nbins * p.P * 4;
  // 8 waves, 3 units per batch: measured fastest against 16 waves and deeper
  // batches (1 fps stream 28.7 vs 32.2 us, hour stream 385 vs 458 us), more
  // bytes in flight per CU did not stream faster
  p.threads = 512;
  // the vector path needs 4-byte aligned frames
  const bool aligned = (reinterpret_cast<uintptr_t>(frames) % 4 == 0) && (sh.frame_bytes % 4 == 0);
  p.units = aligned ? (int)(sh.frame_bytes / kUnitBytes) : 0;
  const int nw = p.threads / 64;
  // one workgroup per frame when there are at least as many frames as CUs,
  // otherwise split frames so that every CU streams
  const int64_t cus = device_cu_count();
  int64_t splits = sh.n >= cus ? 1 : (cus + sh.n - 1) / (sh.n > 0 ? sh.n : 1);
  const int64_t by_units = p.units / (nw * kUnroll);
  if (splits > by_units) splits = by_units;
  if (splits < 1) splits = 1;
  p.splits = (int)splits;
  return p;
}

// Address model of ngff_hist_kernel (dry run): every unit load of every wave
// through the kernel's own index functions, the byte-wise pixels after the
// units, the LDS counters of every bin a pixel can reach, the output row.
template <int KIND, int P, int BC>
void model_hist(const HistArgs& a, int64_t n, int threads, size_t lds) {
  const int nw = threads / 64, G = a.splits * nw;
  const int C = KIND == K_GRAY1 ? 1 : 3;
  dry_range(a.npix * C, 0, a.frame_bytes + 1, "hist: pixels past the frame");
  dry_range((int64_t)a.units * kUnitBytes, 0, a.npix * C + 1, "hist: units past the pixels");
  const int64_t top_bin = KIND == K_PC ? 3 * (int64_t)a.B - 1
                        : (KIND == K_JOINT ? (int64_t)a.B * a.B * a.B - 1 : (int64_t)a.B - 1);
  dry_range(top_bin, 0, a.nbins, "hist: a pixel's bin past the counters");
  if (BC) dry_range(BC, a.B, a.B + 1, "hist: compiled bin count differs");
  dry_lds(0, (int64_t)a.nbins * P * 4, (int64_t)lds, "hist: counters");
  for (int64_t t = 0; t < n; ++t) {
    const int64_t fb = hist_map(t, a.group, a.in_stride, a.in_off) * a.frame_bytes;
    for (int g = 0; g < G; ++g) {
      const int nbatch = g < a.units ? (a.units - g + G * kUnroll - 1) / (G * kUnroll) : 0;
      const int last_b = nbatch > 0 ? 2 * (nbatch / 2) : -1;  // the pipeline loads one batch past an even count
      for (int b = 0; b <= last_b; ++b)
        for (int j = 0; j < kUnroll; ++j)
          dry_access(a.frames, fb + (int64_t)hist_unit(g, b * kUnroll + j, G, a.units) * kUnitBytes, kUnitBytes,
                     "hist: unit load");
    }
    const int64_t p0 = (int64_t)a.units * (kUnitBytes / C);
    if (p0 < a.npix) dry_access(a.frames, fb + p0 * C, (a.npix - p0) * C, "hist: pixels after the units");
    dry_access(a.hist, hist_map(t, a.group, a.out_stride, a.out_off) * a.nbins * 4, (int64_t)a.nbins * 4,
               "hist: histogram row");
  }
}

template <int KIND, int P, int BC>
int launch_hist_t(const HistArgs& args, const HistPlan& p, int64_t n, hipStream_t s) {
  auto k = ngff_hist_kernel<KIND, P, BC>;
  int rc = allow_lds(k, p.lds);
  if (rc) return rc;
  if (dry_run()) {
    if (n * p.splits > 0) model_hist<KIND, P, BC>(args, n, p.threads, p.lds);
    return COFIE_OK;
  }
  return launch("ngff_hist", k, dim3((unsigned)(n * p.splits)), dim3(p.threads), p.lds, s, args);
}

template <int KIND>
int launch_hist_kind(const HistArgs& args, const HistPlan& p, int64_t n, hipStream_t s) {
  switch (p.P) {
    case 64:
      if (args.B == 32) return launch_hist_t<KIND, 64, 32>(args, p, n, s);
      if (args.B == 16) return launch_hist_t<KIND, 64, 16>(args, p, n, s);
      if (KIND == K_JOINT && args.B == 8) return launch_hist_t<KIND, 64, 8>(args, p, n, s);
      return launch_hist_t<KIND, 64, 0>(args, p, n, s);
    case 32:
      return launch_hist_t<KIND, 32, 0>(args, p, n, s);
    case 16:
      return launch_hist_t<KIND, 16, 0>(args, p, n, s);
    default:
      return launch_hist_t<KIND, 8, 0>(args, p, n, s);
  }
}

struct HistMap {  // see HistArgs: group = 0 is the identity
  int64_t group = 0, in_stride = 0, in_off = 0, out_stride = 0, out_off = 0;
  int64_t out_rows = 0;  // rows of the output buffer (for the zero fill), 0 = n
  bool zeroed = false;   // the output rows are known zero: no fill before accumulating
};

// Address model of ngff_sig_kernel (dry run): each frame's rows as the
// vector or byte path reads them, the LDS column table and cell counters,
// the output row.
void model_sig(const SigArgs& a, int64_t n) {
  dry_range(a.W, 1, kSigMaxW + 1, "sig: columns past the column table");
  dry_range((int64_t)a.gh * a.gw, 1, 4097, "sig: cells past the counters");
  dry_range((int64_t)a.H * a.W * a.C, 1, a.frame_bytes + 1, "sig: pixels past the frame");
  const int64_t top_cell = (int64_t)((((int64_t)(a.H - 1) * a.gh) / a.H) * a.gw) + ((int64_t)(a.W - 1) * a.gw) / a.W;
  dry_range(top_cell, 0, (int64_t)a.gh * a.gw, "sig: a pixel's cell");
  for (int64_t b = 0; b < n; ++b) {
    const int64_t f = b * a.frame_bytes;
    const int64_t last_row = f + (int64_t)(a.H - 1) * a.W * a.C;
    if (a.vec) {
      const int x0 = (a.W - 1) / 4 * 4;  // the last 4-pixel group a lane reads
      dry_range(a.W % 4, 0, 1, "sig: 4-pixel loads need W a multiple of 4");
      dry_access(a.frames, f, a.C == 3 ? 12 : 4, "sig: first pixels");
      dry_access(a.frames, last_row + (a.C == 3 ? 3 * (int64_t)x0 : x0), a.C == 3 ? 12 : 4, "sig: last pixels");
    } else {
      dry_access(a.frames, f, a.C, "sig: first pixel");
      dry_access(a.frames, last_row + (int64_t)(a.W - 1) * a.C, a.C, "sig: last pixel");
    }
    dry_access(a.out, 4 * b * a.nsig, 4 * (int64_t)a.nsig, "sig: signature row");
  }
}

// Address model of ngff_band_keep_kernel (dry run): each workgroup's
// histogram rows, its LDS rows (transposed, stride RS) and band block, and
// the band, adjacent-distance and keep-word outputs of its frames.
void model_band_keep(const BandKeepArgs& a, int64_t nwg, int64_t lds) {
  const int L = a.rule.L;
  dry_lds(0, 4 * ((int64_t)a.nbins * a.RS + (int64_t)a.TB * L), lds, "keep: LDS rows and band block");
  for (int64_t b = 0; b < nwg; ++b) {
    const int64_t t0 = b * a.TB, t1 = t0 + a.TB < a.n ? t0 + a.TB : a.n;
    const int64_t r0 = t0 - L > 0 ? t0 - L : 0;
    dry_range(t1 - r0, 1, (int64_t)a.RS + 1, "keep: staged rows past the LDS row stride");
    dry_access(a.hist, 4 * r0 * a.nbins, 4 * (t1 - r0) * a.nbins, "keep: histogram rows");
    // the earliest row a pair reads: t - k >= the stream's first frame and >= r0
    const int64_t seg0 = (t0 / a.rule.seg_len) * a.rule.seg_len;
    const int64_t lo = t0 - L > seg0 ? t0 - L : seg0;
    dry_range(lo - r0, 0, a.RS, "keep: a pair's reference row before the staged rows");
    dry_access(a.band, 4 * t0 * L, 4 * (t1 - t0) * L, "keep: band rows");
    dry_access(a.adj, 4 * t0, 4 * (t1 - t0), "keep: adjacent distances");
    dry_access(a.G, 4 * t0, 4 * (t1 - t0), "keep: keep words");
    if (a.rule.tau_seg) {
      const int64_t s_lo = t0 / a.rule.seg_len, s_hi = (t1 - 1) / a.rule.seg_len;
      dry_access(a.rule.tau_seg, 4 * s_lo, 4 * (s_hi - s_lo + 1), "keep: per-stream thresholds");
    }
  }
}

int run_signature(const uint8_t* frames, const NgffShape& sh, uint32_t* out, hipStream_t s) {
  SigArgs a;
  a.frames = frames;
  a.frame_bytes = sh.frame_bytes;
  a.H = sh.H;
  a.W = sh.W;
  a.C = sh.C;
  a.dhash = sh.mode == COFIE_SIGNAL_DHASH;
  a.gh = a.dhash ? 8 : sh.B;
  a.gw = a.dhash ? 9 : sh.B;
  a.nsig = (int32_t)sh.nbins;
  a.vec = (reinterpret_cast<uintptr_t>(frames) % 4 == 0) && sh.W % 4 == 0 ? 1 : 0;
  a.out = out;
  if (dry_run()) model_sig(a, sh.n);
  return launch("ngff_sig", ngff_sig_kernel, dim3((unsigned)sh.n), dim3(kSigThreads), 0, s, a);
}

int run_histogram(const uint8_t* frames, const NgffShape& sh, uint32_t* hist, hipStream_t s,
                  const HistMap& map = HistMap()) {
  if (sh.n == 0) return COFIE_OK;
  if (sh.mode == COFIE_SIGNAL_FRAMEDIFF || sh.mode == COFIE_SIGNAL_DHASH) return run_signature(frames, sh, hist, s);
  const HistPlan p = plan_hist(sh, frames);
  HistArgs a;
  a.group = map.group;
  a.in_stride = map.in_stride;
  a.in_off = map.in_off;
  a.out_stride = map.out_stride;
  a.out_off = map.out_off;
  a.frames = frames;
  a.frame_bytes = sh.frame_bytes;
  a.npix = sh.npix;
  a.hist = hist;
  a.nbins = (int32_t)sh.nbins;
  a.B = sh.B;
  a.logB = __builtin_ctz(sh.B);
  a.shift = 8 - a.logB;
  a.splits = p.splits;
  a.units = p.units;
  a.atomic = p.splits > 1;
  if (a.atomic && !map.zeroed) {
    const int64_t cnt = (map.out_rows ? map.out_rows : sh.n) * sh.nbins;
    int rc = launch("ngff_fill", fill_u32_kernel, dim3((unsigned)std::min<int64_t>(ceil_div(cnt, 256), 4096)),
                    dim3(256), 0, s, hist, 0u, cnt);
    if (rc) return rc;
  }
  switch (p.kind) {
    case K_PC: return launch_hist_kind<K_PC>(a, p, sh.n, s);
    case K_GRAY1: return launch_hist_kind<K_GRAY1>(a, p, sh.n, s);
    case K_GRAY3: return launch_hist_kind<K_GRAY3>(a, p, sh.n, s);
    default: return launch_hist_kind<K_JOINT>(a, p, sh.n, s);
  }
}

struct RulePlan {
  int64_t seg_len, nseg;
  int32_t L;          // band width (>= 1)
  bool gap_rule;      // L_max >= 1
};

RulePlan plan_rule(const NgffShape& sh, const cofie_keep_rule* r) {
  RulePlan p;
  p.seg_len = (r->segment_len <= 0 || r->segment_len > sh.n) ? (sh.n > 0 ? sh.n : 1) : r->segment_len;
  p.nseg = sh.n > 0 ? (sh.n + p.seg_len - 1) / p.seg_len : 0;
  p.gap_rule = r->L_max >= 1;
  p.L = p.gap_rule ? r->L_max : 1;
  return p;
}

// Launch plan of the band/keep-word kernel: TB frames per workgroup (about
// one workgroup per CU, at most ~48 Ki |difference| terms of band work each),
// the transposed histogram rows (nbins x RS words, RS = TB + L made odd so
// that lanes reading consecutive bins hit distinct banks) and the tile's band
// rows (TB x L words) in LDS.  ok = false when L_max > 31 (one keep-test word
// per frame) or even one frame's rows exceed the LDS budget.
constexpr size_t kLdsBudget = 150 * 1024;

struct BandKeepPlan {
  bool ok;
  int TB, RS;
  size_t lds;
};

BandKeepPlan plan_band_keep(const NgffShape& sh, const RulePlan& rp) {
  BandKeepPlan p;
  const int64_t cus = device_cu_count();
  int64_t tb = (sh.n + cus - 1) / cus;
  int64_t tb_max = 49152 / ((int64_t)rp.L * sh.nbins);
  tb_max = tb_max < 1 ? 1 : (tb_max > 64 ? 64 : tb_max);
  p.TB = (int)(tb < 1 ? 1 : (tb > tb_max ? tb_max : tb));
  auto stage = [&](int TB) {
    const int RS = (TB + rp.L) | 1;
    return (size_t)sh.nbins * RS * 4 + (size_t)TB * rp.L * 4;
  };
  while (p.TB > 1 && stage(p.TB) > kLdsBudget) --p.TB;
  p.RS = (p.TB + rp.L) | 1;
  p.lds = stage(p.TB);
  p.ok = rp.L <= 31 && p.lds <= kLdsBudget;
  return p;
}

// Frames per selection chunk: the stream rounded up to 64, at most 4096.
inline int select_chunk(int64_t seg_len) {
  const int64_t c = (seg_len + 63) / 64 * 64;
  return (int)(c < 4096 ? c : 4096);
}

// Scratch layout of filter/calibrate (same sequence sizes and carves).
struct NgffScratch {
  uint32_t* hist;
  int32_t* band;
  int32_t* next;   // next-keep table of the separate kernels
  uint8_t* flags;  // per-frame flags of the sequential selection (no gap rule)
  int32_t* best;   // calibration: best threshold per stream
  uint32_t* G;     // [n] keep-test words
  int32_t* adj;    // [n] D(t, t-1)
};

NgffScratch carve(Arena& ar, const NgffShape& sh, const RulePlan& rp, bool need_hist) {
  NgffScratch w;
  const size_t nseg = (size_t)(rp.nseg > 0 ? rp.nseg : 1);
  w.hist = need_hist ? ar.take<uint32_t>((size_t)(sh.n * sh.nbins)) : nullptr;
  w.band = ar.take<int32_t>((size_t)(sh.n * rp.L));
  w.next = ar.take<int32_t>((size_t)sh.n);
  w.flags = ar.take<uint8_t>((size_t)sh.n);
  w.best = ar.take<int32_t>(nseg);
  w.G = ar.take<uint32_t>((size_t)sh.n);
  w.adj = ar.take<int32_t>((size_t)sh.n);
  return w;
}

// Separate band kernel (rows read from global memory when they do not fit LDS).
int run_band(const uint32_t* hist, const NgffShape& sh, const RulePlan& rp, int32_t* band,
             hipStream_t s, const uint32_t* window = nullptr, int32_t wrows = 0) {
  BandArgs b;
  b.window = window;
  b.wrows = wrows;
  b.hist = hist;
  b.n = sh.n;
  b.nbins = (int32_t)sh.nbins;
  b.L = rp.L;
  b.seg_len = rp.seg_len;
  const size_t budget = 64 * 1024;
  const size_t row = (size_t)(sh.nbins + 1) * 4;
  // about one workgroup per CU (a 94-row push band took 45 us with 64 frames
  // per workgroup, i.e. two workgroups), at most 64 frames each
  const int64_t cus = device_cu_count();
  int TB = (int)std::min<int64_t>(64, std::max<int64_t>(1, (sh.n + cus - 1) / cus));
  while (TB > 1 && (size_t)(TB + rp.L) * row > budget) TB >>= 1;
  size_t lds = (size_t)(TB + rp.L) * row;
  b.TB = TB;
  b.stride = (int32_t)(sh.nbins + 1);
  if (lds > budget) {  // rows too wide for LDS: read the histogram from global memory
    b.stride = 0;
    lds = 0;
  }
  b.band = band;
  int rc = allow_lds(ngff_band_kernel, lds);
  if (rc) return rc;
  return launch("ngff_band", ngff_band_kernel, dim3((unsigned)ceil_div(sh.n, TB)), dim3(256), lds, s, b);
}

RuleArgs rule_args(const NgffShape& sh, const RulePlan& rp, const cofie_keep_rule* r,
                   const int32_t* band) {
  RuleArgs a;
  a.band = band;
  a.n = sh.n;
  a.seg_len = rp.seg_len;
  a.L = rp.L;
  a.M_min = r->M_min;
  a.twoM = 2 * sh.mass;
  a.tau = r->tau_h;
  a.tau_seg = r->tau_per_segment;
  return a;
}

int validate_rule(const cofie_keep_rule* r) {
  if (!r) return set_error(COFIE_EINVAL, "keep_rule is NULL");
  if (r->segment_len < 0) return set_error(COFIE_EINVAL, "segment_len is negative");
  if (r->M_min < 0) return set_error(COFIE_EINVAL, "M_min is negative");
  if (!r->tau_per_segment && r->tau_h != r->tau_h) return set_error(COFIE_EINVAL, "tau_h is NaN");
  return COFIE_OK;
}

// ---- NGFF as frames arrive ----------------------------------------------------------
// The keep rule decided frame by frame as a stream grows (Sec. 3.1: the model
// sees the current video prefix).  A push histograms the new frames of every
// stream into a per-stream buffer [L window rows | nb new rows] (the window =
// the L = L_max frames before the push, carried in the state), computes the
// band of that buffer, and one workgroup per stream decides the new frames:
// next[r] for the carried last kept frame and every new frame (open at the
// batch end: no keep found within the frames seen -> "beyond"), the chain
// walked from the carried frame, r(t) by a block prefix maximum, the scores.
// The end-of-stream safeguards (last frame, M_min top-up) wait for finish.
struct PushArgs {
  const int32_t* band;   // [S][L + nb][L]
  int32_t L;             // L_max (>= 1): band width and gap rule
  int32_t nb;            // new frames per stream in this push (<= 1024)
  int64_t t0;            // frames of each stream before this push
  int64_t twoM;
  float tau;
  const float* tau_seg;  // [S] or null
  int32_t* r_state;      // [S] last kept frame
  int32_t* kept_state;   // [S] kept frames so far
  float* out_scores;     // row s at out_scores + s * ld
  uint8_t* out_mask;
  int64_t ld;
  uint32_t* comb;        // [S][L + nb][nbins]: rows L.. hold the new frames' histograms
                         // (zeroed here once read, for the next push's accumulation)
  uint32_t* window;      // [S][L][nbins]: histograms of the L frames before t0, updated here
  int64_t nbins;
};

__global__ __launch_bounds__(1024) void ngff_push_kernel(PushArgs a) {
  extern __shared__ int32_t psm[];
  int32_t* bandL = psm;                          // [nb][L]
  int32_t* next_sh = bandL + a.nb * a.L;         // [nb + 1]: slot 0 = carried frame, 1 + j = new frame j
  int32_t* keep_sh = next_sh + a.nb + 1;         // [nb]
  int32_t* incl_sh = keep_sh + a.nb;             // [nb]
  __shared__ int64_t theta_sh;
  __shared__ int wtmp[16];
  const int s = blockIdx.x, tid = threadIdx.x, nthr = blockDim.x;
  const int L = a.L, nb = a.nb;
  const int64_t t0 = a.t0, tend = t0 + nb;
  const int32_t* src = a.band + ((int64_t)s * (L + nb) + L) * L;
  for (int i = tid; i < nb * L; i += nthr) bandL[i] = src[i];
  for (int j = tid; j < nb; j += nthr) keep_sh[j] = 0;
  if (tid == 0) theta_sh = theta_of(a.tau_seg ? a.tau_seg[s] : a.tau, a.twoM);
  const int64_t rc = t0 > 0 ? a.r_state[s] : -1;  // carried last kept frame
  __syncthreads();
  const int64_t theta = theta_sh;
  // next[r]: the first u in (r, r + L] (u >= t0) whose max(D(u, u-1), D(u, r))
  // reaches theta, else r + L (gap rule) if that frame has arrived, else beyond
  for (int q = tid; q <= nb; q += nthr) {
    const int64_t r = q == 0 ? rc : t0 + q - 1;
    int64_t found = tend;
    if (r >= 0) {
      const int64_t ulo = r + 1 > t0 ? r + 1 : t0;
      const int64_t uhi = r + L < tend - 1 ? r + L : tend - 1;
      for (int64_t u = ulo; u <= uhi; ++u) {
        const int32_t* row = bandL + (u - t0) * L;
        const int32_t Dadj = row[0], Dref = row[u - r - 1];
        if ((Dadj > Dref ? Dadj : Dref) >= theta) {
          found = u;
          break;
        }
      }
      if (found == tend && r + L <= tend - 1) found = r + L;
    }
    // relative to t0, nb = beyond; a carried frame is never L or more before
    // t0 (the gap rule), the clamp only keeps a corrupted state in bounds
    next_sh[q] = (int32_t)(found < t0 ? 0 : found - t0);
  }
  __syncthreads();
  if (tid == 0) {
    int64_t r = rc;
    int slot = 0, count = 0;
    if (t0 == 0) {  // the stream's first frame is kept
      keep_sh[0] = 1;
      r = 0;
      slot = 1;
      count = 1;
    }
    for (;;) {
      const int nx = next_sh[slot];
      if (nx >= nb) break;
      keep_sh[nx] = 1;
      ++count;
      r = t0 + nx;
      slot = nx + 1;
    }
    a.r_state[s] = (int32_t)r;
    a.kept_state[s] = (t0 > 0 ? a.kept_state[s] : 0) + count;
  }
  __syncthreads();
  // r(t) = the last kept frame before t: prefix maximum over this push, then the carried frame
  for (int j0 = 0; j0 < nb; j0 += nthr) {
    const int j = j0 + tid;
    const int v = (j < nb && keep_sh[j]) ? j : -1;
    const int x = block_inclusive_max(v, wtmp);
    if (j < nb) incl_sh[j] = x;
  }
  __syncthreads();
  for (int j = tid; j < nb; j += nthr) {
    const int64_t t = t0 + j;
    float score = 1.0f;
    if (t > 0) {
      const int prev = j > 0 ? incl_sh[j - 1] : -1;
      const int64_t rt = prev >= 0 ? t0 + prev : rc;
      const int32_t* row = bandL + j * L;
      const int64_t k = t - rt;  // 1 <= k <= L by the gap rule
      const int32_t Dadj = row[0], Dref = row[k < 1 ? 0 : (k > L ? L - 1 : k - 1)];
      score = score_of(Dadj > Dref ? Dadj : Dref, a.twoM);
    }
    a.out_scores[s * a.ld + j] = score;
    a.out_mask[s * a.ld + j] = (uint8_t)keep_sh[j];
  }
  // the window becomes the last L frames: row q <- row nb + q of (old window,
  // new frames).  When nb < L this shifts the window down in place, so it is
  // copied in chunks, each read completely before any of it is written (later
  // chunks only read above what earlier chunks wrote).
  uint32_t* win = a.window + (int64_t)s * L * a.nbins;
  uint32_t* cs = a.comb + (int64_t)s * (L + nb) * a.nbins;
  const int64_t total = (int64_t)L * a.nbins;
  constexpr int V = 4;
  for (int64_t c0 = 0; c0 < total; c0 += (int64_t)V * nthr) {
    uint32_t v[V];
#pragma unroll
    for (int u = 0; u < V; ++u) {
      const int64_t i = c0 + u * nthr + tid;
      const int64_t q = i / a.nbins;  // window row
      v[u] = i >= total ? 0u : (nb + q < L ? win[i + (int64_t)nb * a.nbins] : cs[i + (int64_t)nb * a.nbins]);
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < V; ++u) {
      const int64_t i = c0 + u * nthr + tid;
      if (i < total) win[i] = v[u];
    }
    __syncthreads();
  }
  // the new frames' rows start the next push at zero (its histogram adds into
  // them when several workgroups share a frame), so that push needs no fill
  for (int64_t i = tid; i < (int64_t)nb * a.nbins; i += nthr) cs[(int64_t)L * a.nbins + i] = 0u;
}

// comb[s][0..L) <- window[s] (dir 0) or window[s] <- comb[s][nb..nb+L) (dir 1)

// End of the streams: frame T-1 kept, then the M_min top-up (one thread per
// stream); out_added row s receives the frames this adds, increasing and -1
// padded to M_min + 1 entries.
__global__ void ngff_finish_kernel(uint8_t* mask_all, int64_t ld, int32_t S, int64_t T, int32_t M_min,
                                   int32_t* kept_state, int32_t* out_added, int32_t* out_count) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= S) return;
  uint8_t* m = mask_all + s * ld;
  const int cap = (M_min > 0 ? M_min : 0) + 1;
  int32_t* add = out_added ? out_added + (int64_t)s * cap : nullptr;
  int na = 0;
  auto record = [&](int64_t u) {
    if (!add) return;
    int i = na++;
    while (i > 0 && add[i - 1] > u) {  // insertion keeps the list increasing
      add[i] = add[i - 1];
      --i;
    }
    add[i] = (int32_t)u;
  };
  int64_t kept = T > 0 ? kept_state[s] : 0;
  if (T > 0) {
    if (!m[T - 1]) {
      m[T - 1] = 1;
      ++kept;
      record(T - 1);
    }
    if (M_min >= 2 && kept < M_min) {
      for (int64_t i = 0; i < M_min; ++i) {
        const int64_t u = (i * (T - 1)) / (M_min - 1);
        if (!m[u]) {
          m[u] = 1;
          ++kept;
          record(u);
        }
      }
    }
  }
  if (add)
    for (int i = na; i < cap; ++i) add[i] = -1;
  kept_state[s] = (int32_t)kept;
  if (out_count) out_count[s] = (int32_t)kept;
}

// Workgroup sizes of the keep-rule kernels: small enough (4 waves, one per
// SIMD) to run beside the QER score kernel's workgroups on the same CUs when
// a caller overlaps the two on separate streams; the selection takes 1024
// threads only for long streams.
constexpr int kKeepThreads = 256;
inline int select_threads(const RulePlan& rp) { return rp.seg_len <= 2048 ? 256 : 1024; }

// cofie_ngff_filter after validation: the histograms of `frames`, or the
// given ones (hist_in), then the keep rule.
int filter_impl(const uint8_t* frames, const uint32_t* hist_in, const NgffShape& sh,
                const cofie_keep_rule* keep_rule, float* out_scores, uint8_t* out_mask, hipStream_t s) {
  int rc;
  const RulePlan rp = plan_rule(sh, keep_rule);
  const bool need_hist = hist_in == nullptr && keep_rule->out_hist == nullptr;
  Arena plan;
  carve(plan, sh, rp, need_hist);
  Scratch scratch;
  rc = scratch.acquire(keep_rule->workspace, keep_rule->workspace_bytes, plan.bytes(), s);
  if (rc) return rc;
  Arena ar;
  ar.base = scratch.ptr();
  NgffScratch w = carve(ar, sh, rp, need_hist);
  const uint32_t* hist = hist_in ? hist_in : (need_hist ? w.hist : keep_rule->out_hist);

  RuleArgs ra = rule_args(sh, rp, keep_rule, w.band);
  if (!hist_in) {
    rc = run_histogram(frames, sh, const_cast<uint32_t*>(hist), s);
    if (rc) return rc;
  }
  const BandKeepPlan bp = plan_band_keep(sh, rp);
  const int chunk = select_chunk(rp.seg_len);
  if (rp.gap_rule && bp.ok) {
    BandKeepArgs bk;
    bk.hist = hist;
    bk.n = sh.n;
    bk.nbins = (int32_t)sh.nbins;
    bk.TB = bp.TB;
    bk.RS = bp.RS;
    bk.rule = ra;
    bk.band = w.band;
    bk.adj = w.adj;
    bk.G = w.G;
    rc = allow_lds(ngff_band_keep_kernel, bp.lds);
    if (rc) return rc;
    if (dry_run()) model_band_keep(bk, ceil_div(sh.n, bp.TB), (int64_t)bp.lds);
    rc = launch("ngff_keep", ngff_band_keep_kernel, dim3((unsigned)ceil_div(sh.n, bp.TB)), dim3(kKeepThreads),
                bp.lds, s, bk);
    if (rc) return rc;
    const size_t lds = select_lds(chunk, true);
    rc = allow_lds(ngff_select_kernel<true>, lds);
    if (rc) return rc;
    rc = launch("ngff_select", ngff_select_kernel<true>, dim3((unsigned)rp.nseg), dim3(select_threads(rp)), lds, s, ra,
                (const uint32_t*)w.G, (const int32_t*)nullptr, (const int32_t*)w.adj, (int32_t)chunk, out_scores,
                out_mask,
                keep_rule->out_count);
  } else if (rp.gap_rule) {
    // L_max > 31 or histogram rows too wide for LDS: band and next[] as
    // kernels of their own
    rc = run_band(hist, sh, rp, w.band, s);
    if (rc) return rc;
    rc = launch("ngff_next", ngff_next_kernel, dim3((unsigned)ceil_div(sh.n, 256)), dim3(256), 0, s, ra,
                w.next);
    if (rc) return rc;
    const size_t lds = select_lds(chunk, false);
    rc = allow_lds(ngff_select_kernel<false>, lds);
    if (rc) return rc;
    rc = launch("ngff_select", ngff_select_kernel<false>, dim3((unsigned)rp.nseg), dim3(select_threads(rp)), lds, s, ra,
                (const uint32_t*)nullptr, (const int32_t*)w.next, (const int32_t*)nullptr, (int32_t)chunk,
                out_scores, out_mask,
                keep_rule->out_count);
  } else {
    rc = run_band(hist, sh, rp, w.band, s);
    if (rc) return rc;
    rc = launch("ngff_select_seq", ngff_select_seq_kernel, dim3((unsigned)rp.nseg), dim3(256), 0, s,
                ra, (const uint32_t*)hist, (int32_t)sh.nbins, w.flags, out_scores, out_mask,
                keep_rule->out_count);
  }
  return rc;
}

}  // namespace
}  // namespace cofie

using namespace cofie;

// ---- online NGFF state --------------------------------------------------------------
struct cofie_ngff_stream {
  int device = 0;
  NgffShape sh{};          // n unused
  int32_t S = 0, L = 0, M_min = 0;
  float tau = 0.f;
  float* tau_dev = nullptr;    // [S] copy of tau_per_segment, or null
  uint32_t* window = nullptr;  // [S][L][nbins]: histograms of the L frames before t0
  int32_t* r = nullptr;        // [S] last kept frame
  int32_t* kept = nullptr;     // [S] kept frames so far
  int64_t t0 = 0;              // frames pushed per stream
  bool finished = false;
  void* scratch = nullptr;     // push scratch (new frames' histograms, band), kept between pushes
  size_t scratch_bytes = 0;
  int32_t zero_nb = -1;        // the push size whose new-frame rows in scratch are known zero
};

namespace cofie {
namespace {
// Host header of a saved stream state; the device arrays follow it.
struct StreamBlobHeader {
  char magic[8];
  int32_t S, L, M_min, mode, H, W, C, B;
  int64_t nbins;
  uint32_t tau_bits;
  int32_t per_segment_tau;
  int64_t t0;
  int32_t finished, pad;
};

StreamBlobHeader blob_header(const cofie_ngff_stream& st) {
  StreamBlobHeader h;
  std::memset(&h, 0, sizeof h);
  std::memcpy(h.magic, "CFNGST01", 8);
  h.S = st.S;
  h.L = st.L;
  h.M_min = st.M_min;
  h.mode = st.sh.mode;
  h.H = st.sh.H;
  h.W = st.sh.W;
  h.C = st.sh.C;
  h.B = st.sh.B;
  h.nbins = st.sh.nbins;
  // the scalar threshold matters only without per-stream thresholds
  const float tau = st.tau_dev ? 0.f : st.tau;
  std::memcpy(&h.tau_bits, &tau, sizeof tau);
  h.per_segment_tau = st.tau_dev ? 1 : 0;
  h.t0 = st.t0;
  h.finished = st.finished ? 1 : 0;
  return h;
}
}  // namespace
}  // namespace cofie

extern "C" {

void cofie_keep_rule_default(cofie_keep_rule* r) {
  if (!r) return;
  r->hist_mode = COFIE_HIST_GRAY;
  r->tau_h = 0.30f;
  r->tau_per_segment = nullptr;
  r->L_max = 30;
  r->M_min = 4;
  r->segment_len = 0;
  r->out_hist = nullptr;
  r->out_count = nullptr;
  r->workspace = nullptr;
  r->workspace_bytes = 0;
}

int64_t cofie_ngff_nbins(int32_t mode, int32_t bins) {
  if (bins < 1) return 0;
  if (mode == COFIE_HIST_GRAY) return bins;
  if (mode == COFIE_HIST_PER_CHANNEL) return 3 * (int64_t)bins;
  if (mode == COFIE_HIST_JOINT3D) return (int64_t)bins * bins * bins;
  if (mode == COFIE_SIGNAL_FRAMEDIFF) return (int64_t)bins * bins;
  if (mode == COFIE_SIGNAL_DHASH) return 64;
  return 0;
}

size_t cofie_ngff_workspace_bytes(int64_t n, int32_t H, int32_t W, int32_t C, int32_t bins,
                                  const cofie_keep_rule* rule) {
  NgffShape sh;
  static const uint8_t dummy = 0;
  if (!rule || validate_frames(n > 0 ? &dummy : nullptr, n, H, W, C, bins, rule->hist_mode, &sh))
    return 0;
  const RulePlan rp = plan_rule(sh, rule);
  Arena ar;
  carve(ar, sh, rp, true);
  return ar.bytes();
}

int cofie_ngff_histogram(const uint8_t* frames, int64_t n, int32_t H, int32_t W, int32_t C,
                         int32_t bins, int32_t hist_mode, uint32_t* out_hist, void* stream) {
  clear_error();
  NgffShape sh;
  int rc = validate_frames(frames, n, H, W, C, bins, hist_mode, &sh);
  if (rc) return rc;
  if (n > 0 && !out_hist) return set_error(COFIE_EINVAL, "out_hist is NULL");
  return run_histogram(frames, sh, out_hist, static_cast<hipStream_t>(stream));
}

int cofie_ngff_filter(const uint8_t* frames, int64_t n, int32_t H, int32_t W, int32_t C,
                      int32_t bins, const cofie_keep_rule* keep_rule, float* out_scores,
                      uint8_t* out_mask, void* stream) {
  clear_error();
  int rc = validate_rule(keep_rule);
  if (rc) return rc;
  NgffShape sh;
  rc = validate_frames(frames, n, H, W, C, bins, keep_rule->hist_mode, &sh);
  if (rc) return rc;
  if (n > 0 && (!out_scores || !out_mask))
    return set_error(COFIE_EINVAL, "out_scores / out_mask is NULL");
  if (n == 0) return COFIE_OK;
  return filter_impl(frames, nullptr, sh, keep_rule, out_scores, out_mask, static_cast<hipStream_t>(stream));
}

int cofie_ngff_filter_hist(const uint32_t* hist, int64_t n, int32_t H, int32_t W, int32_t C, int32_t bins,
                           const cofie_keep_rule* keep_rule, float* out_scores, uint8_t* out_mask,
                           void* stream) {
  clear_error();
  int rc = validate_rule(keep_rule);
  if (rc) return rc;
  NgffShape sh;
  rc = validate_frames(reinterpret_cast<const uint8_t*>(hist), n, H, W, C, bins, keep_rule->hist_mode, &sh);
  if (rc) return rc;
  if (n > 0 && (!out_scores || !out_mask))
    return set_error(COFIE_EINVAL, "out_scores / out_mask is NULL");
  if (n == 0) return COFIE_OK;
  return filter_impl(nullptr, hist, sh, keep_rule, out_scores, out_mask, static_cast<hipStream_t>(stream));
}

int cofie_ngff_calibrate(const uint8_t* frames, int64_t n, int32_t H, int32_t W, int32_t C,
                         int32_t bins, const cofie_keep_rule* keep_rule,
                         int64_t target_per_segment, float* out_tau, void* stream) {
  clear_error();
  if (!keep_rule) return set_error(COFIE_EINVAL, "keep_rule is NULL");
  if (keep_rule->segment_len < 0) return set_error(COFIE_EINVAL, "segment_len is negative");
  if (keep_rule->M_min < 0) return set_error(COFIE_EINVAL, "M_min is negative");
  NgffShape sh;
  int rc = validate_frames(frames, n, H, W, C, bins, keep_rule->hist_mode, &sh);
  if (rc) return rc;
  if (keep_rule->L_max < 1)
    return set_error(COFIE_EUNSUPPORTED, "calibration needs L_max >= 1");
  if (target_per_segment < 0) return set_error(COFIE_EINVAL, "negative target");
  if (n > 0 && !out_tau) return set_error(COFIE_EINVAL, "out_tau is NULL");
  if (n == 0) return COFIE_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const RulePlan rp = plan_rule(sh, keep_rule);
  Arena plan;
  carve(plan, sh, rp, true);
  Scratch scratch;
  rc = scratch.acquire(keep_rule->workspace, keep_rule->workspace_bytes, plan.bytes(), s);
  if (rc) return rc;
  Arena ar;
  ar.base = scratch.ptr();
  NgffScratch w = carve(ar, sh, rp, true);
  rc = run_histogram(frames, sh, w.hist, s);
  if (rc) return rc;
  rc = run_band(w.hist, sh, rp, w.band, s);
  if (rc) return rc;
  RuleArgs ra = rule_args(sh, rp, keep_rule, w.band);
  const int64_t twoM = 2 * sh.mass;
  rc = launch("ngff_calib_init", calib_init_kernel, dim3((unsigned)ceil_div(rp.nseg, 256)), dim3(256),
              0, s, w.best, rp.nseg, twoM);
  if (rc) return rc;
  const int64_t ncand = sh.n * rp.L + 2 * rp.nseg;
  rc = launch("ngff_calib", calib_kernel, dim3((unsigned)ceil_div(ncand, 256)), dim3(256), 0, s, ra,
              rp.nseg, target_per_segment, w.best);
  if (rc) return rc;
  return launch("ngff_calib_final", calib_final_kernel, dim3((unsigned)ceil_div(rp.nseg, 256)),
                dim3(256), 0, s, (const int32_t*)w.best, rp.nseg, twoM, out_tau);
}


int cofie_ngff_stream_create(int32_t n_streams, int32_t H, int32_t W, int32_t C, int32_t bins,
                             const cofie_keep_rule* rule, cofie_ngff_stream** out_state) {
  clear_error();
  if (!out_state) return set_error(COFIE_EINVAL, "out_state is NULL");
  *out_state = nullptr;
  if (dry_run()) return set_error(COFIE_EUNSUPPORTED, "the online filter allocates its state: no dry run");
  if (!rule) return set_error(COFIE_EINVAL, "keep_rule is NULL");
  if (n_streams < 1) return set_error(COFIE_EINVAL, "n_streams = %d must be >= 1", n_streams);
  NgffShape sh;
  int rc = validate_frames(nullptr, 0, H, W, C, bins, rule->hist_mode, &sh);
  if (rc) return rc;
  if (rule->hist_mode == COFIE_SIGNAL_FRAMEDIFF || rule->hist_mode == COFIE_SIGNAL_DHASH)
    return set_error(COFIE_EUNSUPPORTED, "the online state keeps histograms only (not the Table 5 signals)");
  if (rule->L_max < 1) return set_error(COFIE_EUNSUPPORTED, "the streaming keep rule needs L_max >= 1");
  if (rule->M_min < 0) return set_error(COFIE_EINVAL, "M_min is negative");
  if (!rule->tau_per_segment && !(rule->tau_h == rule->tau_h)) return set_error(COFIE_EINVAL, "tau_h is NaN");
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return set_error(COFIE_EHIP, "hipGetDevice failed");
  auto* st = new cofie_ngff_stream();
  st->device = dev;
  st->sh = sh;
  st->S = n_streams;
  st->L = rule->L_max;
  st->M_min = rule->M_min;
  st->tau = rule->tau_h;
  const size_t wbytes = (size_t)n_streams * st->L * sh.nbins * sizeof(uint32_t);
  bool ok = hipMalloc(&st->window, wbytes) == hipSuccess &&
            hipMalloc(&st->r, n_streams * sizeof(int32_t)) == hipSuccess &&
            hipMalloc(&st->kept, n_streams * sizeof(int32_t)) == hipSuccess &&
            hipMemset(st->window, 0, wbytes) == hipSuccess &&
            hipMemset(st->r, 0, n_streams * sizeof(int32_t)) == hipSuccess &&
            hipMemset(st->kept, 0, n_streams * sizeof(int32_t)) == hipSuccess;
  if (ok && rule->tau_per_segment) {
    ok = hipMalloc(&st->tau_dev, n_streams * sizeof(float)) == hipSuccess &&
         hipMemcpy(st->tau_dev, rule->tau_per_segment, n_streams * sizeof(float), hipMemcpyDeviceToDevice) ==
             hipSuccess;
  }
  if (!ok) {
    cofie_ngff_stream_destroy(st);
    return set_error(COFIE_ENOMEM, "allocating the stream state failed");
  }
  *out_state = st;
  return COFIE_OK;
}

int cofie_ngff_stream_destroy(cofie_ngff_stream* st) {
  clear_error();
  if (!st) return COFIE_OK;
  int dev = 0;
  hipGetDevice(&dev);
  if (dev != st->device) hipSetDevice(st->device);
  if (st->window) hipFree(st->window);
  if (st->r) hipFree(st->r);
  if (st->kept) hipFree(st->kept);
  if (st->tau_dev) hipFree(st->tau_dev);
  if (st->scratch) hipFree(st->scratch);
  if (dev != st->device) hipSetDevice(dev);
  delete st;
  return COFIE_OK;
}

int64_t cofie_ngff_stream_frames(const cofie_ngff_stream* st) { return st ? st->t0 : -1; }

size_t cofie_ngff_stream_state_bytes(const cofie_ngff_stream* st) {
  if (!st) return 0;
  return sizeof(StreamBlobHeader) + (st->tau_dev ? (size_t)st->S * sizeof(float) : 0) +
         (size_t)st->S * st->L * st->sh.nbins * sizeof(uint32_t) + 2 * (size_t)st->S * sizeof(int32_t);
}

int cofie_ngff_stream_save(const cofie_ngff_stream* st, void* buf, size_t bytes, void* stream) {
  clear_error();
  if (!st || !buf) return set_error(COFIE_EINVAL, "state or buffer is NULL");
  const size_t need = cofie_ngff_stream_state_bytes(st);
  if (bytes < need) return set_error(COFIE_EINVAL, "buffer of %zu bytes is smaller than the %zu required", bytes, need);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev != st->device)
    return set_error(COFIE_EINVAL, "the current device is not the state's device");
  hipStream_t s = static_cast<hipStream_t>(stream);
  StreamBlobHeader h = blob_header(*st);
  char* p = static_cast<char*>(buf);
  std::memcpy(p, &h, sizeof h);
  p += sizeof h;
  if (st->tau_dev) {
    COFIE_CHECK_HIP(hipMemcpyAsync(p, st->tau_dev, (size_t)st->S * sizeof(float), hipMemcpyDeviceToHost, s));
    p += (size_t)st->S * sizeof(float);
  }
  const size_t wbytes = (size_t)st->S * st->L * st->sh.nbins * sizeof(uint32_t);
  COFIE_CHECK_HIP(hipMemcpyAsync(p, st->window, wbytes, hipMemcpyDeviceToHost, s));
  p += wbytes;
  COFIE_CHECK_HIP(hipMemcpyAsync(p, st->r, (size_t)st->S * sizeof(int32_t), hipMemcpyDeviceToHost, s));
  p += (size_t)st->S * sizeof(int32_t);
  COFIE_CHECK_HIP(hipMemcpyAsync(p, st->kept, (size_t)st->S * sizeof(int32_t), hipMemcpyDeviceToHost, s));
  COFIE_CHECK_HIP(hipStreamSynchronize(s));
  return COFIE_OK;
}

int cofie_ngff_stream_restore(cofie_ngff_stream* st, const void* buf, size_t bytes, void* stream) {
  clear_error();
  if (!st || !buf) return set_error(COFIE_EINVAL, "state or buffer is NULL");
  const size_t need = cofie_ngff_stream_state_bytes(st);
  if (bytes < need) return set_error(COFIE_EINVAL, "buffer of %zu bytes is smaller than the %zu required", bytes, need);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev != st->device)
    return set_error(COFIE_EINVAL, "the current device is not the state's device");
  StreamBlobHeader h;
  std::memcpy(&h, buf, sizeof h);
  const StreamBlobHeader want = blob_header(*st);
  if (std::memcmp(h.magic, want.magic, sizeof h.magic) != 0)
    return set_error(COFIE_EINVAL, "not a saved NGFF stream state (or another format version)");
  if (h.S != want.S || h.L != want.L || h.M_min != want.M_min || h.mode != want.mode || h.H != want.H ||
      h.W != want.W || h.C != want.C || h.B != want.B || h.nbins != want.nbins || h.tau_bits != want.tau_bits ||
      h.per_segment_tau != want.per_segment_tau)
    return set_error(COFIE_EINVAL, "the saved state was made with another frame shape or keep rule");
  if (h.t0 < 0 || h.t0 >= (int64_t(1) << 31) || (h.finished != 0 && h.finished != 1))
    return set_error(COFIE_EINVAL, "corrupt saved state");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const char* p = static_cast<const char*>(buf) + sizeof h;
  if (st->tau_dev) {
    std::vector<float> mine(st->S);
    COFIE_CHECK_HIP(hipMemcpyAsync(mine.data(), st->tau_dev, (size_t)st->S * sizeof(float), hipMemcpyDeviceToHost, s));
    COFIE_CHECK_HIP(hipStreamSynchronize(s));
    if (std::memcmp(mine.data(), p, (size_t)st->S * sizeof(float)) != 0)
      return set_error(COFIE_EINVAL, "the saved state was made with other per-stream thresholds");
    p += (size_t)st->S * sizeof(float);
  }
  const size_t wbytes = (size_t)st->S * st->L * st->sh.nbins * sizeof(uint32_t);
  COFIE_CHECK_HIP(hipMemcpyAsync(st->window, p, wbytes, hipMemcpyHostToDevice, s));
  p += wbytes;
  COFIE_CHECK_HIP(hipMemcpyAsync(st->r, p, (size_t)st->S * sizeof(int32_t), hipMemcpyHostToDevice, s));
  p += (size_t)st->S * sizeof(int32_t);
  COFIE_CHECK_HIP(hipMemcpyAsync(st->kept, p, (size_t)st->S * sizeof(int32_t), hipMemcpyHostToDevice, s));
  COFIE_CHECK_HIP(hipStreamSynchronize(s));
  st->t0 = h.t0;
  st->finished = h.finished != 0;
  return COFIE_OK;
}

int cofie_ngff_stream_push(cofie_ngff_stream* st, const uint8_t* frames, int64_t frames_ld, int32_t b,
                           float* out_scores, uint8_t* out_mask, int64_t ld, void* stream) {
  clear_error();
  if (!st) return set_error(COFIE_EINVAL, "state is NULL");
  if (st->finished) return set_error(COFIE_EINVAL, "the streams were finished");
  if (b < 0) return set_error(COFIE_EINVAL, "b is negative");
  if (b == 0) return COFIE_OK;
  if (!frames || !out_scores || !out_mask) return set_error(COFIE_EINVAL, "frames or an output is NULL");
  if (ld < b) return set_error(COFIE_EINVAL, "ld = %lld is smaller than b = %d", (long long)ld, b);
  if (frames_ld < b) return set_error(COFIE_EINVAL, "frames_ld = %lld is smaller than b = %d", (long long)frames_ld, b);
  if (st->t0 + b >= (int64_t(1) << 31)) return set_error(COFIE_EUNSUPPORTED, "stream longer than 2^31 frames");
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev != st->device)
    return set_error(COFIE_EINVAL, "the current device is not the state's device");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int32_t S = st->S, L = st->L;
  // pushes of at most nbmax frames per stream: the new frames' band rows sit in LDS
  const int32_t nbmax = (int32_t)std::max<int64_t>(1, std::min<int64_t>(1024, 12288 / L));
  for (int32_t j0 = 0; j0 < b; j0 += nbmax) {
    const int32_t nb = std::min(nbmax, b - j0);
    const int64_t rows = (int64_t)S * (L + nb);
    Arena plan;
    plan.take<uint32_t>((size_t)rows * st->sh.nbins);
    plan.take<int32_t>((size_t)rows * L);
    if (plan.bytes() > st->scratch_bytes) {
      // grown once for the largest push; hipFree waits for the pushes that used it
      if (st->scratch) hipFree(st->scratch);
      st->scratch = nullptr;
      st->scratch_bytes = 0;
      if (hipMalloc(&st->scratch, plan.bytes()) != hipSuccess)
        return set_error(COFIE_ENOMEM, "allocating %zu bytes of push scratch failed", plan.bytes());
      st->scratch_bytes = plan.bytes();
      st->zero_nb = -1;
    }
    Arena ar;
    ar.base = static_cast<char*>(st->scratch);
    uint32_t* comb = ar.take<uint32_t>((size_t)rows * st->sh.nbins);
    int32_t* band = ar.take<int32_t>((size_t)rows * L);
    NgffShape sh = st->sh;
    sh.n = (int64_t)S * nb;
    HistMap map;
    map.group = nb;
    map.in_stride = frames_ld;
    map.in_off = j0;
    map.out_stride = L + nb;
    map.out_off = L;
    map.out_rows = rows;
    map.zeroed = st->zero_nb == nb;  // the previous push of this size left the rows at zero
    st->zero_nb = -1;                // until this push's kernel has zeroed them again
    int rc = run_histogram(frames, sh, comb, s, map);
    if (rc) return rc;
    // the band reads each stream's first L rows (the frames before t0) from the window
    NgffShape bsh = st->sh;
    bsh.n = rows;
    RulePlan rp;
    rp.seg_len = L + nb;
    rp.nseg = S;
    rp.gap_rule = true;
    rp.L = L;
    rc = run_band(comb, bsh, rp, band, s, st->window, L);
    if (rc) return rc;
    PushArgs pa;
    pa.band = band;
    pa.L = L;
    pa.nb = nb;
    pa.t0 = st->t0;
    pa.twoM = 2 * st->sh.mass;
    pa.tau = st->tau;
    pa.tau_seg = st->tau_dev;
    pa.r_state = st->r;
    pa.kept_state = st->kept;
    pa.out_scores = out_scores + j0;
    pa.out_mask = out_mask + j0;
    pa.ld = ld;
    pa.comb = comb;
    pa.window = st->window;
    pa.nbins = st->sh.nbins;
    const size_t lds = ((size_t)nb * L + 3 * (size_t)nb + 1) * sizeof(int32_t);
    rc = allow_lds(ngff_push_kernel, lds);
    if (rc) return rc;
    rc = launch("ngff_push", ngff_push_kernel, dim3(S), dim3(1024), lds, s, pa);
    if (rc) return rc;
    st->zero_nb = nb;
    st->t0 += nb;
  }
  return COFIE_OK;
}

int cofie_ngff_stream_finish(cofie_ngff_stream* st, uint8_t* mask_all, int64_t ld, int32_t* out_added,
                             int32_t* out_count, void* stream) {
  clear_error();
  if (!st) return set_error(COFIE_EINVAL, "state is NULL");
  if (st->finished) return set_error(COFIE_EINVAL, "the streams were already finished");
  if (st->t0 > 0 && !mask_all) return set_error(COFIE_EINVAL, "mask_all is NULL");
  if (ld < st->t0) return set_error(COFIE_EINVAL, "ld is smaller than the frames pushed");
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev != st->device)
    return set_error(COFIE_EINVAL, "the current device is not the state's device");
  const int rc = launch("ngff_finish", ngff_finish_kernel, dim3((unsigned)ceil_div(st->S, 64)), dim3(64), 0,
                        static_cast<hipStream_t>(stream), mask_all, ld, st->S, st->t0, st->M_min, st->kept,
                        out_added, out_count);
  if (rc == COFIE_OK) st->finished = true;
  return rc;
}

}  // extern "C"

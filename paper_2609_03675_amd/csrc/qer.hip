// QER -- Query-Specific Evidence Refinement (Sec. 3.3) on gfx950.
//
// LOGIT mode (Eq. 6) folds the head mean into the contraction:
//   a_ij = (scale / H_q) * <q~_i, k~_j>, q~/k~ = all heads side by side,
// so the text-by-vision scores are one GEMM S^T = K Q^T with contraction
// length Lc = H_kv * d.  With grouped-query attention the query heads of a
// group are summed first (q^_g = sum_{h in g} q_h, exact in fp32) and q^ is
// carried as three bf16 terms hi + mid + lo that reproduce the fp32 value, so
// the bf16 MFMA still multiplies exact operands.
//
// qer_score: each wave owns MB x 16 visual tokens and all (<= 64) query rows
//   of one chunk; K rows stream from HBM exactly once in 16-byte lane loads, Q
//   comes from L2.  Workgroups of 4 waves split long contractions over waves
//   (KS) and add the partial tiles through LDS.  The epilogue takes the max
//   over query rows (registers, then 16-lane shuffles) and writes
//   m_j = scale * max_i S_ij: the text-by-vision matrix is never stored.
// qer_frame_mean: one wave per frame, fp64 mean of m over V_f (Eq. 7).
// qer_topk: one workgroup ranks the frames by (score desc, frame asc) on
//   order-preserving 32-bit keys (counting ranks in LDS, or a radix select for
//   very many frames) and writes the top k in chronological order (Eq. 8).
// SOFTMAX mode: per-(head, query) row statistics over all visual keys, merged
//   across workgroups, then a second pass forming the head mean of the
//   normalised probabilities and its max over query rows.
#include <cmath>

#include "common.h"

namespace cofie {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
struct bf16_t {
  uint16_t bits;
};

constexpr int kMB = 2;  // 16-token blocks per wave

template <typename T>
struct Mma;

template <>
struct Mma<bf16_t> {
  static constexpr int EPL = 8;   // elements per lane per 16-byte fragment
  static constexpr int KPS = 32;  // contraction elements per macro step
  __device__ __forceinline__ static void mac(f32x4& acc, const uint4& a, const uint4& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                  __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
  }
};

template <>
struct Mma<float> {
  static constexpr int EPL = 4;
  static constexpr int KPS = 16;
  // lane group g holds elements g*4 + e; MFMA e contracts element e of every
  // group, so 4 MFMAs cover the 16 elements of the macro step.
  __device__ __forceinline__ static void mac(f32x4& acc, const uint4& a, const uint4& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
  }
};

struct ScoreArgs {
  const uint8_t* K;   // [n_vis][Lc] elements
  const uint8_t* Qp;  // [P][nq_total][Lc] elements
  int32_t n_vis;
  int32_t n_q;        // query rows in this chunk (<= 64)
  int32_t q0;         // first query row of the chunk
  int32_t nq_total;
  int32_t Lc;
  int32_t ksteps;     // macro steps over Lc
  int32_t KS;         // waves splitting one token group's contraction (1, 2, 4)
  int32_t per_split;  // macro steps per splitting wave
  float scale;
  float* m;           // [n_vis]
  int32_t accumulate; // take the max with the m already stored (later query chunks)
};

// Loads of one batch of U macro steps starting at macro step `ms`.  Row
// pointers are clamped to valid rows, so every load is unconditional; rows past
// n_vis and query columns past n_q only produce tile entries that are never
// stored.  A partial last macro step (Lc % KPS != 0) is handled separately.
template <typename T, int MB, int NB, int P, int U>
__device__ __forceinline__ void score_load(uint4 (&fa)[U][MB], uint4 (&fb)[U][P][NB],
                                           const uint4* const (&kp)[MB],
                                           const uint4* const (&qp)[P][NB], int ms) {
  constexpr int STEP = Mma<T>::KPS * (int)sizeof(T) / 16;  // uint4 per macro step (= 4)
#pragma unroll
  for (int u = 0; u < U; ++u) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) fa[u][mb] = kp[mb][(ms + u) * STEP];
#pragma unroll
    for (int p = 0; p < P; ++p)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) fb[u][p][nb] = qp[p][nb][(ms + u) * STEP];
  }
}

template <typename T, int MB, int NB, int P, int U>
__device__ __forceinline__ void score_mac(f32x4 (&acc)[MB][NB], const uint4 (&fa)[U][MB],
                                          const uint4 (&fb)[U][P][NB]) {
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int p = 0; p < P; ++p)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) Mma<T>::mac(acc[mb][nb], fa[u][mb], fb[u][p][nb]);
}

template <typename T, int MB, int NB, int P>
__global__ __launch_bounds__(256) void qer_score_kernel(ScoreArgs a) {
  using M = Mma<T>;
  // macro steps per batch: two batches of at most 12 loads in flight
  constexpr int U = (MB + P * NB) <= 6 ? 2 : 1;
  __shared__ f32x4 part[4][MB * NB][64];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int TG = 4 / a.KS;
  const int tg = wave / a.KS, ks = wave - tg * a.KS;
  const int64_t tokbase = ((int64_t)blockIdx.x * TG + tg) * (MB * 16);
  const int64_t rowbytes = (int64_t)a.Lc * sizeof(T);

  // lane's 16-byte column (g4) of its clamped rows
  const uint4* kp[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int64_t tok = tokbase + mb * 16 + r16;
    kp[mb] = reinterpret_cast<const uint4*>(a.K + (tok < a.n_vis ? tok : 0) * rowbytes) + g4;
  }
  const uint4* qp[P][NB];
  bool qok[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int q = nb * 16 + r16;
    qok[nb] = q < a.n_q;
#pragma unroll
    for (int p = 0; p < P; ++p)
      qp[p][nb] = reinterpret_cast<const uint4*>(
                      a.Qp + ((int64_t)p * a.nq_total + a.q0 + (qok[nb] ? q : 0)) * rowbytes) + g4;
  }

  f32x4 acc[MB][NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  // this wave's macro steps [ms0, ms1); whole steps first, then the partial one
  const int full = a.Lc / M::KPS;
  const int ms0 = ks * a.per_split;
  const int ms1 = ms0 + a.per_split < a.ksteps ? ms0 + a.per_split : a.ksteps;
  const int msf = ms1 < full ? ms1 : full;
  int ms = ms0;
  if (ms + U <= msf) {
    // software pipeline: batch i+1 is in flight while batch i is multiplied
    uint4 fa[U][MB], fb[U][P][NB];
    score_load<T, MB, NB, P, U>(fa, fb, kp, qp, ms);
    for (; ms + 2 * U <= msf; ms += U) {
      uint4 ga[U][MB], gb[U][P][NB];
      score_load<T, MB, NB, P, U>(ga, gb, kp, qp, ms + U);
      score_mac<T, MB, NB, P, U>(acc, fa, fb);
#pragma unroll
      for (int u = 0; u < U; ++u) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) fa[u][mb] = ga[u][mb];
#pragma unroll
        for (int p = 0; p < P; ++p)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) fb[u][p][nb] = gb[u][p][nb];
      }
    }
    score_mac<T, MB, NB, P, U>(acc, fa, fb);
    ms += U;
  }
  for (; ms < msf; ++ms) {
    uint4 fa[1][MB], fb[1][P][NB];
    score_load<T, MB, NB, P, 1>(fa, fb, kp, qp, ms);
    score_mac<T, MB, NB, P, 1>(acc, fa, fb);
  }
  if (ms < ms1) {
    // partial macro step (bf16 with Lc % 32 == 16): lane groups past Lc read the
    // previous 16 bytes of their row and contribute zero
    const bool in = ms * M::KPS + g4 * M::EPL < a.Lc;
    const int back = in ? 0 : -2;  // uint4 offset back into the row
    const uint4 zero = {0u, 0u, 0u, 0u};
    constexpr int STEP = M::KPS * (int)sizeof(T) / 16;
    uint4 fa[1][MB], fb[1][P][NB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const uint4 v = kp[mb][ms * STEP + back];
      fa[0][mb] = in ? v : zero;
    }
#pragma unroll
    for (int p = 0; p < P; ++p)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const uint4 v = qp[p][nb][ms * STEP + back];
        fb[0][p][nb] = in ? v : zero;
      }
    score_mac<T, MB, NB, P, 1>(acc, fa, fb);
  }

  if (a.KS > 1) {
    if (ks > 0) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) part[wave][mb * NB + nb][lane] = acc[mb][nb];
    }
    __syncthreads();
    if (ks == 0) {
      for (int j = 1; j < a.KS; ++j)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) acc[mb][nb] += part[wave + j][mb * NB + nb][lane];
    }
  }
  if (ks != 0) return;

  // max over query rows: registers over nb, then the 16 lanes of a row group.
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float v = -INFINITY;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        if (qok[nb]) v = fmaxf(v, acc[mb][nb][r]);
#pragma unroll
      for (int o = 8; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 16));
      const int64_t tok = tokbase + mb * 16 + g4 * 4 + r;
      if (r16 == 0 && tok < a.n_vis) {
        const float x = v * a.scale;
        a.m[tok] = a.accumulate ? fmaxf(a.m[tok], x) : x;
      }
    }
  }
}

// ---- GQA query fold ---------------------------------------------------------------
__device__ __forceinline__ uint16_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf16_val(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// q^[i][g][x] = sum over the G query heads of group g (in head order, fp32).
// bf16 input: written as three bf16 terms [3][n_q][H_kv*d] with hi+mid+lo = q^.
// fp32 input: written as one fp32 term.
template <typename T>
__global__ void qer_fold_kernel(const T* Q, int32_t n_q, int32_t H_q, int32_t H_kv, int32_t d,
                                void* out) {
  const int64_t total = (int64_t)n_q * H_kv * d;
  const int G = H_q / H_kv;
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = e / ((int64_t)H_kv * d);
    const int64_t rem = e - i * H_kv * d;
    const int64_t g = rem / d, x = rem - g * d;
    float s = 0.f;
    for (int h = 0; h < G; ++h) {
      const int64_t src = (i * H_q + g * G + h) * d + x;
      if constexpr (sizeof(T) == 2)
        s += bf16_val(reinterpret_cast<const uint16_t*>(Q)[src]);
      else
        s += reinterpret_cast<const float*>(Q)[src];
    }
    if constexpr (sizeof(T) == 2) {
      uint16_t* o = static_cast<uint16_t*>(out);
      const uint16_t hi = bf16_rne(s);
      const float r1 = s - bf16_val(hi);
      const uint16_t mid = bf16_rne(r1);
      const float r2 = r1 - bf16_val(mid);
      o[e] = hi;
      o[total + e] = mid;
      o[2 * total + e] = bf16_rne(r2);
    } else {
      static_cast<float*>(out)[e] = s;
    }
  }
}

// ---- frame scores and top-k -----------------------------------------------------------
__device__ __forceinline__ uint32_t order_key(float w) {
  if (w != w) w = -INFINITY;  // NaN ranks as -inf
  if (w == 0.f) w = 0.f;      // -0 and +0 tie
  const uint32_t u = __float_as_uint(w);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive prefix sum over the block (blockDim a multiple of 64, <= 1024);
// returns the block total in *total.
__device__ int block_exscan(int v, int* total, int* wsum) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  int before = 0, all = 0;
  for (int i = 0; i < nw; ++i) {
    if (i < wave) before += wsum[i];
    all += wsum[i];
  }
  __syncthreads();
  *total = all;
  return before + x - v;
}

// Eq. 7: w_f = mean over the frame's visual tokens of m_j; one wave per frame,
// fp64 partial sums in a fixed lane order.  Also writes the frame's sort key.
__global__ __launch_bounds__(256) void qer_frame_mean_kernel(const float* m, int32_t n_vis,
                                                             const int32_t* offs, int32_t n_frames,
                                                             float* out_scores, uint32_t* keys) {
  const int lane = threadIdx.x & 63;
  const int64_t f = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (f >= n_frames) return;
  int lo = offs[f], hi = offs[f + 1];
  lo = lo < 0 ? 0 : (lo > n_vis ? n_vis : lo);
  hi = hi < lo ? lo : (hi > n_vis ? n_vis : hi);
  // four loads in flight per lane (clamped indices, masked adds)
  double s = 0.0;
  for (int j0 = lo + lane; j0 < hi; j0 += 256) {
    float v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int j = j0 + 64 * u;
      v[u] = m[j < hi ? j : lo];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) s += (j0 + 64 * u < hi) ? (double)v[u] : 0.0;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
  if (lane == 0) {
    const float w = hi > lo ? (float)(s / (double)(hi - lo)) : -INFINITY;
    out_scores[f] = w;
    keys[f] = order_key(w);
  }
}

constexpr int kRankMax = 4096;  // frames ranked by counting in LDS

// Eq. 8: the k frames of largest score (ties to the lower index), written in
// chronological order and padded with -1.  Up to kRankMax frames, every frame's
// rank is counted against all keys held in LDS; above that, a radix select
// finds the k-th key (8 bits per pass).
__global__ __launch_bounds__(1024) void qer_topk_kernel(const uint32_t* keys_g, int32_t n_frames,
                                                        int32_t k_top, int32_t* out_idx) {
  __shared__ uint32_t keys[kRankMax];
  __shared__ int hist[256];
  __shared__ int wsum[16];
  __shared__ uint32_t sh_prefix;
  __shared__ int sh_remaining;
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int k = k_top < n_frames ? k_top : n_frames;
  if (k > 0) {
    uint32_t kth = 0;
    int take_eq = 0;
    const bool small = n_frames <= kRankMax;
    if (small) {
      for (int f = tid; f < n_frames; f += nthr) keys[f] = keys_g[f];
      __syncthreads();
    } else {
      if (tid == 0) {
        sh_prefix = 0;
        sh_remaining = k;
      }
      uint32_t mask = 0;
      for (int shift = 24; shift >= 0; shift -= 8) {
        for (int i = tid; i < 256; i += nthr) hist[i] = 0;
        __syncthreads();
        const uint32_t prefix = sh_prefix;
        const int need = sh_remaining;
        for (int f = tid; f < n_frames; f += nthr) {
          const uint32_t key = keys_g[f];
          if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1);
        }
        __syncthreads();
        // the digit d with (count of digits > d) < need <= (count of digits >= d)
        if (tid < 256) {
          int above = 0;
          for (int e = 255; e > tid; --e) above += hist[e];
          if (above < need && above + hist[tid] >= need) {
            sh_prefix = prefix | ((uint32_t)tid << shift);
            sh_remaining = need - above;
          }
        }
        mask |= 255u << shift;
        __syncthreads();
      }
      kth = sh_prefix;
      take_eq = sh_remaining;
    }
    int eq_base = 0, out_base = 0;
    for (int f0 = 0; f0 < n_frames; f0 += nthr) {
      const int f = f0 + tid;
      int sel = 0;
      if (small) {
        if (f < n_frames) {
          const uint32_t kf = keys[f];
          int rank = 0;
          for (int g = 0; g < n_frames; ++g) {
            const uint32_t kg = keys[g];
            rank += (kg > kf) || (kg == kf && g < f);
          }
          sel = rank < k;
        }
      } else {
        const uint32_t key = f < n_frames ? keys_g[f] : 0u;
        const int is_eq = (f < n_frames && key == kth) ? 1 : 0;
        int eq_total;
        const int eq_rank = eq_base + block_exscan(is_eq, &eq_total, wsum);
        sel = (f < n_frames) && (key > kth || (is_eq && eq_rank < take_eq)) ? 1 : 0;
        eq_base += eq_total;
      }
      int sel_total;
      const int pos = out_base + block_exscan(sel, &sel_total, wsum);
      if (sel) out_idx[pos] = f;
      out_base += sel_total;
    }
  }
  for (int i = k + tid; i < k_top; i += nthr) out_idx[i] = -1;
}

// ---- SOFTMAX mode -------------------------------------------------------------------
// Per-head scores s^h_ij = scale * <q_i^h, k_j^g(h)> are recomputed in both
// passes (K is read twice).  Pass 1 writes, per workgroup of 32 tokens, the
// (max, sum of exp) of every (h, i) row over its tokens; a merge kernel folds
// them into row statistics; pass 2 forms a_ij = mean_h exp(s - max)/sum and
// m_j = max_i a_ij.
struct SoftArgs {
  const uint8_t* K;   // [n_vis][H_kv][d]
  const uint8_t* Q;   // [n_q][H_q][d]
  int32_t n_vis, n_q, H_q, H_kv, d;
  float scale;
  int32_t q0, nq;     // query chunk (nq <= 64)
  float2* partial;    // pass 1: [nblocks][H_q][n_q] (max, sumexp)
  const float2* stats;// pass 2: [H_q][n_q] (max, sumexp)
  float* m;           // pass 2 output [n_vis]
  int32_t accumulate;
};

// One wave computes the 32 x (NB*16) tile of head h for its tokens.
template <typename T, int NB>
__device__ __forceinline__ void head_tile(const SoftArgs& a, int h, int64_t tokbase, f32x4 (&acc)[kMB][NB]) {
  using M = Mma<T>;
  const int lane = threadIdx.x & 63, r16 = lane & 15, g4 = lane >> 4;
  const int g = h / (a.H_q / a.H_kv);
  const uint4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int mb = 0; mb < kMB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int steps = (a.d + M::KPS - 1) / M::KPS;
  for (int s = 0; s < steps; ++s) {
    const int kk = s * M::KPS + g4 * M::EPL;
    const bool kin = kk < a.d;
    uint4 fa[kMB], fb[NB];
#pragma unroll
    for (int mb = 0; mb < kMB; ++mb) {
      const int64_t tok = tokbase + mb * 16 + r16;
      fa[mb] = (kin && tok < a.n_vis)
                   ? *reinterpret_cast<const uint4*>(a.K + ((tok * a.H_kv + g) * a.d + kk) * (int64_t)sizeof(T))
                   : zero;
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int q = nb * 16 + r16;
      fb[nb] = (kin && q < a.nq)
                   ? *reinterpret_cast<const uint4*>(a.Q + (((int64_t)(a.q0 + q) * a.H_q + h) * a.d + kk) * (int64_t)sizeof(T))
                   : zero;
    }
#pragma unroll
    for (int mb = 0; mb < kMB; ++mb)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) M::mac(acc[mb][nb], fa[mb], fb[nb]);
  }
}

// Pass 1: workgroup = 4 waves over the same 32 tokens, heads strided over waves.
template <typename T, int NB>
__global__ __launch_bounds__(256) void qer_soft_stats_kernel(SoftArgs a) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, r16 = lane & 15, g4 = lane >> 4;
  const int64_t tokbase = (int64_t)blockIdx.x * (kMB * 16);
  for (int h = wave; h < a.H_q; h += 4) {
    f32x4 acc[kMB][NB];
    head_tile<T, NB>(a, h, tokbase, acc);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      // column (query) statistics over the valid token rows of this tile
      float mx = -INFINITY;
#pragma unroll
      for (int mb = 0; mb < kMB; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (tokbase + mb * 16 + g4 * 4 + r < a.n_vis) mx = fmaxf(mx, acc[mb][nb][r] * a.scale);
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      float se = 0.f;
#pragma unroll
      for (int mb = 0; mb < kMB; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (tokbase + mb * 16 + g4 * 4 + r < a.n_vis) se += __expf(acc[mb][nb][r] * a.scale - mx);
      se += __shfl_xor(se, 16);
      se += __shfl_xor(se, 32);
      const int q = nb * 16 + r16;
      if (g4 == 0 && q < a.nq)
        a.partial[((int64_t)blockIdx.x * a.H_q + h) * a.n_q + a.q0 + q] = make_float2(mx, se);
    }
  }
}

// Merge per-workgroup (max, sumexp) pairs into row statistics, fixed order.
__global__ void qer_soft_merge_kernel(const float2* partial, int64_t nblocks, int32_t rows,
                                      float2* stats) {
  const int64_t r = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (r >= rows) return;
  float mx = -INFINITY;
  for (int64_t b = 0; b < nblocks; ++b) mx = fmaxf(mx, partial[b * rows + r].x);
  double z = 0.0;
  for (int64_t b = 0; b < nblocks; ++b) {
    const float2 p = partial[b * rows + r];
    if (p.y > 0.f) z += (double)p.y * exp((double)p.x - (double)mx);
  }
  stats[r] = make_float2(mx, (float)z);
}

template <typename T, int NB>
__global__ __launch_bounds__(256) void qer_soft_score_kernel(SoftArgs a) {
  __shared__ f32x4 part[4][kMB * NB][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, r16 = lane & 15, g4 = lane >> 4;
  const int64_t tokbase = (int64_t)blockIdx.x * (kMB * 16);
  f32x4 prob[kMB][NB];
#pragma unroll
  for (int mb = 0; mb < kMB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) prob[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int h = wave; h < a.H_q; h += 4) {
    f32x4 acc[kMB][NB];
    head_tile<T, NB>(a, h, tokbase, acc);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int q = nb * 16 + r16;
      const float2 st = q < a.nq ? a.stats[(int64_t)h * a.n_q + a.q0 + q] : make_float2(0.f, 1.f);
      const float inv = 1.0f / st.y;
#pragma unroll
      for (int mb = 0; mb < kMB; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r) prob[mb][nb][r] += __expf(acc[mb][nb][r] * a.scale - st.x) * inv;
    }
  }
#pragma unroll
  for (int mb = 0; mb < kMB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) part[wave][mb * NB + nb][lane] = prob[mb][nb];
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int mb = 0; mb < kMB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      prob[mb][nb] = part[0][mb * NB + nb][lane] + part[1][mb * NB + nb][lane] +
                     part[2][mb * NB + nb][lane] + part[3][mb * NB + nb][lane];
  const float invH = 1.0f / (float)a.H_q;
#pragma unroll
  for (int mb = 0; mb < kMB; ++mb) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float v = -INFINITY;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        if (nb * 16 + r16 < a.nq) v = fmaxf(v, prob[mb][nb][r]);
#pragma unroll
      for (int o = 8; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 16));
      const int64_t tok = tokbase + mb * 16 + g4 * 4 + r;
      if (r16 == 0 && tok < a.n_vis) {
        const float x = v * invH;
        a.m[tok] = a.accumulate ? fmaxf(a.m[tok], x) : x;
      }
    }
  }
}

// ---- host side --------------------------------------------------------------------------

struct QerPlan {
  int64_t Lc;
  int P;           // query terms per contraction (3 for folded bf16 GQA)
  bool fold;
  size_t esize;
  int64_t nblk_soft;
};

struct QerScratch {
  float* m;
  uint32_t* keys;
  uint8_t* qp;
  float2* partial;
  float2* stats;
};

QerScratch carve_qer(Arena& ar, const cofie_qer_desc& h, const QerPlan& p) {
  QerScratch w;
  w.m = ar.take<float>((size_t)(h.n_vis > 0 ? h.n_vis : 1));
  w.keys = ar.take<uint32_t>((size_t)(h.n_frames > 0 ? h.n_frames : 1));
  w.qp = p.fold ? ar.take<uint8_t>((size_t)p.P * h.n_q * p.Lc * p.esize) : nullptr;
  if (h.score_mode == COFIE_SCORE_SOFTMAX) {
    w.partial = ar.take<float2>((size_t)p.nblk_soft * h.H_q * h.n_q);
    w.stats = ar.take<float2>((size_t)h.H_q * h.n_q);
  } else {
    w.partial = nullptr;
    w.stats = nullptr;
  }
  return w;
}

QerPlan plan_qer(const cofie_qer_desc& h) {
  QerPlan p;
  p.esize = h.dtype == COFIE_BF16 ? 2 : 4;
  p.fold = h.score_mode == COFIE_SCORE_LOGIT && h.H_q != h.H_kv;
  p.Lc = (int64_t)(p.fold ? h.H_kv : h.H_q) * h.d;  // MHA: H_q == H_kv
  p.P = (p.fold && h.dtype == COFIE_BF16) ? 3 : 1;
  p.nblk_soft = (h.n_vis + kMB * 16 - 1) / (kMB * 16);
  return p;
}

int validate_qer(const void* Q, const void* K, const int32_t* offs, const cofie_qer_desc* h,
                 int32_t k_top, const float* out_scores, const int32_t* out_idx) {
  if (!h) return set_error(COFIE_EINVAL, "heads descriptor is NULL");
  if (h->n_q < 1) return set_error(COFIE_EINVAL, "n_q = %d must be >= 1", h->n_q);
  if (h->n_vis < 0 || h->n_frames < 0) return set_error(COFIE_EINVAL, "negative n_vis or n_frames");
  if (h->H_q < 1 || h->H_kv < 1 || h->d < 1) return set_error(COFIE_EINVAL, "H_q, H_kv, d must be >= 1");
  if (h->H_q % h->H_kv != 0)
    return set_error(COFIE_EINVAL, "H_q = %d is not a multiple of H_kv = %d", h->H_q, h->H_kv);
  if (h->dtype != COFIE_F32 && h->dtype != COFIE_BF16) return set_error(COFIE_EINVAL, "unknown dtype");
  if (h->score_mode != COFIE_SCORE_LOGIT && h->score_mode != COFIE_SCORE_SOFTMAX)
    return set_error(COFIE_EINVAL, "unknown score_mode");
  if (h->d % 16 != 0) return set_error(COFIE_EUNSUPPORTED, "d = %d is not a multiple of 16", h->d);
  if (k_top < 0) return set_error(COFIE_EINVAL, "k_top is negative");
  if (!Q) return set_error(COFIE_EINVAL, "Q is NULL");
  if (h->n_vis > 0 && !K) return set_error(COFIE_EINVAL, "K is NULL");
  if (!offs) return set_error(COFIE_EINVAL, "frame_offsets is NULL");
  if (h->n_frames > 0 && !out_scores) return set_error(COFIE_EINVAL, "out_scores is NULL");
  if (k_top > 0 && !out_idx) return set_error(COFIE_EINVAL, "out_idx is NULL");
  if ((reinterpret_cast<uintptr_t>(Q) | reinterpret_cast<uintptr_t>(K)) % 16 != 0)
    return set_error(COFIE_EINVAL, "Q and K must be 16-byte aligned");
  if ((int64_t)h->n_q * h->H_q * h->d >= (int64_t(1) << 31) ||
      (int64_t)h->n_vis * h->H_kv * h->d >= (int64_t(1) << 40))
    return set_error(COFIE_EUNSUPPORTED, "tensor too large");
  return COFIE_OK;
}

template <typename T, int MB, int NB, int P>
int launch_score_t(const ScoreArgs& sa, unsigned grid, hipStream_t s) {
  return launch("qer_score", qer_score_kernel<T, MB, NB, P>, dim3(grid), dim3(256), 0, s, sa);
}

// Tokens per wave: 64 (MB = 4) halves the L2 traffic of the query fragments
// relative to the streamed keys; 32 (MB = 2) when the query side is wide.
template <typename T, int P>
int launch_score_p(const ScoreArgs& sa, int MB, int NB, unsigned grid, hipStream_t s) {
  if (MB == 4) {
    switch (NB) {
      case 1: return launch_score_t<T, 4, 1, P>(sa, grid, s);
      case 2: return launch_score_t<T, 4, 2, P>(sa, grid, s);
      case 3: return launch_score_t<T, 4, 3, P>(sa, grid, s);
      default: return launch_score_t<T, 4, 4, P>(sa, grid, s);
    }
  }
  switch (NB) {
    case 1: return launch_score_t<T, 2, 1, P>(sa, grid, s);
    case 2: return launch_score_t<T, 2, 2, P>(sa, grid, s);
    case 3: return launch_score_t<T, 2, 3, P>(sa, grid, s);
    default: return launch_score_t<T, 2, 4, P>(sa, grid, s);
  }
}

template <typename T, int NB>
int launch_soft_t(SoftArgs sa, int64_t nblk, int pass, hipStream_t s) {
  if (pass == 1)
    return launch("qer_soft_stats", qer_soft_stats_kernel<T, NB>, dim3((unsigned)nblk), dim3(256), 0, s, sa);
  return launch("qer_soft_score", qer_soft_score_kernel<T, NB>, dim3((unsigned)nblk), dim3(256), 0, s, sa);
}

template <typename T>
int launch_soft(const SoftArgs& sa, int NB, int64_t nblk, int pass, hipStream_t s) {
  switch (NB) {
    case 1: return launch_soft_t<T, 1>(sa, nblk, pass, s);
    case 2: return launch_soft_t<T, 2>(sa, nblk, pass, s);
    case 3: return launch_soft_t<T, 3>(sa, nblk, pass, s);
    default: return launch_soft_t<T, 4>(sa, nblk, pass, s);
  }
}

}  // namespace
}  // namespace cofie

using namespace cofie;

extern "C" {

size_t cofie_qer_workspace_bytes(const cofie_qer_desc* heads, int32_t k_top) {
  static const uint64_t dummy[4] = {0, 0, 0, 0};
  static const int32_t doffs = 0;
  float dscore;
  int32_t didx;
  if (validate_qer(dummy, dummy, &doffs, heads, k_top, &dscore, &didx)) return 0;
  Arena ar;
  carve_qer(ar, *heads, plan_qer(*heads));
  return ar.bytes();
}

int cofie_qer_rank(const void* Q, const void* K, const int32_t* frame_offsets,
                   const cofie_qer_desc* heads, int32_t k_top, float* out_scores,
                   int32_t* out_idx, void* stream) {
  clear_error();
  int rc = validate_qer(Q, K, frame_offsets, heads, k_top, out_scores, out_idx);
  if (rc) return rc;
  const cofie_qer_desc& h = *heads;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const QerPlan p = plan_qer(h);
  Arena plan;
  carve_qer(plan, h, p);
  Scratch scratch;
  rc = scratch.acquire(h.workspace, h.workspace_bytes, plan.bytes(), s);
  if (rc) return rc;
  Arena ar;
  ar.base = scratch.ptr();
  QerScratch w = carve_qer(ar, h, p);
  const bool bf16 = h.dtype == COFIE_BF16;
  const float base_scale = h.scale > 0.f ? h.scale : (float)(1.0 / std::sqrt((double)h.d));

  if (h.n_vis > 0) {
    if (h.score_mode == COFIE_SCORE_LOGIT) {
      const uint8_t* qp = static_cast<const uint8_t*>(Q);
      if (p.fold) {
        const int64_t total = (int64_t)h.n_q * p.Lc;
        const unsigned grid = (unsigned)std::min<int64_t>(ceil_div(total, 256), 8192);
        rc = bf16 ? launch("qer_fold", qer_fold_kernel<bf16_t>, dim3(grid), dim3(256), 0, s,
                           static_cast<const bf16_t*>(Q), h.n_q, h.H_q, h.H_kv, h.d, (void*)w.qp)
                  : launch("qer_fold", qer_fold_kernel<float>, dim3(grid), dim3(256), 0, s,
                           static_cast<const float*>(Q), h.n_q, h.H_q, h.H_kv, h.d, (void*)w.qp);
        if (rc) return rc;
        qp = w.qp;
      }
      ScoreArgs sa;
      sa.K = static_cast<const uint8_t*>(K);
      sa.Qp = qp;
      sa.n_vis = h.n_vis;
      sa.nq_total = h.n_q;
      sa.Lc = (int32_t)p.Lc;
      const int kps = bf16 ? Mma<bf16_t>::KPS : Mma<float>::KPS;
      sa.ksteps = (int32_t)((p.Lc + kps - 1) / kps);
      sa.KS = sa.ksteps >= 32 ? 4 : (sa.ksteps >= 8 ? 2 : 1);
      sa.per_split = (sa.ksteps + sa.KS - 1) / sa.KS;
      sa.scale = (float)((double)base_scale / (double)h.H_q);
      sa.m = w.m;
      const int MB = (p.P == 1) ? 4 : 2;
      const int tokens_per_wg = (4 / sa.KS) * MB * 16;
      const unsigned grid = (unsigned)ceil_div(h.n_vis, tokens_per_wg);
      for (int q0 = 0; q0 < h.n_q; q0 += 64) {
        sa.q0 = q0;
        sa.n_q = std::min(64, h.n_q - q0);
        sa.accumulate = q0 > 0;
        const int NB = (sa.n_q + 15) / 16;
        if (bf16)
          rc = p.P == 3 ? launch_score_p<bf16_t, 3>(sa, MB, NB, grid, s)
                        : launch_score_p<bf16_t, 1>(sa, MB, NB, grid, s);
        else
          rc = launch_score_p<float, 1>(sa, MB, NB, grid, s);
        if (rc) return rc;
      }
    } else {
      SoftArgs sa;
      sa.K = static_cast<const uint8_t*>(K);
      sa.Q = static_cast<const uint8_t*>(Q);
      sa.n_vis = h.n_vis;
      sa.n_q = h.n_q;
      sa.H_q = h.H_q;
      sa.H_kv = h.H_kv;
      sa.d = h.d;
      sa.scale = base_scale;
      sa.partial = w.partial;
      sa.stats = w.stats;
      sa.m = w.m;
      const int32_t rows = h.H_q * h.n_q;
      for (int q0 = 0; q0 < h.n_q; q0 += 64) {
        sa.q0 = q0;
        sa.nq = std::min(64, h.n_q - q0);
        const int NB = (sa.nq + 15) / 16;
        rc = bf16 ? launch_soft<bf16_t>(sa, NB, p.nblk_soft, 1, s) : launch_soft<float>(sa, NB, p.nblk_soft, 1, s);
        if (rc) return rc;
      }
      rc = launch("qer_soft_merge", qer_soft_merge_kernel, dim3((unsigned)ceil_div(rows, 256)), dim3(256),
                  0, s, (const float2*)w.partial, p.nblk_soft, rows, w.stats);
      if (rc) return rc;
      for (int q0 = 0; q0 < h.n_q; q0 += 64) {
        sa.q0 = q0;
        sa.nq = std::min(64, h.n_q - q0);
        sa.accumulate = q0 > 0;
        const int NB = (sa.nq + 15) / 16;
        rc = bf16 ? launch_soft<bf16_t>(sa, NB, p.nblk_soft, 2, s) : launch_soft<float>(sa, NB, p.nblk_soft, 2, s);
        if (rc) return rc;
      }
    }
  }
  if (h.n_frames > 0) {
    rc = launch("qer_frame_mean", qer_frame_mean_kernel, dim3((unsigned)ceil_div(h.n_frames, 4)),
                dim3(256), 0, s, (const float*)w.m, h.n_vis, frame_offsets, h.n_frames, out_scores,
                w.keys);
    if (rc) return rc;
  }
  if (k_top == 0) return COFIE_OK;
  return launch("qer_topk", qer_topk_kernel, dim3(1), dim3(1024), 0, s, (const uint32_t*)w.keys,
                h.n_frames, k_top, out_idx);
}

int64_t cofie_qer_k_from_ratio(double rho, int64_t n) {
  if (rho != rho || rho < 0) return -1;
  if (n <= 0) return 0;
  const double x = rho * (double)n;
  double r = std::nearbyint(x);  // default rounding mode: half to even
  int64_t k = (int64_t)r;
  return k < 1 ? 1 : k;
}

double cofie_drop_total(double d_ngff, double d_qer) { return 1.0 - (1.0 - d_ngff) * (1.0 - d_qer); }

}  // extern "C"

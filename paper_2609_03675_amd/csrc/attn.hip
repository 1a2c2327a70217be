// Last-layer prefill attention with QER read from its own QK^T tiles
// (Sec. 3.3: the scores QER needs are the ones the prefill attention already
// forms, so ranking adds no pass over the keys) on gfx950.
//
// One launch, two kinds of workgroup (8 waves each, d = 128, bf16 in, fp32
// accumulation):
//
//  * visual-row workgroups: causal flash attention of 384 visual query rows
//    (48 per wave, two waves per SIMD in a ping-pong) for one head.  Keys and
//    values stream through LDS in stages of 64 tokens (four buffers); each
//    wave
//    forms S^T = K Q^T with bf16 MFMA 16x16x32 (the queries sit in registers
//    as the B operand), keeps the running row max and sum in the base-2
//    domain, and accumulates O^T = V^T P^T with P taken straight from the
//    S^T accumulators (the key order inside a 32-key step is permuted so that
//    the accumulator layout is the B operand layout; V is stored transposed
//    in LDS in the same order).  Heaviest query blocks first; the blocks of
//    one head are kept on one XCD so that its L2 serves their key reads.
//  * text-row workgroups (first in the grid): one per 256-token chunk of the
//    key sequence and group of 128 text rows (one 16-row tile per wave),
//    looping over every head.  The per-head S^T tiles serve both the text
//    rows' attention (a partial softmax over the chunk, merged afterwards)
//    and QER: their sum over heads, kept in registers for the chunk's keys,
//    is the head-mean logit of Eq. 6 up to the factor scale / H; its max over
//    the group's text rows is m_j (Eq. 7) for the chunk's visual keys (with
//    several groups, a partial that attn_m_max reduces).
//
// attn_vt first writes V transposed (d-major rows of tokens, in the operand
// order of the value product) into the workspace; attn_merge combines the
// text rows' chunk partials (and attn_m_max the row groups' m_j);
// qer_rank_from_m then takes the frame means and the top-k (Eqs. 7-8).
#include <algorithm>
#include <cmath>

#include "common.h"

namespace cofie {

int qer_rank_from_m(const float* m, int32_t n_vis, const int32_t* offs, int32_t n_frames, int32_t k_top,
                    float* out_scores, uint32_t* keys, int32_t* out_idx, hipStream_t s);

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kD = 128;          // head dimension
constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kNT = 3;           // 16-row query tiles per wave (visual rows)
constexpr int kRowsA = 16 * kNT; // visual rows per wave
constexpr int kBM = kWaves * kRowsA;  // visual rows per workgroup
constexpr int kBN = 64;          // tokens per LDS stage
constexpr int kChunk = 256;      // tokens per text-row workgroup
constexpr int kStages = kChunk / kBN;
constexpr int kTextRows = 16 * kWaves;  // text rows per text workgroup

struct AttnArgs {
  const uint16_t* Q;  // [L][H_q][128]
  const uint16_t* K;  // [L][H_kv][128]
  const uint16_t* Vt; // [H_kv][128][Lp]: V transposed, tokens permuted (vpos32) in 32-token groups
  uint16_t* O;        // [L][H_q][128]
  int32_t L, Lp, H_q, H_kv, vb, ve, n_text, ntp;  // Lp: L rounded up to 64; ntp: text rows to 16
  int32_t n_chunks, n_rg, nb_pad, qb;  // chunks, text row groups, text workgroups (padded to 8), query blocks per head
  float c2;          // scale * log2(e)
  float qer_scale;   // scale / H_q
  float* m;          // [n_rg][ve - vb]: each row group's max (one group: m_j itself)
  float* part_o;     // [n_chunks][H_q][ntp][128]
  float2* part_ml;   // [n_chunks][H_q][ntp]: (row max, base 2; row sum)
};

__device__ __forceinline__ void mfma(f32x4& acc, const uint4& a, const uint4& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                acc, 0, 0, 0);
}

__device__ __forceinline__ uint32_t pack2(float a, float b) {
  const bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

// ---- LDS stage: 64 tokens of one key/value head ---------------------------------------
// K: [64 tokens][256 B]; V^T: [128 d][64 tokens = 128 B] (from the pre-pass
// below, already transposed, and inside each 32-token step with token k at
// vpos32(k), so that the 8 tokens lane group g of an S^T accumulator holds
// (4g..4g+3 and 16+4g..16+4g+3) are contiguous).  Both are filled by
// global-to-LDS DMA: a load instruction writes 64 lanes x 16 B to 1 KiB of
// consecutive LDS, so the bank swizzle is applied on the global side -- the
// 16-byte chunk c of key token t sits at slot c ^ (t & 15), chunk c of V^T row
// d at slot c ^ ((d >> 1) & 7).  A fragment read then touches 16 different
// bank groups, and every fragment of a stage is a per-lane base plus an
// immediate.
constexpr int kKBytes = kBN * kD * 2;              // 16 KiB
constexpr int kStageBytes = kKBytes + kD * kBN * 2;  // + 16 KiB
constexpr int kBufs = 4;                            // stage buffers of a visual-row workgroup

__host__ __device__ constexpr int vpos32(int kk) { return 8 * ((kk & 15) >> 2) + 4 * (kk >> 4) + (kk & 3); }

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void global_void;

// DMA of stage k0 of head g into st: 32 load instructions of 1 KiB, each wave
// issuing kDma of them (keys: 4 tokens each, rows clamped to the sequence;
// values: 8 rows of V^T each, k0 clamped to its last stage).
constexpr int kDma = 32 / kWaves;

// Source element (from the tensor's base) of lane l in DMA instruction i of
// stage k0 of head g: keys (i < 16) token 4 i + l / 16 of the stage (row
// clamped to the sequence), swizzled 16-byte chunk; V^T (i >= 16) row d of
// the head's transposed values, 8 tokens at the stage start (clamped to its
// last stage) plus the swizzled chunk.  The LDS destination of instruction i
// is 1 KiB at st + 1024 i (keys) or st + kKBytes + 1024 (i - 16) (values).
__host__ __device__ __forceinline__ int64_t dma_src(int i, int l, int k0, int g, int L, int Lp, int H_kv) {
  if (i < 16) {
    const int tok = 4 * i + (l >> 4), c = (l & 15) ^ (tok & 15);
    const int row = k0 + tok < L - 1 ? k0 + tok : L - 1;
    return ((int64_t)row * H_kv + g) * kD + 8 * c;
  }
  const int kv = k0 < Lp - kBN ? k0 : Lp - kBN;
  const int d = 8 * (i - 16) + (l >> 3), c = (l & 7) ^ ((d >> 1) & 7);
  return ((int64_t)g * kD + d) * Lp + kv + 8 * c;
}

__device__ __forceinline__ void stage_dma(const AttnArgs& a, int g, int k0, char* st) {
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < kDma; ++j) {
    const int i = wave + kWaves * j;  // instruction 0..31
    if (i < 16)
      __builtin_amdgcn_global_load_lds((global_void*)(a.K + dma_src(i, l, k0, g, a.L, a.Lp, a.H_kv)),
                                       (lds_void*)(st + 1024 * i), 16, 0, 0);
    else
      __builtin_amdgcn_global_load_lds((global_void*)(a.Vt + dma_src(i, l, k0, g, a.L, a.Lp, a.H_kv)),
                                       (lds_void*)(st + kKBytes + 1024 * (i - 16)), 16, 0, 0);
  }
}

// The same DMA issued through asm, for the visual rows: the compiler does not
// see these loads, so it adds no wait for them (vmcnt(0)) before LDS reads it
// cannot prove disjoint from their destination.  The visual loop orders them
// itself: each wave waits for its share of a stage before the barrier that
// publishes it, and for all of them before it ends.  M0 holds the LDS
// destination, bound through the operand constraint so that the compiler
// writes it and knows it (one wait state between that write and the load).
__device__ __forceinline__ void dma16(const void* src, char* dst) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(size_t)(lds_void*)dst);
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "{m0}"(m0) : "memory");
}

__device__ __forceinline__ void stage_dma_async(const AttnArgs& a, int g, int k0, char* st) {
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < kDma; ++j) {
    const int i = wave + kWaves * j;  // instruction 0..31
    if (i < 16)
      dma16(a.K + dma_src(i, l, k0, g, a.L, a.Lp, a.H_kv), st + 1024 * i);
    else
      dma16(a.Vt + dma_src(i, l, k0, g, a.L, a.Lp, a.H_kv), st + kKBytes + 1024 * (i - 16));
  }
}

// this wave's DMA has landed in LDS (vmcnt(0); expcnt and lgkmcnt untouched)
__device__ __forceinline__ void dma_wait() { __builtin_amdgcn_s_waitcnt(0x0F70); }
// all of this wave's DMA but its last stage (kDma loads) has landed: vector
// memory loads count down in issue order
static_assert(kDma < 16, "vmcnt field");
__device__ __forceinline__ void dma_wait_but_last() { __builtin_amdgcn_s_waitcnt(0x0F70 | kDma); }

// lane bases of the fragment reads: ka[s] for contraction step s (key tile
// kt adds kt * 4 KiB), va[sub] for token step sub (d tile dt adds dt * 2 KiB)
struct FragBase {
  int ka[4];
  int va[2];
};
__host__ __device__ __forceinline__ FragBase frag_base_of(int l) {
  const int g = l >> 4, r = l & 15;
  FragBase f;
#pragma unroll
  for (int s = 0; s < 4; ++s) f.ka[s] = r * 256 + 16 * ((4 * s + g) ^ r);
#pragma unroll
  for (int sub = 0; sub < 2; ++sub) f.va[sub] = kKBytes + r * 128 + 16 * ((4 * sub + g) ^ ((r >> 1) & 7));
  return f;
}
__device__ __forceinline__ FragBase frag_base() { return frag_base_of(threadIdx.x & 63); }
// A operand of S^T for key tile kt (16 tokens) and contraction step s (32 d)
__device__ __forceinline__ uint4 k_frag(const char* st, const FragBase& f, int kt, int s) {
  return *reinterpret_cast<const uint4*>(st + f.ka[s] + kt * 4096);
}
// A operand of O^T for d tile dt (16 d) and token step sub (32 tokens)
__device__ __forceinline__ uint4 v_frag(const char* st, const FragBase& f, int dt, int sub) {
  return *reinterpret_cast<const uint4*>(st + f.va[sub] + dt * 2048);
}

// LDS-only barrier: the stage buffers are the only shared state.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Barrier of the visual-row loop.  Its stage buffers are written only by DMA,
// and each wave waits for its own share of a stage (dma_wait_but_last) before
// the barrier that publishes it, so the barrier itself waits only for this
// wave's LDS reads (a buffer is refilled only after the barrier that follows
// its last read).  The fences of lds_barrier would add a wait for every DMA
// still in flight (vmcnt(0)) and expose the DMA latency at each barrier; the
// asm's memory clobber keeps the compiler from moving LDS reads across it.
__device__ __forceinline__ void stage_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ __forceinline__ float wave_max4(float x) {
  x = fmaxf(x, __shfl_xor(x, 16));
  return fmaxf(x, __shfl_xor(x, 32));
}
__device__ __forceinline__ float wave_sum4(float x) {
  x += __shfl_xor(x, 16);
  return x + __shfl_xor(x, 32);
}

// One head's online-softmax update for NT row tiles over a 64-token stage:
// S^T accumulators s[kt][rt] (raw dot products), masked where token > row.
template <int NT>
__device__ __forceinline__ void softmax_stage(f32x4 (&s)[4][NT], float (&m)[NT], float (&lsum)[NT],
                                              f32x4 (&o)[8][NT], uint4 (&p)[2][NT], const int (&row)[NT],
                                              int k0, bool masked, float c2) {
  const int l = threadIdx.x & 63;
#pragma unroll
  for (int rt = 0; rt < NT; ++rt) {
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float v = s[kt][rt][e] * c2;
        if (masked && k0 + 16 * kt + 4 * (l >> 4) + e > row[rt]) v = -INFINITY;
        s[kt][rt][e] = v;
        mx = fmaxf(mx, v);
      }
    mx = wave_max4(mx);
    const float mn = fmaxf(m[rt], mx);
    // a row with every token so far masked keeps m = -inf and p = 0
    const float alpha = mn == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m[rt] - mn);
    m[rt] = mn;
    lsum[rt] *= alpha;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[dt][rt] *= alpha;
    float ps[4][4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float v = mn == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(s[kt][rt][e] - mn);
        ps[kt][e] = v;
        lsum[rt] += v;
      }
#pragma unroll
    for (int sub = 0; sub < 2; ++sub)
      p[sub][rt] = make_uint4(pack2(ps[2 * sub][0], ps[2 * sub][1]), pack2(ps[2 * sub][2], ps[2 * sub][3]),
                              pack2(ps[2 * sub + 1][0], ps[2 * sub + 1][1]),
                              pack2(ps[2 * sub + 1][2], ps[2 * sub + 1][3]));
  }
}

template <int NT>
__device__ __forceinline__ void pv_stage(const char* st, const FragBase& f, f32x4 (&o)[8][NT],
                                         const uint4 (&p)[2][NT]) {
#pragma unroll
  for (int sub = 0; sub < 2; ++sub)
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      const uint4 vf = v_frag(st, f, dt, sub);
#pragma unroll
      for (int rt = 0; rt < NT; ++rt) mfma(o[dt][rt], vf, p[sub][rt]);
    }
}

template <int NT>
__device__ __forceinline__ void qk_stage(const char* st, const FragBase& f, f32x4 (&s)[4][NT],
                                         const uint4 (&q)[4][NT]) {
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
    for (int rt = 0; rt < NT; ++rt) s[kt][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const uint4 kf = k_frag(st, f, kt, ks);
#pragma unroll
      for (int rt = 0; rt < NT; ++rt) mfma(s[kt][rt], kf, q[ks][rt]);
    }
  }
}

// B operand of S^T for a query row (16 B of its head h, contraction step s)
__device__ __forceinline__ uint4 q_frag(const AttnArgs& a, int pos, int h, int s) {
  const int l = threadIdx.x & 63;
  return *reinterpret_cast<const uint4*>(a.Q + ((int64_t)pos * a.H_q + h) * kD + 32 * s + 8 * (l >> 4));
}

// ---- visual rows: causal flash attention -----------------------------------------------------
// Eight waves of 48 rows, two per SIMD, in a ping-pong: waves 4-7 run one
// barrier interval behind waves 0-3, and each wave alternates an interval of
// matrix work (the value product of one 32-token step and the key product of
// the next) with an interval of softmax, so in every interval one wave of a
// SIMD feeds the matrix core while the other uses the VALU.  Four stage
// buffers: the lagging waves still multiply the values of stage st - 1 while
// the leading ones start stage st + 1's keys, and stages st + 2 and st + 3
// are in flight (a DMA has two stages to land).  The running max is raised
// lazily: the accumulators are rescaled only when a row's max grows by more
// than kLazy (base 2), so probabilities stay below 2^kLazy and most steps
// skip the rescale.
constexpr float kLazy = 8.f;

// Max over lanes l, l ^ 16, l ^ 32 and l ^ 48: each swap hands every lane
// its own value and its partner's (one of the two pair elements is the
// lane's own).  The pair elements are read as values (__uint_as_float), not
// through __builtin_bit_cast of the vector subscript, which this compiler
// turns into two reads of element 0, i.e. no exchange at all.
__device__ __forceinline__ float max_xor16_32(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(x, fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1])));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(x, fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1])));
}

// S^T of one 32-token step (key tiles 2 half, 2 half + 1 of the stage)
__device__ __forceinline__ void qk_half(const char* st, const FragBase& f, int half, f32x4 (&s)[2][kNT],
                                        const uint4 (&q)[4][kNT]) {
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int rt = 0; rt < kNT; ++rt) s[j][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
  uint4 a = k_frag(st, f, 2 * half, 0), b = k_frag(st, f, 2 * half + 1, 0);
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    uint4 c = a, d = b;
    if (ks + 1 < 4) {
      c = k_frag(st, f, 2 * half, ks + 1);
      d = k_frag(st, f, 2 * half + 1, ks + 1);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int rt = 0; rt < kNT; ++rt) mfma(s[0][rt], a, q[ks][rt]);
#pragma unroll
    for (int rt = 0; rt < kNT; ++rt) mfma(s[1][rt], b, q[ks][rt]);
    __builtin_amdgcn_sched_barrier(0);
    a = c;
    b = d;
  }
}

// softmax of one 32-token step -> P (B operand of O^T), lazy max.  A row's
// four lanes agree on its running max m, so the max over the step's 32 keys
// is exchanged across them only when some row of the wave grows: a row's max
// exceeds m + kLazy exactly when one of its lanes' own maxima does (the
// product with c2 > 0 is monotone).  The row sums add the probabilities as
// the value product sees them, rounded to bf16, two per dot product with 1.
__device__ __forceinline__ void softmax_half(f32x4 (&s)[2][kNT], float (&m)[kNT], float (&lsum)[kNT], f32x4 (&o)[8][kNT],
                                             uint4 (&p)[kNT], const int (&row)[kNT], int k0, bool masked, float c2) {
  const int l = threadIdx.x & 63;
  if (masked) {
#pragma unroll
    for (int rt = 0; rt < kNT; ++rt)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (k0 + 16 * j + 4 * (l >> 4) + e > row[rt]) s[j][rt][e] = -INFINITY;
  }
  float mx[kNT];  // this lane's max of the raw scores
  bool grow = false;
#pragma unroll
  for (int rt = 0; rt < kNT; ++rt) {
    float v = -INFINITY;
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) v = fmaxf(v, s[j][rt][e]);
    mx[rt] = v;
    grow |= v * c2 > m[rt] + kLazy;
  }
  if (__builtin_amdgcn_ballot_w64(grow)) {
#pragma unroll
    for (int rt = 0; rt < kNT; ++rt) {
      const float r = max_xor16_32(mx[rt]) * c2;
      if (r > m[rt] + kLazy) {
        const float alpha = __builtin_amdgcn_exp2f(m[rt] - r);  // m = -inf: 0
        m[rt] = r;
        lsum[rt] *= alpha;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) o[dt][rt] *= alpha;
      }
    }
  }
  constexpr uint32_t kOnes = 0x3f803f80u;  // bf16 pair (1, 1)
#pragma unroll
  for (int rt = 0; rt < kNT; ++rt) {
    float pv[2][4];
    const float nm = -m[rt];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) pv[j][e] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[j][rt][e], c2, nm));
    const uint32_t u0 = pack2(pv[0][0], pv[0][1]), u1 = pack2(pv[0][2], pv[0][3]);
    const uint32_t u2 = pack2(pv[1][0], pv[1][1]), u3 = pack2(pv[1][2], pv[1][3]);
    float ls = lsum[rt];
    ls = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, u0), __builtin_bit_cast(bf16x2, kOnes), ls, false);
    ls = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, u1), __builtin_bit_cast(bf16x2, kOnes), ls, false);
    ls = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, u2), __builtin_bit_cast(bf16x2, kOnes), ls, false);
    ls = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, u3), __builtin_bit_cast(bf16x2, kOnes), ls, false);
    lsum[rt] = ls;
    p[rt] = make_uint4(u0, u1, u2, u3);
  }
}

__device__ __forceinline__ void pv_half(const char* st, const FragBase& f, int half, f32x4 (&o)[8][kNT],
                                        const uint4 (&p)[kNT]) {
  // fragment reads one pair ahead of the pair being multiplied (the order is
  // pinned: by itself the scheduler waits for each pair right after its reads)
  uint4 a = v_frag(st, f, 0, half), b = v_frag(st, f, 1, half);
#pragma unroll
  for (int dt = 0; dt < 8; dt += 2) {
    uint4 c = a, d = b;
    if (dt + 2 < 8) {
      c = v_frag(st, f, dt + 2, half);
      d = v_frag(st, f, dt + 3, half);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int rt = 0; rt < kNT; ++rt) mfma(o[dt][rt], a, p[rt]);
#pragma unroll
    for (int rt = 0; rt < kNT; ++rt) mfma(o[dt + 1][rt], b, p[rt]);
    __builtin_amdgcn_sched_barrier(0);
    a = c;
    b = d;
  }
}

// Visual workgroup b: its head and query block (the blocks of one XCD take
// consecutive work; heaviest, i.e. latest, blocks first within a head).
__host__ __device__ __forceinline__ void visual_map(int b, int n_qb, int H_q, int& h, int& qb) {
  const int total = n_qb * H_q, t8 = total / 8;
  const int w = b < 8 * t8 ? (b % 8) * t8 + b / 8 : b;
  h = w / n_qb;
  qb = n_qb - 1 - w % n_qb;
}

__device__ void visual_block(const AttnArgs& a, int b, char* lds) {
  int h, qb;
  visual_map(b, a.qb, a.H_q, h, qb);
  const int g = h / (a.H_q / a.H_kv);
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  const bool lag = wave >= kWaves / 2;  // one interval behind
  const int r0 = a.vb + kBM * qb, rw = r0 + kRowsA * wave;
  const int last = min(r0 + kBM, a.ve) - 1;  // last query row of the block
  const int nst = last / kBN + 1;
  // stages this wave sees (0 if it has no rows): tokens up to its last row
  const int nsw = rw < a.ve ? min(nst, (min(rw + kRowsA, a.ve) - 1) / kBN + 1) : 0;

  uint4 q[4][kNT];
  int row[kNT];
#pragma unroll
  for (int rt = 0; rt < kNT; ++rt) {
    row[rt] = rw + 16 * rt + (l & 15);
    const int pos = min(row[rt], a.L - 1);
#pragma unroll
    for (int s = 0; s < 4; ++s) q[s][rt] = q_frag(a, pos, h, s);
  }
  f32x4 o[8][kNT];
  float m[kNT], lsum[kNT];
#pragma unroll
  for (int rt = 0; rt < kNT; ++rt) {
    m[rt] = -INFINITY;
    lsum[rt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[dt][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const FragBase fb = frag_base();

  // the query fragments have arrived: the compiler then tracks no load of
  // its own into the loop, where its counted waits would also wait for the
  // stage DMA in flight
  dma_wait();
  stage_dma_async(a, g, 0, lds);
  stage_dma_async(a, g, kBN, lds + kStageBytes);
  stage_dma_async(a, g, 2 * kBN, lds + 2 * kStageBytes);
  dma_wait_but_last();  // stages 0 and 1
  stage_barrier();
  if (lag) stage_barrier();

  f32x4 s[2][kNT];
  uint4 p[kNT];
  for (int st = 0; st <= nst; ++st) {
    const char* cur = lds + (st % kBufs) * kStageBytes;
    const char* prev = lds + ((st + kBufs - 1) % kBufs) * kStageBytes;
    const int k0 = st * kBN;
    const bool on = st < nsw, was = st > 0 && st - 1 < nsw;
    const bool masked = k0 + kBN - 1 > rw;
    // Stage st + 3 goes into the buffer of stage st - 1 in the interval after
    // that buffer's last read (a lagging wave's interval 0): the leading waves
    // in their interval 2, the lagging ones in their interval 1 -- the same
    // interval of the workgroup.  Each wave first waits for its share of stage
    // st + 1 (stage st + 2's may still be in flight), which the following
    // barrier then publishes.
    char* next = lds + ((st + kBufs - 1) % kBufs) * kStageBytes;
    // interval 0: values of the previous stage's second step, keys of this
    // stage's first step
    if (was) pv_half(prev, fb, 1, o, p);
    if (on) qk_half(cur, fb, 0, s, q);
    stage_barrier();
    if (st == nst) break;
    // interval 1: softmax of the first step
    if (lag) {
      dma_wait_but_last();
      stage_dma_async(a, g, k0 + 3 * kBN, next);
    }
    if (on) softmax_half(s, m, lsum, o, p, row, k0, masked, a.c2);
    stage_barrier();
    // interval 2: values of the first step, keys of the second
    if (!lag) {
      dma_wait_but_last();
      stage_dma_async(a, g, k0 + 3 * kBN, next);
    }
    if (on) {
      pv_half(cur, fb, 0, o, p);
      qk_half(cur, fb, 1, s, q);
    }
    stage_barrier();
    // interval 3: softmax of the second step
    if (on) softmax_half(s, m, lsum, o, p, row, k0 + 32, masked, a.c2);
    stage_barrier();
  }
  if (!lag) stage_barrier();
  dma_wait();  // no DMA may land in LDS after the workgroup is gone
  if (nsw == 0) return;
#pragma unroll
  for (int rt = 0; rt < kNT; ++rt) {
    float ls = lsum[rt];
    ls += __shfl_xor(ls, 16);
    ls += __shfl_xor(ls, 32);
    const float inv = 1.f / ls;
    if (row[rt] >= a.ve) continue;
    uint16_t* out = a.O + ((int64_t)row[rt] * a.H_q + h) * kD + 4 * (l >> 4);
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      const f32x4 v = o[dt][rt] * inv;
      *reinterpret_cast<uint2*>(out + 16 * dt) = make_uint2(pack2(v[0], v[1]), pack2(v[2], v[3]));
    }
  }
}

// ---- text rows: chunk partials of their attention, and QER's m_j --------------------------
__device__ void text_block(const AttnArgs& a, int c, int rg, char* lds, float* red) {
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int c0 = c * kChunk;
  const int nst = min(kStages, (a.L - c0 + kBN - 1) / kBN);
  const int tr = kTextRows * rg + 16 * wave + (l & 15);  // text row of this lane
  const bool valid = tr < a.n_text;
  const int pos = tr < a.vb ? tr : a.ve + (tr - a.vb);
  const bool active = kTextRows * rg + 16 * wave < a.n_text;
  int row[1] = {valid ? pos : -1};      // an invalid row sees no token

  f32x4 acc[kStages][4];                // sum over heads of S^T, the chunk's tokens
#pragma unroll
  for (int i = 0; i < kStages; ++i)
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) acc[i][kt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int per = a.H_q / a.H_kv;
  const FragBase fb = frag_base();
  stage_dma(a, 0, c0, lds);
  dma_wait();
  lds_barrier();
  int buf = 0;
  for (int h = 0; h < a.H_q; ++h) {
    uint4 q[4][1];
    const int qpos = valid ? pos : 0;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      q[s][0] = q_frag(a, qpos, h, s);
      if (!valid) q[s][0] = make_uint4(0, 0, 0, 0);
    }
    f32x4 o[8][1];
    float m[1] = {-INFINITY}, lsum[1] = {0.f};
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[dt][0] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < kStages; ++st) {
      if (st < nst) {
        const int k0 = c0 + st * kBN;
        const bool more = st + 1 < nst || h + 1 < a.H_q;
        if (more) {  // into the other buffer, whose readers passed the last barrier
          const int nh = st + 1 < nst ? h : h + 1;
          stage_dma(a, nh / per, st + 1 < nst ? k0 + kBN : c0, lds + (buf ^ 1) * kStageBytes);
        }
        const char* cur = lds + buf * kStageBytes;
        if (active) {
          f32x4 s[4][1];
          uint4 p[2][1];
          qk_stage<1>(cur, fb, s, q);
#pragma unroll
          for (int kt = 0; kt < 4; ++kt) acc[st][kt] += s[kt][0];
          softmax_stage<1>(s, m, lsum, o, p, row, k0, true, a.c2);
          pv_stage<1>(cur, fb, o, p);
        }
        dma_wait();
        lds_barrier();
        buf ^= 1;
      }
    }
    const float ltot = wave_sum4(lsum[0]);
    if (valid) {
      const int64_t pr = ((int64_t)c * a.H_q + h) * a.ntp + tr;
      if ((l >> 4) == 0) a.part_ml[pr] = make_float2(m[0], ltot);
      float* po = a.part_o + pr * kD + 4 * (l >> 4);
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) *reinterpret_cast<f32x4*>(po + 16 * dt) = o[dt][0];
    }
  }

  dma_wait();
  // m_j: max over the text rows of the head sum, the chunk's visual tokens
  for (int i = threadIdx.x; i < kWaves * kChunk; i += kThreads) red[i] = -INFINITY;
  __syncthreads();
  if (active) {
#pragma unroll
    for (int st = 0; st < kStages; ++st)
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float v = valid ? acc[st][kt][e] : -INFINITY;
          // max over the 16 lanes of the row (rotations within a DPP row)
          v = fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                                             0x128, 0xF, 0xF, false)));
          v = fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                                             0x124, 0xF, 0xF, false)));
          v = fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                                             0x122, 0xF, 0xF, false)));
          v = fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                                             0x121, 0xF, 0xF, false)));
          if ((l & 15) == 0) red[wave * kChunk + st * kBN + 16 * kt + 4 * (l >> 4) + e] = v;
        }
  }
  __syncthreads();
  float* m = a.m + (int64_t)rg * (a.ve - a.vb);
  for (int i = threadIdx.x; i < kChunk; i += kThreads) {
    const int tok = c0 + i;
    if (tok >= a.vb && tok < a.ve) {
      float v = red[i];
#pragma unroll
      for (int w = 1; w < kWaves; ++w) v = fmaxf(v, red[w * kChunk + i]);
      m[tok - a.vb] = v * a.qer_scale;
    }
  }
}

// m_j over several text row groups: the max of their partial maxima.
__global__ void attn_m_max_kernel(const float* part, int32_t n_vis, int32_t n_rg, float* m) {
  for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < n_vis; j += (int64_t)gridDim.x * blockDim.x) {
    float v = part[j];
    for (int r = 1; r < n_rg; ++r) v = fmaxf(v, part[(int64_t)r * n_vis + j]);
    m[j] = v;
  }
}

__global__ __launch_bounds__(kThreads, 1) void attn_qer_kernel(AttnArgs a) {
  extern __shared__ __align__(16) char lds[];
  const int b = blockIdx.x;
  if (b < a.nb_pad) {
    if (b < a.n_chunks * a.n_rg)
      text_block(a, b % a.n_chunks, b / a.n_chunks, lds, reinterpret_cast<float*>(lds + 2 * kStageBytes));
    return;
  }
  visual_block(a, b - a.nb_pad, lds);
}

// V^T for the value stages: Vt[g][d][p] = V[k][g][d] with p = 32 (k / 32) +
// vpos32(k % 32), zero past L.  One workgroup per 64 tokens and head, the
// tile transposed through LDS; 16-byte loads and stores.
constexpr int kLoads = 1024 / kThreads;  // 16-byte chunks per thread of a 64-token tile

__global__ __launch_bounds__(kThreads) void attn_vt_kernel(const uint16_t* V, int32_t L, int32_t H_kv, int32_t Lp,
                                                           uint16_t* Vt) {
  __shared__ __align__(16) uint16_t tile[kBN][kD + 8];
  const int k0 = blockIdx.x * kBN, g = blockIdx.y, t = threadIdx.x;
#pragma unroll
  for (int i = 0; i < kLoads; ++i) {
    const int id = t + kThreads * i, tok = id >> 4, c = id & 15;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (k0 + tok < L) v = *reinterpret_cast<const uint4*>(V + ((int64_t)(k0 + tok) * H_kv + g) * kD + 8 * c);
    *reinterpret_cast<uint4*>(&tile[tok][8 * c]) = v;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kLoads; ++i) {
    const int id = t + kThreads * i, d = id >> 3, q = id & 7;
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      uint32_t pair = 0;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int p = 8 * q + 2 * e + h;  // position in the stage
        const int half = p >> 5, pp = p & 31, grp = pp >> 3, j = pp & 7;
        const int tok = 32 * half + 4 * grp + (j & 3) + 16 * (j >> 2);  // the token at position p
        pair |= (uint32_t)tile[tok][d] << (16 * h);
      }
      w[e] = pair;
    }
    *reinterpret_cast<uint4*>(Vt + ((int64_t)g * kD + d) * Lp + k0 + 8 * q) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// Text rows: O = sum_c 2^(m_c - M) O_c / sum_c 2^(m_c - M) l_c over the chunks.
__global__ __launch_bounds__(kD) void attn_merge_kernel(AttnArgs a) {
  // One workgroup per text row and head, a thread per d.  The chunks' maxima
  // are read in parallel (a thread per chunk), then the chunks are taken in
  // blocks of kD: their weights exp2(m_c - M) go through LDS and every thread
  // accumulates its d over the block with independent loads (a chunk no key
  // of which the row sees has m_c = -inf, weight 0 and a zero partial).
  __shared__ float red[kD / 64];
  __shared__ float wsh[kD];
  const int tr = blockIdx.x, h = blockIdx.y, d = threadIdx.x;
  const int pos = tr < a.vb ? tr : a.ve + (tr - a.vb);
  const int64_t base = (int64_t)h * a.ntp + tr, cstride = (int64_t)a.H_q * a.ntp;
  float M = -INFINITY;
  for (int c = d; c < a.n_chunks; c += kD) M = fmaxf(M, a.part_ml[c * cstride + base].x);
  for (int o = 32; o > 0; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
  if ((d & 63) == 0) red[d >> 6] = M;
  __syncthreads();
  M = red[0];
#pragma unroll
  for (int w = 1; w < kD / 64; ++w) M = fmaxf(M, red[w]);
  float lpart = 0.f, acc = 0.f;
  for (int c0 = 0; c0 < a.n_chunks; c0 += kD) {
    const int c = c0 + d;
    float wgt = 0.f;
    if (c < a.n_chunks) {
      const float2 ml = a.part_ml[c * cstride + base];
      if (ml.x != -INFINITY) {
        wgt = exp2f(ml.x - M);
        lpart += wgt * ml.y;
      }
    }
    __syncthreads();  // the previous block's weights have been read
    wsh[d] = wgt;
    __syncthreads();
    const int n = a.n_chunks - c0 < kD ? a.n_chunks - c0 : kD;
    const float* po = a.part_o + (c0 * cstride + base) * kD + d;
#pragma unroll 8
    for (int j = 0; j < n; ++j) acc = fmaf(wsh[j], po[j * cstride * kD], acc);
  }
  for (int o = 32; o > 0; o >>= 1) lpart += __shfl_xor(lpart, o);
  __syncthreads();
  if ((d & 63) == 0) red[d >> 6] = lpart;
  __syncthreads();
  float lsum = 0.f;
#pragma unroll
  for (int w = 0; w < kD / 64; ++w) lsum += red[w];
  const __bf16 v = (__bf16)(acc / lsum);
  a.O[((int64_t)pos * a.H_q + h) * kD + d] = __builtin_bit_cast(uint16_t, v);
}

struct AttnPlan {
  int32_t n_vis, n_text, ntp, n_chunks, n_rg, nb_pad, qb, Lp;
};

AttnPlan plan_attn(const cofie_attn_desc& h) {
  AttnPlan p;
  p.n_vis = h.vis_end - h.vis_begin;
  p.n_text = h.L - p.n_vis;
  p.ntp = (p.n_text + 15) / 16 * 16;
  p.n_chunks = ceil_div(h.L, kChunk);
  p.n_rg = ceil_div(p.n_text, kTextRows);
  p.nb_pad = (p.n_chunks * p.n_rg + 7) / 8 * 8;
  p.qb = ceil_div(p.n_vis, kBM);
  p.Lp = ceil_div(h.L, kBN) * kBN;
  return p;
}

void carve_attn(Arena& ar, const cofie_attn_desc& h, const AttnPlan& p, float** m, float** mpart, uint32_t** keys,
                float** po, float2** pml, uint16_t** vt) {
  *vt = ar.take<uint16_t>((size_t)h.H_kv * kD * p.Lp);
  *m = ar.take<float>((size_t)(p.n_vis > 0 ? p.n_vis : 1));
  *mpart = p.n_rg > 1 ? ar.take<float>((size_t)p.n_rg * (p.n_vis > 0 ? p.n_vis : 1)) : *m;
  *keys = ar.take<uint32_t>((size_t)(h.n_frames > 0 ? h.n_frames : 1));
  *po = ar.take<float>((size_t)p.n_chunks * h.H_q * p.ntp * kD);
  *pml = ar.take<float2>((size_t)p.n_chunks * h.H_q * p.ntp);
}

int validate_attn(const void* Q, const void* K, const void* V, const int32_t* offs, const cofie_attn_desc* h,
                  int32_t k_top, const void* out, const float* out_scores, const int32_t* out_idx) {
  if (!h) return set_error(COFIE_EINVAL, "descriptor is NULL");
  if (h->L < 1) return set_error(COFIE_EINVAL, "L = %d must be >= 1", h->L);
  if (h->H_q < 1 || h->H_kv < 1 || h->H_q % h->H_kv != 0)
    return set_error(COFIE_EINVAL, "H_q = %d, H_kv = %d: both >= 1 and H_q a multiple of H_kv", h->H_q, h->H_kv);
  if (h->d != kD) return set_error(COFIE_EUNSUPPORTED, "head dimension %d (only 128 is built)", h->d);
  if (h->vis_begin < 0 || h->vis_end < h->vis_begin || h->vis_end > h->L)
    return set_error(COFIE_EINVAL, "visual range [%d, %d) outside [0, L = %d]", h->vis_begin, h->vis_end, h->L);
  const int32_t n_text = h->L - (h->vis_end - h->vis_begin);
  if (n_text < 1) return set_error(COFIE_EINVAL, "no text token outside the visual range");
  if (h->n_frames < 0) return set_error(COFIE_EINVAL, "n_frames is negative");
  if (k_top < 0) return set_error(COFIE_EINVAL, "k_top is negative");
  if (!Q || !K || !V || !out) return set_error(COFIE_EINVAL, "Q, K, V or out is NULL");
  if (!offs) return set_error(COFIE_EINVAL, "frame_offsets is NULL");
  if (h->n_frames > 0 && !out_scores) return set_error(COFIE_EINVAL, "out_scores is NULL");
  if (k_top > 0 && !out_idx) return set_error(COFIE_EINVAL, "out_idx is NULL");
  if ((reinterpret_cast<uintptr_t>(Q) | reinterpret_cast<uintptr_t>(K) | reinterpret_cast<uintptr_t>(V) |
       reinterpret_cast<uintptr_t>(out)) % 16 != 0)
    return set_error(COFIE_EINVAL, "Q, K, V and out must be 16-byte aligned");
  if ((int64_t)h->L * h->H_q * kD >= (int64_t(1) << 40)) return set_error(COFIE_EUNSUPPORTED, "tensor too large");
  return COFIE_OK;
}

constexpr size_t kLdsBytes = kBufs * kStageBytes;  // 128 KiB (the text rows use 2 stages + 8 KiB)
static_assert(2 * kStageBytes + kWaves * kChunk * sizeof(float) <= kLdsBytes, "text rows' LDS");

// Address model of the fused call (dry run): the transpose pre-pass, every
// visual and text workgroup's DMA stages (at both ends of their affine
// ranges), fragment reads, query loads and stores, the merge and the
// row-group maximum, through the kernels' own index functions.
void model_attn(const AttnArgs& a, const uint16_t* V, int H_q) {
  const int64_t lds = (int64_t)kLdsBytes;
  // fragment reads: inside one stage, for every lane
  for (int l = 0; l < 64; ++l) {
    const FragBase f = frag_base_of(l);
    for (int s = 0; s < 4; ++s) {
      dry_range(f.ka[s] + 3 * 4096 + 16, 0, kKBytes + 1, "attn: key fragment past the stage's keys");
      dry_range(f.ka[s], 0, kKBytes, "attn: key fragment");
    }
    for (int sub = 0; sub < 2; ++sub) {
      dry_range(f.va[sub] + 7 * 2048 + 16, kKBytes, kStageBytes + 1, "attn: value fragment past the stage");
      dry_range(f.va[sub], kKBytes, kStageBytes, "attn: value fragment");
    }
  }
  // one DMA stage: the extreme lanes of each instruction (rows and columns
  // are monotone in the token, the swizzled chunk stays in its row)
  auto dma = [&](int g, int k0, int64_t st) {
    for (int i = 0; i < 32; ++i) {
      dry_lds(st + (i < 16 ? 1024 * i : kKBytes + 1024 * (i - 16)), 1024, lds, "attn: DMA destination");
      for (int l : {0, 15, 48, 63}) {
        const int64_t e = dma_src(i, l, k0, g, a.L, a.Lp, a.H_kv);
        dry_access(i < 16 ? (const void*)a.K : (const void*)a.Vt, 2 * e, 16, "attn: DMA source");
      }
    }
  };
  // V^T pre-pass: token tiles of 64 for every key head
  for (int g = 0; g < a.H_kv; ++g)
    for (int k0 = 0; k0 < a.Lp; k0 += kBN) {
      const int last = k0 + kBN - 1 < a.L - 1 ? k0 + kBN - 1 : a.L - 1;
      if (k0 < a.L) dry_access(V, 2 * (((int64_t)last * a.H_kv + g) * kD + 8 * 15), 16, "attn: V load");
      dry_access(a.Vt, 2 * (((int64_t)g * kD + kD - 1) * a.Lp + k0 + 56), 16, "attn: V^T store");
    }
  const int per = a.H_q / a.H_kv;
  // text workgroups: chunk c, row group rg, every head
  for (int b = 0; b < a.n_chunks * a.n_rg; ++b) {
    const int c = b % a.n_chunks, rg = b / a.n_chunks, c0 = c * kChunk;
    const int nst = (a.L - c0 + kBN - 1) / kBN < kStages ? (a.L - c0 + kBN - 1) / kBN : kStages;
    int buf = 0;
    dma(0, c0, 0);
    for (int h = 0; h < a.H_q; ++h)
      for (int st = 0; st < nst; ++st) {
        const int k0 = c0 + st * kBN;
        if (st + 1 < nst || h + 1 < a.H_q)
          dma((st + 1 < nst ? h : h + 1) / per, st + 1 < nst ? k0 + kBN : c0, (buf ^ 1) * (int64_t)kStageBytes);
        buf ^= 1;
      }
    for (int wave = 0; wave < kWaves; ++wave) {
      const int tr_hi = kTextRows * rg + 16 * wave + 15, tr_lo = kTextRows * rg + 16 * wave;
      if (tr_lo >= a.n_text) continue;
      const int tr = tr_hi < a.n_text ? tr_hi : a.n_text - 1;
      const int pos = tr < a.vb ? tr : a.ve + (tr - a.vb);
      dry_range(pos, 0, a.L, "attn: text row position");
      dry_access(a.Q, 2 * (((int64_t)pos * a.H_q + H_q - 1) * kD + 32 * 3 + 8 * 3), 16, "attn: text query load");
      const int64_t pr = ((int64_t)c * a.H_q + H_q - 1) * a.ntp + tr;
      dry_access(a.part_ml, 8 * pr, 8, "attn: text row statistics");
      dry_access(a.part_o, 4 * (pr * kD + 4 * 3 + 16 * 7), 16, "attn: text row partial");
      dry_lds(2 * (int64_t)kStageBytes + 4 * (wave * kChunk + kChunk - 1), 4, lds, "attn: row-group maxima");
    }
    const int lo = c0 > a.vb ? c0 : a.vb, hi = c0 + kChunk < a.ve ? c0 + kChunk : a.ve;
    if (hi > lo) dry_access(a.m, 4 * ((int64_t)rg * (a.ve - a.vb) + lo - a.vb), 4 * (int64_t)(hi - lo), "attn: m_j");
  }
  // visual workgroups
  for (int b = 0; b < a.qb * a.H_q; ++b) {
    int h, qb;
    visual_map(b, a.qb, a.H_q, h, qb);
    dry_range(h, 0, a.H_q, "attn: visual head");
    const int g = h / per;
    const int r0 = a.vb + kBM * qb;
    const int last = (r0 + kBM < a.ve ? r0 + kBM : a.ve) - 1;
    const int nst = last / kBN + 1;
    for (int st = 0; st < kBufs - 1; ++st) dma(g, st * kBN, st * (int64_t)kStageBytes);
    for (int st = 0; st < nst; ++st) dma(g, (st + 3) * kBN, ((st + 3) % kBufs) * (int64_t)kStageBytes);
    const int pos_lo = r0 < a.L - 1 ? r0 : a.L - 1;
    const int pos_hi = r0 + kBM - 1 < a.L - 1 ? r0 + kBM - 1 : a.L - 1;
    dry_access(a.Q, 2 * (((int64_t)pos_lo * a.H_q + h) * kD), 16, "attn: visual query load");
    dry_access(a.Q, 2 * (((int64_t)pos_hi * a.H_q + h) * kD + 32 * 3 + 8 * 3), 16, "attn: visual query load");
    if (last >= r0) {
      dry_access(a.O, 2 * (((int64_t)r0 * a.H_q + h) * kD), 8, "attn: output row");
      dry_access(a.O, 2 * (((int64_t)last * a.H_q + h) * kD + 4 * 3 + 16 * 7), 8, "attn: output row");
    }
  }
  // merge of the text rows (every chunk's partials) and their outputs
  if (a.n_text > 0) {
    const int tr = a.n_text - 1, pos = tr < a.vb ? tr : a.ve + (tr - a.vb);
    const int64_t pr = ((int64_t)(a.n_chunks - 1) * a.H_q + a.H_q - 1) * a.ntp + tr;
    dry_access(a.part_ml, 8 * pr, 8, "attn: merge statistics");
    dry_access(a.part_o, 4 * (pr * kD + kD - 1), 4, "attn: merge partial");
    dry_access(a.O, 2 * (((int64_t)pos * a.H_q + a.H_q - 1) * kD + kD - 1), 2, "attn: merged output");
  }
}


}  // namespace
}  // namespace cofie

using namespace cofie;

extern "C" {

size_t cofie_attn_qer_workspace_bytes(const cofie_attn_desc* desc) {
  static const uint64_t dummy[4] = {0, 0, 0, 0};
  static const int32_t doffs = 0;
  float ds;
  int32_t di;
  if (validate_attn(dummy, dummy, dummy, &doffs, desc, 0, dummy, &ds, &di)) return 0;
  Arena ar;
  float *m, *mpart, *po;
  uint32_t* keys;
  float2* pml;
  uint16_t* vt;
  carve_attn(ar, *desc, plan_attn(*desc), &m, &mpart, &keys, &po, &pml, &vt);
  return ar.bytes();
}

int cofie_attn_qer(const void* Q, const void* K, const void* V, const int32_t* frame_offsets,
                   const cofie_attn_desc* desc, int32_t k_top, void* out, float* out_scores, int32_t* out_idx,
                   void* stream) {
  clear_error();
  int rc = validate_attn(Q, K, V, frame_offsets, desc, k_top, out, out_scores, out_idx);
  if (rc) return rc;
  const cofie_attn_desc& h = *desc;
  const AttnPlan p = plan_attn(h);
  hipStream_t s = static_cast<hipStream_t>(stream);
  Arena plan;
  float *m, *mpart, *po;
  uint32_t* keys;
  float2* pml;
  uint16_t* vt;
  carve_attn(plan, h, p, &m, &mpart, &keys, &po, &pml, &vt);
  Scratch scratch;
  rc = scratch.acquire(h.workspace, h.workspace_bytes, plan.bytes(), s);
  if (rc) return rc;
  Arena ar;
  ar.base = scratch.ptr();
  carve_attn(ar, h, p, &m, &mpart, &keys, &po, &pml, &vt);

  AttnArgs a;
  a.Q = static_cast<const uint16_t*>(Q);
  a.K = static_cast<const uint16_t*>(K);
  a.Vt = vt;
  a.O = static_cast<uint16_t*>(out);
  a.L = h.L;
  a.Lp = p.Lp;
  a.H_q = h.H_q;
  a.H_kv = h.H_kv;
  a.vb = h.vis_begin;
  a.ve = h.vis_end;
  a.n_text = p.n_text;
  a.ntp = p.ntp;
  a.n_chunks = p.n_chunks;
  a.n_rg = p.n_rg;
  a.nb_pad = p.nb_pad;
  a.qb = p.qb;
  const double scale = h.scale > 0.f ? (double)h.scale : 1.0 / std::sqrt((double)kD);
  a.c2 = (float)(scale * 1.4426950408889634);
  a.qer_scale = (float)(scale / (double)h.H_q);
  a.m = mpart;
  a.part_o = po;
  a.part_ml = pml;
  if (dry_run()) model_attn(a, static_cast<const uint16_t*>(V), h.H_q);
  rc = launch("attn_vt", attn_vt_kernel, dim3((unsigned)(p.Lp / kBN), (unsigned)h.H_kv), dim3(kThreads), 0, s,
              static_cast<const uint16_t*>(V), h.L, h.H_kv, p.Lp, vt);
  if (rc) return rc;
  rc = allow_lds(attn_qer_kernel, kLdsBytes);
  if (rc) return rc;
  const int64_t blocks = (int64_t)p.nb_pad + (int64_t)p.qb * h.H_q;
  rc = launch("attn_qer", attn_qer_kernel, dim3((unsigned)blocks), dim3(kThreads), kLdsBytes, s, a);
  if (rc) return rc;
  rc = launch("attn_merge", attn_merge_kernel, dim3((unsigned)p.n_text, (unsigned)h.H_q), dim3(kD), 0, s, a);
  if (rc) return rc;
  if (p.n_rg > 1 && p.n_vis > 0) {
    if (dry_run()) {
      dry_access(mpart, 0, 4 * (int64_t)p.n_rg * p.n_vis, "attn: row-group maxima");
      dry_access(m, 0, 4 * (int64_t)p.n_vis, "attn: m_j");
    }
    rc = launch("attn_m_max", attn_m_max_kernel, dim3((unsigned)std::min(ceil_div(p.n_vis, 256), 1024)), dim3(256), 0,
                s, (const float*)mpart, p.n_vis, p.n_rg, m);
    if (rc) return rc;
  }
  return qer_rank_from_m(m, p.n_vis, frame_offsets, h.n_frames, k_top, out_scores, keys, out_idx, s);
}

}  // extern "C"

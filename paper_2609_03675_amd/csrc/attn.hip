// Last-layer prefill attention with QER read from its own QK^T tiles
// (Sec. 3.3: the scores QER needs are the ones the prefill attention already
// forms, so ranking adds no pass over the keys) on gfx950.
//
// One launch, two kinds of workgroup (4 waves each, d = 128, bf16 in, fp32
// accumulation):
//
//  * visual-row workgroups: causal flash attention of 256 visual query rows
//    (64 per wave) for one head.  Keys and values stream through LDS in
//    stages of 64 tokens (double buffered, one barrier per stage); each wave
//    forms S^T = K Q^T with bf16 MFMA 16x16x32 (the queries sit in registers
//    as the B operand), keeps the running row max and sum in the base-2
//    domain, and accumulates O^T = V^T P^T with P taken straight from the
//    S^T accumulators (the key order inside a 32-key step is permuted so that
//    the accumulator layout is the B operand layout; V is stored transposed
//    in LDS in the same order).  Heaviest query blocks first; the blocks of
//    one head are kept on one XCD so that its L2 serves their key reads.
//  * text-row workgroups (first in the grid): one per 512-token chunk of the
//    key sequence, all text rows (<= 64, one 16-row tile per wave), looping
//    over every head.  The per-head S^T tiles serve both the text rows'
//    attention (a partial softmax over the chunk, merged afterwards) and QER:
//    their sum over heads, kept in registers for the chunk's keys, is the
//    head-mean logit of Eq. 6 up to the factor scale / H; its max over the
//    text rows is m_j (Eq. 7) for the chunk's visual keys.
//
// attn_merge combines the text rows' chunk partials; qer_rank_from_m then
// takes the frame means and the top-k (Eqs. 7-8).
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
constexpr int kThreads = 256;    // 4 waves
constexpr int kRowsA = 64;       // visual rows per wave
constexpr int kBM = 4 * kRowsA;  // visual rows per workgroup
constexpr int kBN = 64;          // tokens per LDS stage
constexpr int kChunk = 512;      // tokens per text-row workgroup
constexpr int kStages = kChunk / kBN;
constexpr int kMaxText = 64;

struct AttnArgs {
  const uint16_t* Q;  // [L][H_q][128]
  const uint16_t* K;  // [L][H_kv][128]
  const uint16_t* V;
  uint16_t* O;        // [L][H_q][128]
  int32_t L, H_q, H_kv, vb, ve, n_text, ntp;  // ntp: text rows rounded up to 16
  int32_t n_chunks, nb_pad, qb;               // text workgroups (padded to 8), query blocks per head
  float c2;          // scale * log2(e)
  float qer_scale;   // scale / H_q
  float* m;          // [ve - vb]
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
// K: [64 tokens][16 chunks of 16 B], chunk c of token t at (c ^ (t & 15)).
// V^T: [128 d][64 tokens] (128 B rows, 8 chunks of 16 B).  Inside each
// 32-token step, token k sits at vpos(k) so that the 8 tokens lane group g of
// an S^T accumulator holds (4g..4g+3 and 16+4g..16+4g+3) are contiguous;
// chunk q of row d is stored at (q ^ vswz(d)).
constexpr int kKWords = kBN * kD / 8;          // uint4 per K stage
constexpr int kVWords = kD * kBN / 2;          // uint32 per V^T stage
constexpr int kStageU4 = kKWords + kVWords / 4;  // 16 KiB + 16 KiB

__device__ __forceinline__ int vpos(int k) {
  const int kk = k & 31;
  return (k & 32) + 8 * ((kk & 15) >> 2) + 4 * (kk >> 4) + (kk & 3);
}
__device__ __forceinline__ int vswz(int d) { return (d ^ (d >> 3)) & 7; }

struct StageRegs {
  uint4 k[4];
  uint4 v[4];
};

// Global loads of tokens k0..k0+63 of head g (rows clamped to the sequence).
// Every load instruction covers 4 tokens x 256 contiguous bytes.
__device__ __forceinline__ void stage_load(StageRegs& r, const AttnArgs& a, int g, int k0) {
  const int t = threadIdx.x, c = t & 15, kr = t >> 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int tok = min(k0 + kr + 16 * i, a.L - 1);
    r.k[i] = *reinterpret_cast<const uint4*>(a.K + ((int64_t)tok * a.H_kv + g) * kD + 8 * c);
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int tok = min(k0 + 2 * kr + p + 32 * i, a.L - 1);
      r.v[2 * i + p] = *reinterpret_cast<const uint4*>(a.V + ((int64_t)tok * a.H_kv + g) * kD + 8 * c);
    }
}

__device__ __forceinline__ void stage_store(const StageRegs& r, uint4* st) {
  const int t = threadIdx.x, c = t & 15, kr = t >> 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int tok = kr + 16 * i;
    st[tok * 16 + (c ^ (tok & 15))] = r.k[i];
  }
  uint32_t* vt = reinterpret_cast<uint32_t*>(st + kKWords);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int tok = 2 * kr + 32 * i;  // even: tok and tok + 1 are neighbours in V^T
    const int p = vpos(tok);
    const uint32_t w0[4] = {r.v[2 * i].x, r.v[2 * i].y, r.v[2 * i].z, r.v[2 * i].w};
    const uint32_t w1[4] = {r.v[2 * i + 1].x, r.v[2 * i + 1].y, r.v[2 * i + 1].z, r.v[2 * i + 1].w};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int d = 8 * c + e;
      const uint32_t lo = (w0[e >> 1] >> (16 * (e & 1))) & 0xffffu;
      const uint32_t hi = (w1[e >> 1] >> (16 * (e & 1))) & 0xffffu;
      vt[d * 32 + (((p >> 3) ^ vswz(d)) << 2) + ((p & 7) >> 1)] = lo | (hi << 16);
    }
  }
}

// A operand of S^T for key tile kt (16 tokens) and contraction step s (32 d)
__device__ __forceinline__ uint4 k_frag(const uint4* st, int kt, int s) {
  const int l = threadIdx.x & 63, tok = 16 * kt + (l & 15);
  return st[tok * 16 + ((4 * s + (l >> 4)) ^ (tok & 15))];
}

// A operand of O^T for d tile dt (16 d) and token step sub (32 tokens)
__device__ __forceinline__ uint4 v_frag(const uint4* st, int dt, int sub) {
  const int l = threadIdx.x & 63, d = 16 * dt + (l & 15);
  return st[kKWords + d * 8 + ((4 * sub + (l >> 4)) ^ vswz(d))];
}

// LDS-only barrier: the stage buffers are the only shared state.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

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
__device__ __forceinline__ void pv_stage(const uint4* st, f32x4 (&o)[8][NT], const uint4 (&p)[2][NT]) {
#pragma unroll
  for (int sub = 0; sub < 2; ++sub)
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      const uint4 vf = v_frag(st, dt, sub);
#pragma unroll
      for (int rt = 0; rt < NT; ++rt) mfma(o[dt][rt], vf, p[sub][rt]);
    }
}

template <int NT>
__device__ __forceinline__ void qk_stage(const uint4* st, f32x4 (&s)[4][NT], const uint4 (&q)[4][NT]) {
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
    for (int rt = 0; rt < NT; ++rt) s[kt][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const uint4 kf = k_frag(st, kt, ks);
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
__device__ void visual_block(const AttnArgs& a, int b, uint4* lds) {
  const int total = a.qb * a.H_q, t8 = total / 8;
  const int w = b < 8 * t8 ? (b % 8) * t8 + b / 8 : b;  // the blocks of one XCD: consecutive work
  const int h = w / a.qb, qb = a.qb - 1 - w % a.qb;        // heaviest first within a head
  const int g = h / (a.H_q / a.H_kv);
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int r0 = a.vb + kBM * qb, rw = r0 + kRowsA * wave;
  const int last = min(r0 + kBM, a.ve) - 1;  // last query row of the block
  const int nst = last / kBN + 1;
  const bool active = rw < a.ve;              // wave has rows

  uint4 q[4][4];
  int row[4];
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) {
    row[rt] = rw + 16 * rt + (l & 15);
    const int pos = min(row[rt], a.L - 1);
#pragma unroll
    for (int s = 0; s < 4; ++s) q[s][rt] = q_frag(a, pos, h, s);
  }
  f32x4 o[8][4];
  float m[4], lsum[4];
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) {
    m[rt] = -INFINITY;
    lsum[rt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[dt][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  StageRegs r;
  stage_load(r, a, g, 0);
  stage_store(r, lds);
  lds_barrier();
  for (int st = 0; st < nst; ++st) {
    const int k0 = st * kBN;
    if (st + 1 < nst) stage_load(r, a, g, k0 + kBN);
    const uint4* cur = lds + (st & 1) * kStageU4;
    if (active && k0 <= rw + kRowsA - 1) {  // some token of the stage is visible to the wave
      f32x4 s[4][4];
      uint4 p[2][4];
      qk_stage<4>(cur, s, q);
      softmax_stage<4>(s, m, lsum, o, p, row, k0, k0 + kBN - 1 > rw, a.c2);
      pv_stage<4>(cur, o, p);
    }
    if (st + 1 < nst) stage_store(r, lds + ((st + 1) & 1) * kStageU4);
    lds_barrier();
  }
  if (!active) return;
#pragma unroll
  for (int rt = 0; rt < 4; ++rt) {
    const float inv = 1.f / wave_sum4(lsum[rt]);
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
__device__ void text_block(const AttnArgs& a, int c, uint4* lds, float* red) {
  const int wave = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int c0 = c * kChunk;
  const int nst = min(kStages, (a.L - c0 + kBN - 1) / kBN);
  const int tr = 16 * wave + (l & 15);  // text row of this lane
  const bool valid = tr < a.n_text;
  const int pos = tr < a.vb ? tr : a.ve + (tr - a.vb);
  const bool active = 16 * wave < a.n_text;
  int row[1] = {valid ? pos : -1};      // an invalid row sees no token

  f32x4 acc[kStages][4];                // sum over heads of S^T, the chunk's tokens
#pragma unroll
  for (int i = 0; i < kStages; ++i)
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) acc[i][kt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int per = a.H_q / a.H_kv;
  StageRegs r;
  stage_load(r, a, 0, c0);
  stage_store(r, lds);
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
        if (more) {
          const int nh = st + 1 < nst ? h : h + 1;
          stage_load(r, a, nh / per, st + 1 < nst ? k0 + kBN : c0);
        }
        const uint4* cur = lds + buf * kStageU4;
        if (active) {
          f32x4 s[4][1];
          uint4 p[2][1];
          qk_stage<1>(cur, s, q);
#pragma unroll
          for (int kt = 0; kt < 4; ++kt) acc[st][kt] += s[kt][0];
          softmax_stage<1>(s, m, lsum, o, p, row, k0, true, a.c2);
          pv_stage<1>(cur, o, p);
        }
        if (more) stage_store(r, lds + (buf ^ 1) * kStageU4);
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

  // m_j: max over the text rows of the head sum, the chunk's visual tokens
  for (int i = threadIdx.x; i < 4 * kChunk; i += kThreads) red[i] = -INFINITY;
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
  for (int i = threadIdx.x; i < kChunk; i += kThreads) {
    const int tok = c0 + i;
    if (tok >= a.vb && tok < a.ve) {
      const float v = fmaxf(fmaxf(red[i], red[kChunk + i]), fmaxf(red[2 * kChunk + i], red[3 * kChunk + i]));
      a.m[tok - a.vb] = v * a.qer_scale;
    }
  }
}

__global__ __launch_bounds__(kThreads, 1) void attn_qer_kernel(AttnArgs a) {
  extern __shared__ uint4 lds[];
  const int b = blockIdx.x;
  if (b < a.nb_pad) {
    if (b < a.n_chunks) text_block(a, b, lds, reinterpret_cast<float*>(lds + 2 * kStageU4));
    return;
  }
  visual_block(a, b - a.nb_pad, lds);
}

// Text rows: O = sum_c 2^(m_c - M) O_c / sum_c 2^(m_c - M) l_c over the chunks.
__global__ __launch_bounds__(kD) void attn_merge_kernel(AttnArgs a) {
  const int tr = blockIdx.x, h = blockIdx.y, d = threadIdx.x;
  const int pos = tr < a.vb ? tr : a.ve + (tr - a.vb);
  float M = -INFINITY;
  for (int c = 0; c < a.n_chunks; ++c) M = fmaxf(M, a.part_ml[((int64_t)c * a.H_q + h) * a.ntp + tr].x);
  float lsum = 0.f, acc = 0.f;
  for (int c = 0; c < a.n_chunks; ++c) {
    const int64_t pr = ((int64_t)c * a.H_q + h) * a.ntp + tr;
    const float2 ml = a.part_ml[pr];
    if (ml.x == -INFINITY) continue;
    const float wgt = exp2f(ml.x - M);
    lsum += wgt * ml.y;
    acc += wgt * a.part_o[pr * kD + d];
  }
  const __bf16 v = (__bf16)(acc / lsum);
  a.O[((int64_t)pos * a.H_q + h) * kD + d] = __builtin_bit_cast(uint16_t, v);
}

struct AttnPlan {
  int32_t n_vis, n_text, ntp, n_chunks, nb_pad, qb;
};

AttnPlan plan_attn(const cofie_attn_desc& h) {
  AttnPlan p;
  p.n_vis = h.vis_end - h.vis_begin;
  p.n_text = h.L - p.n_vis;
  p.ntp = (p.n_text + 15) / 16 * 16;
  p.n_chunks = ceil_div(h.L, kChunk);
  p.nb_pad = (p.n_chunks + 7) / 8 * 8;
  p.qb = ceil_div(p.n_vis, kBM);
  return p;
}

void carve_attn(Arena& ar, const cofie_attn_desc& h, const AttnPlan& p, float** m, uint32_t** keys, float** po,
                float2** pml) {
  *m = ar.take<float>((size_t)(p.n_vis > 0 ? p.n_vis : 1));
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
  if (n_text < 1 || n_text > kMaxText)
    return set_error(COFIE_EUNSUPPORTED, "%d text tokens (1 to %d supported)", n_text, kMaxText);
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

constexpr size_t kLdsBytes = 2 * kStageU4 * sizeof(uint4) + 4 * kChunk * sizeof(float);  // 64 KiB + 8 KiB

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
  float *m, *po;
  uint32_t* keys;
  float2* pml;
  carve_attn(ar, *desc, plan_attn(*desc), &m, &keys, &po, &pml);
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
  float *m, *po;
  uint32_t* keys;
  float2* pml;
  carve_attn(plan, h, p, &m, &keys, &po, &pml);
  Scratch scratch;
  rc = scratch.acquire(h.workspace, h.workspace_bytes, plan.bytes(), s);
  if (rc) return rc;
  Arena ar;
  ar.base = scratch.ptr();
  carve_attn(ar, h, p, &m, &keys, &po, &pml);

  AttnArgs a;
  a.Q = static_cast<const uint16_t*>(Q);
  a.K = static_cast<const uint16_t*>(K);
  a.V = static_cast<const uint16_t*>(V);
  a.O = static_cast<uint16_t*>(out);
  a.L = h.L;
  a.H_q = h.H_q;
  a.H_kv = h.H_kv;
  a.vb = h.vis_begin;
  a.ve = h.vis_end;
  a.n_text = p.n_text;
  a.ntp = p.ntp;
  a.n_chunks = p.n_chunks;
  a.nb_pad = p.nb_pad;
  a.qb = p.qb;
  const double scale = h.scale > 0.f ? (double)h.scale : 1.0 / std::sqrt((double)kD);
  a.c2 = (float)(scale * 1.4426950408889634);
  a.qer_scale = (float)(scale / (double)h.H_q);
  a.m = m;
  a.part_o = po;
  a.part_ml = pml;
  rc = allow_lds(attn_qer_kernel, kLdsBytes);
  if (rc) return rc;
  const int64_t blocks = (int64_t)p.nb_pad + (int64_t)p.qb * h.H_q;
  rc = launch("attn_qer", attn_qer_kernel, dim3((unsigned)blocks), dim3(kThreads), kLdsBytes, s, a);
  if (rc) return rc;
  rc = launch("attn_merge", attn_merge_kernel, dim3((unsigned)p.n_text, (unsigned)h.H_q), dim3(kD), 0, s, a);
  if (rc) return rc;
  return qer_rank_from_m(m, p.n_vis, frame_offsets, h.n_frames, k_top, out_scores, keys, out_idx, s);
}

}  // extern "C"

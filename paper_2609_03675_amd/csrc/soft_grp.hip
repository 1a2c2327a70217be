// SOFTMAX-mode QER for grouped query heads on gfx950 (Sec. 3.3: Eq. 6's
// attention of the text rows to the visual keys, here the per-head softmax
// over the visual keys, its head mean, then Eq. 7's max over the text rows).
//
// Where G = H_q / H_kv query heads share each key head, both passes are one
// exponential per score (H_q n_q of them per key), and the general score
// kernel spends most of its VALU instructions around them (the operand select
// and rotation of its key rows, reductions across lanes at every head,
// masks).  Here the keys are the A operand straight from K (a lane's row and
// 16 bytes of each 64-byte step), the query fragments sit in LDS in MFMA
// operand order (4 KiB per head and 16-row block), each wave takes pairs of
// 16-key tiles (one fragment read feeds both), and a lane holds one query
// row and four keys of each tile (the accumulator layout), so a score costs
// one fma, one exp2 and one add:
//  * pass 1 (per-head statistics) needs no sum over heads, so a workgroup
//    takes one key head, up to four 16-row blocks and a range of key tiles:
//    each key byte is read once per launch and each key fragment feeds the
//    G x blocks products of its query heads.  A lane keeps per (head, block)
//    its sum of exp2 over its own keys against a reference (0 at first); the
//    reference moves only when a pair's sum leaves (2^-64, 2^64) (the pair is
//    then summed again against its own max, or the reference if that is
//    larger), and lanes and waves are combined once, at the end (the key
//    ranges by the merge kernel);
//  * pass 2 (the head mean of the probabilities) needs every head of a row,
//    so a workgroup takes one 16-row block with all H_q heads and a range of
//    key tiles: it adds exp2(s c2 - L) over all heads (L = M log2 e + log2 Z
//    of the row; +inf for rows past the query, which then add 0), takes the
//    max over the block's 16 rows with DPP and max-accumulates it into m: the
//    values are not negative, so their bit patterns order as unsigned
//    integers (pass 1 zeroed m), and the result does not depend on the order.
// The products run one unit (head, or head and block) ahead of the
// exponentials and the fragments two ahead; the keys one pair ahead (pass 1)
// or one key head ahead (pass 2), so the matrix core works on unit u + 1
// while the VALU finishes unit u.
// Workgroup b runs on XCD b mod 8; consecutive workgroups of one XCD take one
// key range (pass 2: its row blocks, whose key reads its L2 serves).
#include <algorithm>
#include <climits>
#include <cmath>

#include "common.h"
#include "soft_grp.h"

namespace cofie {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));

constexpr int kGrpWaves = 8;
constexpr int kGrpThreads = 64 * kGrpWaves;
constexpr int kGrpPairStride = 2 * kGrpWaves;  // tiles between a wave's pairs

// Pass-2 workgroup b: its row block, key range and tiles [t_lo, t_hi).
__host__ __device__ __forceinline__ void grp_map(int b, int nb, int ranges, int tiles, int& rb, int& range, int& t_lo,
                                                 int& t_hi) {
  const int s = b >> 3;
  rb = s % nb;
  range = (s / nb) * 8 + (b & 7);
  t_lo = (int)((int64_t)tiles * range / ranges);
  t_hi = (int)((int64_t)tiles * (range + 1) / ranges);
}
// Pass-1 workgroup b: its key head, row-block set, key range and tiles.
__host__ __device__ __forceinline__ void grp_map1(int b, int hkv, int nbs, int ranges, int tiles, int& g, int& rs,
                                                  int& range, int& t_lo, int& t_hi) {
  const int s = b >> 3;
  g = s % hkv;
  rs = (s / hkv) % nbs;
  range = (s / (hkv * nbs)) * 8 + (b & 7);
  t_lo = (int)((int64_t)tiles * range / ranges);
  t_hi = (int)((int64_t)tiles * (range + 1) / ranges);
}
// Key fragment of lane l: tile t, key head g, contraction step ks (16-byte
// index into K; rows past the last key repeat it).
__host__ __device__ __forceinline__ int64_t grp_key_u4(int t, int g, int ks, int l, int n_vis, int hkv) {
  const int64_t t16 = 16 * (int64_t)t + (l & 15);
  const int64_t row = t16 < n_vis ? t16 : n_vis - 1;
  return (row * hkv + g) * 16 + 4 * ks + (l >> 4);
}
// Query fragment slot (16-byte LDS index) of head h, step ks, lane l, and the
// element of Q it holds (query row 16 rb + l % 16; -1: past the rows).
__host__ __device__ __forceinline__ int grp_q_slot(int h, int ks, int l) { return (h * 4 + ks) * 64 + l; }
__host__ __device__ __forceinline__ int64_t grp_q_src(int rb, int h, int ks, int l, int n_q, int hq) {
  const int q = 16 * rb + (l & 15);
  return q < n_q ? ((int64_t)q * hq + h) * 16 + 4 * ks + (l >> 4) : -1;
}
// Partial statistics slot of row r (= h n_q + q) for key range `range`.
__host__ __device__ __forceinline__ int64_t grp_part(int64_t r, int range, int ranges) {
  return ((r >> 4) * ranges + range) * 16 + (r & 15);
}
// LDS: pass 2 first L of hq x 16 rows (hq * 4 uint4), then the fragments of
// all hq heads of one row block; pass 1 the fragments of the g query heads
// of one key head for nbw row blocks ([block][head][step][lane]), reused at
// the end for the combine buffer of kGrpWaves x nbw g x 16 pairs
__host__ __device__ constexpr int grp_frag0(int hq, int pass) { return pass == 2 ? hq * 4 : 0; }
__host__ __device__ constexpr size_t grp_lds(int hq, int g, int nbw, int pass) {
  return pass == 2 ? (size_t)hq * 4096 + (size_t)grp_frag0(hq, pass) * 16 : (size_t)nbw * g * 4096;
}

__device__ __forceinline__ float dpp_max16(float v) {  // max over the 16 lanes of a DPP row
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xF, 0xF, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x124, 0xF, 0xF, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x122, 0xF, 0xF, false)));
  return fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x121, 0xF, 0xF, false)));
}
// (m1, z1) and (m2, z2), sums of exp2(x - m): both against max(m1, m2), or
// the one reference with a sum (an empty side's reference is no max)
__device__ __forceinline__ void grp_combine(float& m1, float& z1, float m2, float z2) {
  const float m = z1 > 0.f ? (z2 > 0.f ? fmaxf(m1, m2) : m1) : m2;
  z1 = (z1 > 0.f ? z1 * __builtin_amdgcn_exp2f(m1 - m) : 0.f) + (z2 > 0.f ? z2 * __builtin_amdgcn_exp2f(m2 - m) : 0.f);
  m1 = m;
}

template <int HKV, int G, int PASS, int NBW>
__global__ __launch_bounds__(kGrpThreads) void qer_soft_grp_kernel(SoftGrpArgs a) {
  constexpr int HQ = HKV * G;
  static_assert(HQ % 2 == 0, "query heads alternate between two register sets");
  extern __shared__ uint4 lds_u4[];
  uint4* const qs = lds_u4 + grp_frag0(HQ, PASS);
  const int tid = threadIdx.x, l = tid & 63, wave = tid >> 6;
  const float c2 = a.c2;
  const uint4* qlane = qs + l;
  auto load_k = [&](uint4 (&f)[2][4], int t0, int g) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) f[j][ks] = a.K[grp_key_u4(t0 + j, g, ks, l, a.n_vis, HKV)];
  };
  // (fragments from a base per G heads, a runtime multiple of the head count:
  // each read is then that base plus an immediate, where up to 128 KiB of
  // constant offsets from one base would take a register per address)
  auto q_read = [&](const uint4* qg, int hl, uint4 (&f)[4]) __attribute__((always_inline)) {
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) f[ks] = qg[grp_q_slot(hl, ks, 0)];
  };
  auto products = [&](f32x4 (&s)[2], const uint4 (&k)[2][4], const uint4 (&q)[4]) __attribute__((always_inline)) {
    s[0] = s[1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        s[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, k[j][ks]),
                                                       __builtin_bit_cast(bf16x8, q[ks]), s[j], 0, 0, 0);
  };

  if constexpr (PASS == 1) {
    // one key head g, row blocks NBW rs + [0, NBW), keys [16 t_lo, 16 t_hi);
    // unit u = rbw G + hl (block rbw, query head g G + hl)
    constexpr int U = NBW * G;
    int g, rs, range, t_lo, t_hi;
    grp_map1((int)blockIdx.x, HKV, a.nbs, a.ranges1, a.tiles, g, rs, range, t_lo, t_hi);
    for (int64_t i = (int64_t)blockIdx.x * kGrpThreads + tid; i < a.n_vis; i += (int64_t)gridDim.x * kGrpThreads)
      a.m[i] = 0.f;
    if (blockIdx.x == 0 && a.clear)
      for (int i = tid; i < a.nclear; i += kGrpThreads) a.clear[i] = 0;
    {
      // the fragments, zero past the rows: every load before the first store
      constexpr int NF = (U * 256 + kGrpThreads - 1) / kGrpThreads;
      uint4 v[NF];
#pragma unroll
      for (int i = 0; i < NF; ++i) {
        const int e = tid + i * kGrpThreads, u = e >> 8;
        const int64_t src = e < U * 256 ? grp_q_src(NBW * rs + u / G, g * G + u % G, (e >> 6) & 3, e & 63, a.n_q, HQ)
                                        : -1;
        v[i] = src >= 0 ? a.Q[src] : uint4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int i = 0; i < NF; ++i) {
        const int e = tid + i * kGrpThreads;
        if (e < U * 256) qs[grp_q_slot(e >> 8, (e >> 6) & 3, e & 63)] = v[i];
      }
    }
    __syncthreads();

    const int npairs = (t_hi - t_lo + 1) >> 1;
    auto q_at = [&](int u, uint4 (&f)[4]) __attribute__((always_inline)) {
      q_read(qlane + (u / G) * a.q_gstride, u % G, f);
    };
    float mh[U], zh[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      mh[u] = 0.f;  // a reference, not yet a max: most scores' exp2 against 0 is in range
      zh[u] = 0.f;
    }
    uint4 kb[2][2][4];  // this pair's keys, the next pair's
    uint4 qf[2][4];
    f32x4 sc[2][2];
    int p = wave;
    load_k(kb[0], t_lo + 2 * p, g);
    q_at(0, qf[0]);
    q_at(1 % U, qf[1]);
    for (; p < npairs; p += 2 * kGrpWaves) {
#pragma unroll
      for (int v = 0; v < 2; ++v) {
        const int pv = p + v * kGrpWaves;
        load_k(kb[v ^ 1], t_lo + 2 * (pv + kGrpWaves), g);
        if (pv < npairs) {
          // (with U odd the fragments of unit u alternate sets from pair to pair)
          const int flip = (U & 1) ? v : 0;
          const int t0 = t_lo + 2 * pv;
          const bool has1 = t0 + 1 < t_hi;
          const bool full = has1 && 16 * (t0 + 2) <= a.n_vis;
          // this lane's keys of the pair that exist: bit 4 j + e (tile j, key 4 (l / 16) + e)
          uint32_t valid = 0xFFu;
          if (!full)
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
              for (int e = 0; e < 4; ++e)
                if ((j == 1 && !has1) || 16 * (t0 + j) + 4 * (l >> 4) + e >= a.n_vis) valid &= ~(1u << (4 * j + e));
          products(sc[0], kb[v], qf[flip]);
          q_at(2 % U, qf[flip]);
#pragma unroll
          for (int u = 0; u < U; ++u) {
            if (u + 1 < U) {
              products(sc[(u + 1) & 1], kb[v], qf[(u + 1 + flip) & 1]);
              q_at((u + 3) % U, qf[(u + 1 + flip) & 1]);
            }
            __builtin_amdgcn_sched_barrier(0);
            f32x4 (&s)[2] = sc[u & 1];
            if (!full)
#pragma unroll
              for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                  if (!((valid >> (4 * j + e)) & 1u)) s[j][e] = -INFINITY;
            float ex[8];
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
              for (int e = 0; e < 4; ++e) ex[4 * j + e] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[j][e], c2, -mh[u]));
            const float zt = ((ex[0] + ex[1]) + (ex[2] + ex[3])) + ((ex[4] + ex[5]) + (ex[6] + ex[7]));
            if (zt < 0x1p64f && zt > 0x1p-64f) {
              zh[u] += zt;
            } else {
              // the reference is too low, or far too high for this pair (or
              // the pair has no key): sum the pair against the larger of its
              // own max and the reference (its own max while nothing is
              // summed), rescaling what came before
              float pm = -INFINITY;
#pragma unroll
              for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int e = 0; e < 4; ++e) pm = fmaxf(pm, s[j][e]);
              const float mx = zh[u] > 0.f ? fmaxf(mh[u], pm * c2) : pm * c2;
              if (pm > -INFINITY) {
                float z = 0.f;
#pragma unroll
                for (int j = 0; j < 2; ++j)
#pragma unroll
                  for (int e = 0; e < 4; ++e) z += __builtin_amdgcn_exp2f(__builtin_fmaf(s[j][e], c2, -mx));
                zh[u] = (zh[u] > 0.f ? zh[u] * __builtin_amdgcn_exp2f(mh[u] - mx) : 0.f) + z;
                mh[u] = mx;
              }
            }
            __builtin_amdgcn_sched_barrier(0);
          }
        }
      }
    }
    // lanes l, l ^ 16, l ^ 32, l ^ 48 hold the same row: combine them, then
    // the waves (in LDS, over the fragments), in a fixed order
    __syncthreads();
    float2* comb = reinterpret_cast<float2*>(qs);  // [wave][U][16]
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float m1 = mh[u], z1 = zh[u];
      grp_combine(m1, z1, __shfl_xor(m1, 16), __shfl_xor(z1, 16));
      grp_combine(m1, z1, __shfl_xor(m1, 32), __shfl_xor(z1, 32));
      if (l < 16) comb[(wave * U + u) * 16 + l] = make_float2(m1, z1);
    }
    __syncthreads();
    for (int i = tid; i < U * 16; i += kGrpThreads) {
      const int u = i >> 4, q = 16 * (NBW * rs + u / G) + (i & 15), h = g * G + u % G;
      float2 c = comb[i];
      for (int w = 1; w < kGrpWaves; ++w) {
        const float2 o = comb[w * U * 16 + i];
        grp_combine(c.x, c.y, o.x, o.y);
      }
      if (q < a.n_q)  // in the natural-log units of the merge: max * scale
        a.stats_part[grp_part((int64_t)h * a.n_q + q, range, a.ranges1)] =
            c.y > 0.f ? make_float2(c.x * 0.6931471805599453f, c.y) : make_float2(-INFINITY, 0.f);
    }
  } else {
    // one 16-row block rb with every query head, keys [16 t_lo, 16 t_hi)
    int rb, range, t_lo, t_hi;
    grp_map((int)blockIdx.x, a.nb, a.ranges, a.tiles, rb, range, t_lo, t_hi);
    {
      constexpr int NF = (HQ * 256 + kGrpThreads - 1) / kGrpThreads;
      uint4 v[NF];
#pragma unroll
      for (int i = 0; i < NF; ++i) {
        const int e = tid + i * kGrpThreads;
        const int64_t src = e < HQ * 256 ? grp_q_src(rb, e >> 8, (e >> 6) & 3, e & 63, a.n_q, HQ) : -1;
        v[i] = src >= 0 ? a.Q[src] : uint4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int i = 0; i < NF; ++i) {
        const int e = tid + i * kGrpThreads;
        if (e < HQ * 256) qs[grp_q_slot(e >> 8, (e >> 6) & 3, e & 63)] = v[i];
      }
    }
    float* ls = reinterpret_cast<float*>(lds_u4);
    for (int i = tid; i < HQ * 16; i += kGrpThreads) {
      const int h = i >> 4, q = 16 * rb + (i & 15);
      float L = INFINITY;
      if (q < a.n_q) {
        const float2 st = a.stats[(int64_t)h * a.n_q + q];
        L = st.x * 1.4426950408889634f + __log2f(st.y);
      }
      ls[i] = L;
    }
    __syncthreads();

    const int npairs = (t_hi - t_lo + 1) >> 1;
    const float* lrow = ls + (l & 15);  // L of this lane's row, head h at lrow[16 h]
    auto q_at = [&](int h, uint4 (&f)[4]) __attribute__((always_inline)) {
      q_read(qlane + (h / G) * a.q_gstride, h % G, f);
    };
    // wave w: pairs w + 8 k, every query head; the keys one key head ahead
    // (the next pair's first during the last), in two register sets
    uint4 kf[2][2][4];
    uint4 qf[2][4];
    float lq[2];
    f32x4 sc[2][2];
    int p = wave;
    load_k(kf[0], t_lo + 2 * p, 0);
    q_at(0, qf[0]);
    q_at(1, qf[1]);
    for (; p < npairs; p += kGrpWaves) {
      const int t0 = t_lo + 2 * p;
      const bool has1 = t0 + 1 < t_hi;
      f32x4 prob[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
      load_k(kf[1], t0, 1);
      products(sc[0], kf[0], qf[0]);
      q_at(2 % HQ, qf[0]);
      lq[0] = lrow[0];
#pragma unroll
      for (int h = 0; h < HQ; ++h) {
        if (h + 1 < HQ) {
          const int g1 = (h + 1) / G;
          // the key head after g1 (the next pair's first after the last) into
          // the set of g1 - 1, whose last products were issued before this
          if ((h + 1) % G == 0) {
            if (g1 + 1 < HKV) load_k(kf[(g1 + 1) & 1], t0, g1 + 1);
            else load_k(kf[0], t0 + kGrpPairStride, 0);
          }
          products(sc[(h + 1) & 1], kf[g1 & 1], qf[(h + 1) & 1]);
          q_at((h + 3) % HQ, qf[(h + 1) & 1]);
          lq[(h + 1) & 1] = lrow[16 * (h + 1)];
        }
        __builtin_amdgcn_sched_barrier(0);
        f32x4 (&s)[2] = sc[h & 1];
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) prob[j][e] += __builtin_amdgcn_exp2f(__builtin_fmaf(s[j][e], c2, -lq[h & 1]));
        // the sums exist here (else the compiler defers every head's
        // exponentials to the end of the pair, keeping all their products live)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) asm volatile("" : "+v"(prob[j][e]));
        __builtin_amdgcn_sched_barrier(0);
      }
      // max over the block's 16 rows, then into m (keys that exist only)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float v = dpp_max16(prob[j][e]);
          const int tok = 16 * (t0 + j) + 4 * (l >> 4) + e;
          if ((l & 15) == 0 && (j == 0 || has1) && tok < a.n_vis)
            atomicMax(reinterpret_cast<unsigned int*>(a.m + tok), __float_as_uint(v * a.inv_h));
        }
    }
  }
}

// Address model of qer_soft_grp_kernel<HKV, G, PASS, NBW> (grid nwg, `lds`
// bytes of LDS): the zeroing, every workgroup's query-fragment loads and LDS
// slots, the statistics it reads or writes, the keys of every pair it loads
// (the extreme key heads, steps and lanes of each tile: the index is affine
// in each, and rows past the last key repeat it) and its stores into m.
template <int HKV, int G, int PASS, int NBW>
void model_grp(const SoftGrpArgs& a, int nwg, size_t lds) {
  constexpr int HQ = HKV * G;
  dry_range((int64_t)lds, 0, 160 * 1024 + 1, "soft grp: LDS beyond a CU's 160 KiB");
  dry_range((int64_t)a.nb, (a.n_q + 15) / 16, (a.n_q + 15) / 16 + 1, "soft grp: row blocks");
  auto keys = [&](int t, int g0, int g1) {
    for (int g : {g0, g1})
      for (int ks : {0, 3})
        for (int l : {0, 63}) dry_access(a.K, grp_key_u4(t, g, ks, l, a.n_vis, HKV) * 16, 16, "soft grp: keys");
  };
  auto frag = [&](int rb, int h, int slot_h, int64_t f0) {  // query head h of row block rb at slot head slot_h
    const int last = std::min(16 * rb + 15, a.n_q - 1) - 16 * rb;  // the block's last row (lane % 16), < 0: none
    for (int ks = 0; ks < 4; ++ks)
      for (int l : {0, 63, 48 + std::max(last, 0)}) {
        const int64_t src = grp_q_src(rb, h, ks, l, a.n_q, HQ);
        if (src >= 0) dry_access(a.Q, src * 16, 16, "soft grp: query fragment");
        dry_lds(f0 + (int64_t)grp_q_slot(slot_h, ks, l) * 16, 16, (int64_t)lds, "soft grp: query fragment slot");
      }
  };
  if (PASS == 1) {
    constexpr int U = NBW * G;
    dry_range(a.ranges1 % 8, 0, 1, "soft grp: key ranges not whole XCD groups");
    dry_range((int64_t)a.nbw, NBW, NBW + 1, "soft grp: row blocks per workgroup");
    dry_range((int64_t)a.nbs, (a.nb + NBW - 1) / NBW, (a.nb + NBW - 1) / NBW + 1, "soft grp: row-block sets");
    dry_range((int64_t)nwg, (int64_t)HKV * a.nbs * a.ranges1, (int64_t)HKV * a.nbs * a.ranges1 + 1, "soft grp: grid");
    dry_range((int64_t)a.q_gstride, (int64_t)G * 256, (int64_t)G * 256 + 1, "soft grp: fragment stride");
    dry_access(a.m, 0, 4 * (int64_t)a.n_vis, "soft grp: zeroing m");
    if (a.clear && a.nclear > 0) dry_access(a.clear, 0, 4 * (int64_t)a.nclear, "soft grp: arrival trees");
    dry_lds(0, (int64_t)kGrpWaves * U * 16 * 8, (int64_t)lds, "soft grp: combine buffer");
    for (int b = 0; b < nwg; ++b) {
      int g, rs, range, t_lo, t_hi;
      grp_map1(b, HKV, a.nbs, a.ranges1, a.tiles, g, rs, range, t_lo, t_hi);
      dry_range(g, 0, HKV, "soft grp: key head");
      dry_range(rs, 0, a.nbs, "soft grp: row-block set");
      dry_range(range, 0, a.ranges1, "soft grp: key range");
      dry_range(t_hi, t_lo, (int64_t)a.tiles + 1, "soft grp: tiles");
      for (int u = 0; u < U; ++u) {
        // unit u: its fragments at slot head u (block u / G at u / G * q_gstride uint4)
        frag(NBW * rs + u / G, g * G + u % G, u, 0);
        const int q0 = 16 * (NBW * rs + u / G), qn = std::min(16, a.n_q - q0);
        for (int q = q0; q < q0 + qn; ++q)
          dry_access(a.stats_part, grp_part((int64_t)(g * G + u % G) * a.n_q + q, range, a.ranges1) * 8, 8,
                     "soft grp: partial statistics");
      }
      const int npairs = (t_hi - t_lo + 1) >> 1;
      for (int w = 0; w < kGrpWaves; ++w) {
        // the wave's first pair (loaded ahead of the loop, whether or not it
        // exists), then for each step of two pairs the pair after each
        keys(t_lo + 2 * w, g, g);
        keys(t_lo + 2 * w + 1, g, g);
        for (int p = w; p < npairs; p += 2 * kGrpWaves)
          for (int v = 0; v < 2; ++v) {
            const int pn = p + v * kGrpWaves + kGrpWaves;
            keys(t_lo + 2 * pn, g, g);
            keys(t_lo + 2 * pn + 1, g, g);
          }
      }
    }
  } else {
    dry_range(a.ranges % 8, 0, 1, "soft grp: key ranges not whole XCD groups");
    dry_range((int64_t)nwg, (int64_t)a.nb * a.ranges, (int64_t)a.nb * a.ranges + 1, "soft grp: grid");
    dry_range((int64_t)a.q_gstride, (int64_t)G * 256, (int64_t)G * 256 + 1, "soft grp: fragment stride");
    const int64_t f0 = (int64_t)grp_frag0(HQ, PASS) * 16;  // the fragments' first byte
    dry_lds(0, (int64_t)HQ * 16 * 4, (int64_t)lds, "soft grp: L");
    for (int b = 0; b < nwg; ++b) {
      int rb, range, t_lo, t_hi;
      grp_map(b, a.nb, a.ranges, a.tiles, rb, range, t_lo, t_hi);
      dry_range(rb, 0, a.nb, "soft grp: row block");
      dry_range(range, 0, a.ranges, "soft grp: key range");
      dry_range(t_hi, t_lo, (int64_t)a.tiles + 1, "soft grp: tiles");
      for (int h = 0; h < HQ; ++h) frag(rb, h, h, f0);
      const int q0 = 16 * rb, qn = std::min(16, a.n_q - q0);
      for (int h = 0; h < HQ; ++h)
        dry_access(a.stats, ((int64_t)h * a.n_q + q0) * 8, 8 * (int64_t)qn, "soft grp: statistics");
      const int npairs = (t_hi - t_lo + 1) >> 1;
      for (int w = 0; w < kGrpWaves; ++w) {
        // the first pair loaded ahead of the loop, then each pair's successor
        keys(t_lo + 2 * w, 0, HKV - 1);
        keys(t_lo + 2 * w + 1, 0, HKV - 1);
        for (int p = w; p < npairs; p += kGrpWaves) {
          const int t0 = t_lo + 2 * p;
          keys(t0 + kGrpPairStride, 0, HKV - 1);
          keys(t0 + kGrpPairStride + 1, 0, HKV - 1);
          for (int j = 0; j < 2; ++j)
            if (j == 0 || t0 + 1 < t_hi) {
              const int tok0 = 16 * (t0 + j), cnt = std::min(16, a.n_vis - tok0);
              if (cnt > 0) dry_access(a.m, 4 * (int64_t)tok0, 4 * (int64_t)cnt, "soft grp: m");
            }
        }
      }
    }
  }
}

template <int HKV, int G, int PASS, int NBW>
int launch_grp_k(const SoftGrpArgs& a, int nwg, hipStream_t s) {
  const size_t lds = grp_lds(HKV * G, G, NBW, PASS);
  auto k = qer_soft_grp_kernel<HKV, G, PASS, NBW>;
  if (dry_run()) model_grp<HKV, G, PASS, NBW>(a, nwg, lds);
  const int rc = allow_lds(k, lds);
  if (rc) return rc;
  return launch(PASS == 1 ? "qer_soft_stats_grp" : "qer_soft_score_grp", k, dim3((unsigned)nwg), dim3(kGrpThreads),
                lds, s, a);
}

template <int HKV, int G>
int launch_grp_t(const SoftGrpArgs& a, int pass, hipStream_t s) {
  if (pass == 2) return launch_grp_k<HKV, G, 2, 1>(a, a.nb * a.ranges, s);
  const int nwg = HKV * a.nbs * a.ranges1;
  switch (a.nbw) {
    case 1: return launch_grp_k<HKV, G, 1, 1>(a, nwg, s);
    case 2: return launch_grp_k<HKV, G, 1, 2>(a, nwg, s);
    case 3: return launch_grp_k<HKV, G, 1, 3>(a, nwg, s);
    case 4: return launch_grp_k<HKV, G, 1, 4>(a, nwg, s);
    default: return set_error(COFIE_EINVAL, "grouped SOFTMAX: %d row blocks per workgroup", a.nbw);
  }
}

}  // namespace

// (key heads, query heads per key head) with an instance: the high-res
// workload's 4 x 7 and the common grouped-query ratios
bool grp_has_instance(int hkv, int g) {
  return (hkv == 4 && (g == 7 || g == 8 || g == 2)) || (hkv == 2 && (g == 4 || g == 8));
}

int grp_nbw(int g, int nb) { return std::max(1, std::min({nb, 4, 36 / g})); }

int launch_grp(const SoftGrpArgs& a, int hkv, int g, int pass, hipStream_t s) {
  if (a.nb < 1 || a.ranges < 8 || a.ranges % 8 != 0 || a.ranges1 < 8 || a.ranges1 % 8 != 0 || a.n_vis < 1 ||
      a.n_q < 1 || a.q_gstride != g * 256 || a.nbw != grp_nbw(g, a.nb) || a.nbs != (a.nb + a.nbw - 1) / a.nbw)
    return set_error(COFIE_EINVAL, "grouped SOFTMAX plan: %d row blocks, %d key ranges", a.nb, a.ranges);
  if (hkv == 4 && g == 7) return launch_grp_t<4, 7>(a, pass, s);
  if (hkv == 4 && g == 8) return launch_grp_t<4, 8>(a, pass, s);
  if (hkv == 4 && g == 2) return launch_grp_t<4, 2>(a, pass, s);
  if (hkv == 2 && g == 4) return launch_grp_t<2, 4>(a, pass, s);
  if (hkv == 2 && g == 8) return launch_grp_t<2, 8>(a, pass, s);
  return set_error(COFIE_EUNSUPPORTED, "grouped SOFTMAX: no instance for %d key heads x %d query heads", hkv, g);
}

}  // namespace cofie

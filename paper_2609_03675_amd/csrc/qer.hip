// QER -- Query-Specific Evidence Refinement (Sec. 3.3) on gfx950.
//
// LOGIT mode (Eq. 6) folds the head mean into the contraction:
//   a_ij = (scale / H_q) * <q~_i, k~_j>, q~/k~ = all heads side by side,
// so the text-by-vision scores are one GEMM S^T = K Q^T with contraction
// length Lc = H_kv * d.  With grouped-query attention the query heads of a
// group are summed first, in fp32 and in head order (q^_g = sum_{h in g} q_h,
// rounded once per addition: exact only while the heads' exponents stay
// within fp32's 24 bits of each other), and that rounded fp32 q^ is carried
// as three bf16 terms hi + mid + lo whose sum is exactly it, so the bf16 MFMA
// multiplies exact representations of the fp32 sum.
//
// qer_score: one 8-wave workgroup per CU; each wave owns MB x 16 visual tokens
//   and all (<= 64, or 128 in eight blocks) query rows of one chunk, over the
//   whole contraction, or over one of NS slices of it where tiles are too few
//   to give every wave of the chip one (the slices' sums meet in LDS).  K rows
//   stream from HBM exactly once, in 128-byte row segments that a lane select
//   and a DPP swap turn into MFMA operands; the query fragments are staged in
//   LDS phase by phase.  The epilogue takes the max over query rows
//   (registers, then 16-lane shuffles) and writes m_j = scale * max_i S_ij:
//   the text-by-vision matrix is never stored.
// qer_frame_mean: one wave per frame, fp64 mean of m over V_f (Eq. 7); the
//   last workgroup to finish (an arrival counter the score kernel clears)
//   ranks the frames by (score desc, frame asc) on order-preserving 32-bit
//   keys (counting ranks, or a 4-pass radix select) and writes the top k in
//   chronological order (Eq. 8).
// qer_topk: the same selection as a kernel of its own (the SOFTMAX fallback
//   kernels, the fused attention path, cofie_topk).
// SOFTMAX mode: per-(head, query) row statistics over all visual keys, merged
//   across waves and workgroups, then a second pass forming the head mean of
//   the normalised probabilities and its max over query rows.  Where every
//   head is whole 128-byte segments of a key row, both passes are qer_score
//   with a per-head epilogue (the contraction runs over the query heads in
//   order, grouped heads reading their key head through a segment map);
//   other head sizes take per-head kernels of their own.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstring>
#include <mutex>
#include <vector>

#include "common.h"
#include "soft_grp.h"

namespace cofie {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4v __attribute__((ext_vector_type(4)));
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

// ---- LDS-staged query fragments -------------------------------------------------------
// One workgroup of 8 waves per CU.  Each wave keeps the whole contraction of
// its MB tiles of 16 tokens in registers; vector memory carries only the key
// stream and, once per phase, the query fragments of the phase.
//
// Key loads.  An MFMA operand holds 16 rows x 64 bytes per register, and a
// load instruction in that shape (16 rows, 64 bytes each) streams at roughly
// half the per-CU rate of one that takes 128 or 256 contiguous bytes from each
// of 8 or 4 rows.  The contraction order is free as long as keys and queries
// agree, so each row is read in segments of SEGC = 64/R 16-byte chunks with
// R rows per load: per segment and tile, load q (q < VPS = 16/R) covers rows
// R q .. R q + R-1, lane s taking row R q + s%R and chunk
// VPS*(s/16) + ((s%16)/R - q) mod VPS.  Lane l then finds chunk VPS*g + k
// (g = l/16) of its own row l%16 in load ((l%16)/R - k) mod VPS ... of lane
// l + R k within its 16-lane row: a per-lane register select and one DPP row
// rotation make operand k.  Segment m so yields VPS operands, "virtual steps"
// VPS m + k, whose lane group g covers 16-byte chunk SEGC m + VPS g + k.  A
// contraction tail shorter than a segment is read in plain MFMA shape.
//
// Query fragments.  The contraction is cut into phases of S virtual steps; a
// phase's query fragments sit in LDS in MFMA operand order ([slice][step]
// [term][16-query block][lane], 16 bytes per lane, read by every wave with
// conflict-free 16-byte LDS loads), double buffered: the fragments of phase
// i+1 are fetched into registers at the start of phase i and written to LDS
// one batch later.
// One key sequence of a launch over several (cofie_qer_rank_streams) and the
// stacked query rows that read it: its tiles sit at [tile0, tile0 + ntiles)
// of the launch's tile space, side by side with the other sequences'.
struct QerStreamDesc {
  int64_t key0;    // first key row
  int32_t n_keys;  // key rows
  int32_t tile0;   // first tile
  int32_t ntiles;  // ceil(n_keys / 16)
  int32_t q0;      // first stacked query row (of each query term)
  int32_t n_rows;  // query rows (whole queries, at most 16 NB)
  int32_t pad;
};

struct ScoreLdsArgs {
  const uint8_t* K;   // [n_vis][Lc] elements
  const uint8_t* Qp;  // [P][nq_total][Lc] elements
  int32_t n_vis;
  int32_t n_q;        // query rows in this chunk (<= 64; <= 128 with eight blocks)
  int32_t q0;
  int32_t nq_total;
  int32_t Lc;
  int32_t nseg;       // whole segments per row
  int32_t ksteps;     // virtual steps: VPS nseg + tail steps
  int32_t S;          // virtual steps per phase (a multiple of the batch length)
  int32_t nphase;
  int32_t tiles;      // 16-token tiles
  int32_t nwg;        // workgroups
  float scale;
  float* m;
  int32_t accumulate;
  int32_t group_rows;  // > 0: query rows form queries of this many rows (a multiple of
                       // 16), each with its own row of m: m[g * m_stride + j]
  int64_t m_stride;
  int32_t* clear;      // workgroup 0 zeroes clear[0, nclear) (the frame-mean kernel's
  int32_t nclear;      // arrival counters), may be null
  int32_t lgS;         // log2 S
  int32_t split_u4;    // contraction split NS ways: 16-byte columns from one slice to the next
  int32_t k_row_u4;    // 16-byte chunks per key row (shorter than a query row in SOFTMAX GQA)
  // SOFTMAX passes (the contraction runs over the query heads in order, one
  // head every sph segments; query head h reads key head h / G)
  int32_t sph;         // segments per head
  int32_t H;           // query heads
  int32_t G;           // query heads per key head
  float soft_scale;    // scale inside the exponent
  // pass 1: (max, sum of exp) of row r = h * nq_total + q per wave and round,
  // part b = (workgroup * 8 + wave) * rounds + round at
  // stats_part[((r / 16) * nparts + b) * 16 + r % 16]
  float2* stats_part;
  int32_t rounds;      // rounds per workgroup
  int32_t nparts;      // nwg * 8 * rounds
  const float2* stats; // pass 2: [H][nq_total] (max, sum of exp) over all keys
  // pass 1 with several queries (group_rows > 0): query g's rows see only the
  // keys of its first soft_nf[g] frames, [0, soft_offs[soft_nf[g]]); null: all
  const int32_t* soft_offs;
  const int32_t* soft_nf;
  // several key sequences (LOGIT, one contraction slice; null: one): tiles is
  // the total over them, and a workgroup's share is taken one sequence at a
  // time, with that sequence's keys, token count and query rows
  const QerStreamDesc* streams;
  int32_t n_streams;
  int32_t xcd_order;   // shares in XCD order: consecutive shares to the workgroups of one XCD
};

constexpr int kModeLogit = 0;     // Eq. 6-7: m_j = max_i a_ij
constexpr int kModeSoftStats = 1; // SOFTMAX pass 1: per-head row statistics
constexpr int kModeSoftProb = 2;  // SOFTMAX pass 2: m_j = max_i mean_h P^h_ij
constexpr int kModeGqa = 4;       // flag: grouped query heads read their key head through a segment map
constexpr int kModeSeq = 8;       // flag (LOGIT): several key sequences, each with its own query rows

constexpr int kLdsWaves = 8;
constexpr int kLdsThreads = kLdsWaves * 64;
// uint4 per thread per phase fill (a phase buffer holds q_regs * 512 uint4):
// 32 KiB phases when the query side is narrow (fewer registers held, a shorter
// first fill: 1 fps stream 47.2 vs 48.8 us), 64 KiB otherwise (fewer phases:
// high-res 20.4 vs 23.1 us)
// With the contraction split NS ways inside the workgroup (NS > 1) a phase
// holds NS slices and takes the 64 KiB buffer.
__host__ __device__ constexpr int lds_q_regs(int PNB, int NS = 1) { return NS == 1 && PNB <= 2 ? 4 : 8; }

// virtual steps per batch: 8 key loads per batch and wave (two batches in
// flight), fewer where the query fragments and accumulators of wide query
// blocks take the registers, or where NS slices of a phase of U steps would
// not fit its buffer; at least one segment (16/R steps)
__host__ __device__ constexpr int lds_batch(int MB, int PNB, int R, int NS = 1) {
  int u = MB == 1 ? (PNB <= 4 ? 8 : 4) : (PNB <= 2 ? 4 : 2);
  while (u > 1 && NS * u * PNB * 64 > lds_q_regs(PNB, NS) * kLdsThreads) u >>= 1;
  return u > 16 / R ? u : 16 / R;
}

template <int N>
__device__ __forceinline__ uint32_t row_ror(uint32_t v) {  // lane i <- lane (i - N) mod 16 of its row
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x120 + N, 0xF, 0xF, false);
}
template <int N>
__device__ __forceinline__ uint4 row_ror4(const uint4& v) {
  if constexpr (N == 0) return v;
  else return uint4{row_ror<N>(v.x), row_ror<N>(v.y), row_ror<N>(v.z), row_ror<N>(v.w)};
}

// Reductions over lanes l and l ^ 16 (l ^ 32) in the VALU: gfx950's
// v_permlane16_swap / v_permlane32_swap hand each lane the pair (value of the
// lower lane, value of the upper lane), in that order in both lanes (checked
// on the device), so both lanes compute the same result.
__device__ __forceinline__ float max_x16(float v) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
}
__device__ __forceinline__ float max_x32(float v) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
}
__device__ __forceinline__ float sum_x16(float v) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}
__device__ __forceinline__ float sum_x32(float v) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}

// rows per key load.  8 (128-byte segments) measured faster than 4 (256-byte
// segments) in this kernel on the 1 fps stream workload (48.9 vs 51.1 us).
__host__ __device__ constexpr int lds_rows(int, int) { return 8; }

// The score kernel's batch (virtual steps per key batch): the host plan's,
// halved for SOFTMAX pass 1 with three or more query blocks and for pass 2
// (MHA heads) with eight, one tile per wave: the full batch would spill (the
// grouped-head pass 2 spills with the half batch instead).  S, the phase
// length, stays a multiple of it.
__host__ __device__ constexpr int score_batch(int MB, int NB, int P, int NS, int mode) {
  return lds_batch(MB, P * NB, lds_rows(MB, P * NB), NS) /
         (MB == 1 && (((mode & 3) == kModeSoftStats && P * NB >= 3) || (mode == kModeSoftProb && P * NB >= 8)) ? 2
                                                                                                            : 1);
}

// ---- address arithmetic of qer_score_kernel, shared with its address model ---------
// Key load q (of 16 / R per segment) of lane `lane` for the tile whose first
// token is t0: 16-byte index from the key base of its load in segment 0
// (segment m adds 64 / R m).  Rows past the last key repeat the last.
template <int R>
__host__ __device__ __forceinline__ int64_t score_key_u4(int64_t t0, int q, int lane, int64_t last, int64_t krow_u4) {
  constexpr int VPS = 16 / R;
  const int64_t t = t0 + R * q + lane % R;
  const int64_t tok = t < last ? t : last;
  return tok * krow_u4 + VPS * (lane >> 4) + ((((lane & 15) / R) - q) & (VPS - 1));
}
// Plain MFMA-shaped key load of the contraction tail (lane: row lane % 16,
// 16-byte column col + lane / 16 of that row, or two columns back where that
// column is past the row: the value is then multiplied by zero).
__host__ __device__ __forceinline__ int64_t score_tail_u4(int64_t t0, int lane, int64_t last, int64_t krow_u4, int col,
                                                          bool in) {
  const int64_t t = t0 + (lane & 15);
  return (t < last ? t : last) * krow_u4 + (lane >> 4) + col + (in ? 0 : -2);
}
// Query fragment load: element e of phase ph (16-byte units): the query row
// (of term p) and column it takes, and whether it is real (else it loads row
// q0 of term 0, column 0, and stores zero).
template <int NB, int NS, int FPS, int EPL>
__host__ __device__ __forceinline__ int64_t score_q_u4(int32_t n_q, int32_t q0, int32_t nq_total, int32_t Lc,
                                                       int32_t split_u4, int e, int ph, int lgC, int64_t row_u4,
                                                       bool& ok) {
  constexpr int LGNS = NS == 4 ? 2 : (NS == 2 ? 1 : 0);
  const int row = e >> (lgC + LGNS), f = row >> 4;
  const int p = f / NB, nb = f - p * NB;
  const int q = nb * 16 + (row & 15);
  const int sl = (e >> lgC) & (NS - 1);
  const int col = sl * split_u4 + (ph << lgC) + (e & ((1 << lgC) - 1));
  ok = f < FPS && q < n_q && col * EPL < Lc;
  const int64_t grow = ok ? (int64_t)p * nq_total + q0 + q : (int64_t)q0;
  return grow * row_u4 + (ok ? col : 0);
}
// Query fragments in LDS, one phase buffer: [slice][step][fragment][lane],
// 16 bytes per lane.  Phase column c of a query row (a 16-byte chunk) belongs
// to virtual step ls = VPS (c / SEGC) + c % VPS and lane group
// g = (c % SEGC) / VPS, the order in which the key segments are read; row r
// of fragment f sits at lane 16 g + (r ^ score_swz(ls, g)).  The swizzle
// (step mod the batch length U, a power of two <= 8, and g: 16 values)
// spreads the 64 stores of a contiguous query-row load over the banks.
template <int U>
__host__ __device__ __forceinline__ int score_swz(int ls, int g) {
  constexpr int LOGU = U >= 8 ? 3 : (U >= 4 ? 2 : 1);
  return ((ls & (U - 1)) | (g << LOGU)) & 15;
}
// slot of column c, fragment f, row r within a slice's steps
template <int U, int VPS, int SEGC, int FPS>
__host__ __device__ __forceinline__ int score_q_slot_c(int c, int f, int r) {
  const int ls = VPS * (c / SEGC) + c % VPS, g = (c % SEGC) / VPS;
  return ((ls * FPS + f) << 6) + (g << 4) + (r ^ score_swz<U>(ls, g));
}
// The slot element e of a phase's row-major query load is stored to: slice
// (e >> lgC) % NS, row (e >> lgC) / NS (fragment row / 16, row row % 16),
// column e % 2^lgC; spare elements past the fragments keep slot e (their value
// is zero and never read).
template <int U, int VPS, int SEGC, int FPS, int NS>
__host__ __device__ __forceinline__ int score_q_slot(int e, int lgC, int lgS) {
  constexpr int LGNS = NS == 4 ? 2 : (NS == 2 ? 1 : 0);
  const int row = e >> (lgC + LGNS), f = row >> 4;
  const int sl = (e >> lgC) & (NS - 1);
  if (f >= FPS) return e;
  return ((sl * FPS) << (lgS + 6)) + score_q_slot_c<U, VPS, SEGC, FPS>(e & ((1 << lgC) - 1), f, row & 15);
}

// NS > 1 splits the contraction inside the workgroup: wave w multiplies slice
// w % NS (a.split_u4 columns from the previous one) of the tiles of wave group
// w / NS, and the slices' accumulators are added in slice order through LDS
// before the maximum over the query rows, so that few tiles still occupy every
// wave of every CU.
//
// MODE selects the epilogue: kModeLogit as above; the SOFTMAX passes close
// every head (sph segments of the contraction) in registers: pass 1 writes the
// head's (max, sum of exp) over the wave's tokens for every query row, pass 2
// adds exp(s - max) / sum over the heads and ends like LOGIT with the head
// mean's maximum over the query rows.
template <typename T, int MB, int NB, int P, int NS, int MODE>
__global__ __launch_bounds__(kLdsThreads) void qer_score_kernel(ScoreLdsArgs a) {
  using M = Mma<T>;
  constexpr int BASE = MODE & 3;  // kModeLogit, kModeSoftStats or kModeSoftProb
  constexpr bool GQA = (MODE & kModeGqa) != 0;
  constexpr bool SEQ = (MODE & kModeSeq) != 0;
  constexpr int R = lds_rows(MB, P * NB);
  constexpr int VPS = 16 / R;   // virtual steps (= loads per tile) per segment
  constexpr int SEGC = 64 / R;  // 16-byte chunks per segment
  constexpr int U = score_batch(MB, NB, P, NS, MODE);
  constexpr int FPS = P * NB;   // fragments per virtual step
  constexpr int kQRegs = lds_q_regs(FPS, NS);
  constexpr int kPhaseU4 = kQRegs * kLdsThreads;
  constexpr int TW = kLdsWaves / NS;  // waves per slice (tiles per round when MB = 1)
  constexpr int LGNS = NS == 4 ? 2 : (NS == 2 ? 1 : 0);
  static_assert(U % VPS == 0, "batches hold whole segments");
  static_assert(NS == 1 || NS == 2 || NS == 4, "1, 2 or 4 slices");
  static_assert(NS == 1 || MB == 1, "split contractions take one tile per wave");
  static_assert(BASE == kModeLogit || (NS == 1 && P == 1), "SOFTMAX passes: one query term, no split");
  static_assert(!GQA || BASE != kModeLogit, "the segment map is for the SOFTMAX passes");
  static_assert(!SEQ || (BASE == kModeLogit && NS == 1), "several key sequences: LOGIT, one slice");
  // [2][kPhaseU4]: [NS][S][P][NB][64] each; with NS > 1 followed by the
  // slice accumulators [NS - 1][TW][MB][NB][4][64] floats
  extern __shared__ uint4 qs[];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int slice = wave & (NS - 1), tw = wave >> LGNS;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int qs_lane = r16 / R;  // load index holding this lane's own row
  // Query fragments in LDS: a phase of S steps per buffer in the layout of
  // score_q_slot_c (the tail steps past the whole segments use the same
  // order); readers undo the swizzle.
  int lsw[U];  // this lane's swizzled slot for steps congruent to u mod U
#pragma unroll
  for (int u = 0; u < U; ++u) lsw[u] = lane ^ score_swz<U>(u, g4);
  const int pfull = VPS * a.nseg;
  const int64_t row_u4 = (int64_t)a.Lc * sizeof(T) / 16;
  const int64_t krow_u4 = a.k_row_u4;
  const uint4* const K0 = reinterpret_cast<const uint4*>(a.K) + (NS > 1 ? slice * a.split_u4 : 0);
  const uint4* Kq = K0;
  const uint4* Qq = reinterpret_cast<const uint4*>(a.Qp);
  // This workgroup's share of the tiles.  Workgroups are dealt to the XCDs in
  // turn (workgroup b to XCD b % 8), so with xcd_order the shares are ordered
  // by XCD: the workgroups of one XCD take consecutive shares, and a key
  // sequence's query rows are read into few XCDs' L2.
  const int wg = a.xcd_order ? (int)((blockIdx.x & 7) * (a.nwg >> 3) + (blockIdx.x >> 3)) : (int)blockIdx.x;
  const int f_begin = (int)((int64_t)a.tiles * wg / a.nwg);
  const int f_end = (int)((int64_t)a.tiles * (wg + 1) / a.nwg);
  int sidx = 0;  // several sequences: the first one whose tiles reach f_begin
  if constexpr (SEQ)
    while (sidx + 1 < a.n_streams && a.streams[sidx].tile0 + a.streams[sidx].ntiles <= f_begin) ++sidx;
  if (blockIdx.x == 0 && a.clear)
    for (int i = tid; i < a.nclear; i += kLdsThreads) a.clear[i] = 0;

  // pass 1: exp(scale acc - m) = exp2(acc c2 - m log2 e), one FMA and
  // v_exp_f32 (pass 2 keeps __expf: the FMA form made the grouped-head,
  // two-tile, 48-row variant spill)
  const float c2 = a.soft_scale * 1.44269504088896341f;
  // SOFTMAX passes: past the phase buffers, pass 2's row statistics of this
  // query chunk ([H][n_q]: max, 1 / sum of exp) and, for grouped heads, the
  // key segment of every contraction segment.  The first barrier of the round
  // loop publishes them.
  float2* st_sh = reinterpret_cast<float2*>(qs + (a.nphase > 1 ? 2 : 1) * kPhaseU4);
  int32_t* seg_map = reinterpret_cast<int32_t*>(st_sh + (BASE == kModeSoftProb ? a.H * a.n_q : 0));
  // pass 1: the keys each 16-row block's query sees (padding blocks none)
  int64_t key_lim[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    key_lim[nb] = a.n_vis;
    if constexpr (BASE == kModeSoftStats) {
      if (a.soft_nf) {
        int64_t l = 0;
        if (nb * 16 < a.n_q) {
          l = a.soft_offs[a.soft_nf[(a.q0 + nb * 16) / a.group_rows]];
          l = l < 0 ? 0 : (l > a.n_vis ? a.n_vis : l);
        }
        key_lim[nb] = l;
      }
    }
  }
  if constexpr (BASE != kModeLogit) {
    if constexpr (GQA)
      for (int v = tid; v < a.nseg; v += kLdsThreads) seg_map[v] = (v / a.sph / a.G) * a.sph + v % a.sph;
    if constexpr (BASE == kModeSoftProb)
      for (int i = tid; i < a.H * a.n_q; i += kLdsThreads) {
        const int hh = i / a.n_q, q = i - hh * a.n_q;
        const float2 st = a.stats[(int64_t)hh * a.nq_total + a.q0 + q];
        // L = M log2 e + log2 Z: p = exp2(s scale log2 e - L)
        st_sh[i] = make_float2(st.x * 1.44269504088896341f + __log2f(st.y), 0.f);
      }
  }

  bool qok[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) qok[nb] = nb * 16 + r16 < a.n_q;

  // fragments of phase ph.  The phase covers the 16-byte columns
  // [4 S ph, 4 S ph + 4 S) of every query row (its S virtual steps, 4 lane
  // groups each), so element e = tid + kLdsThreads * i is taken in row-major
  // order: row e / 4S, column 4 S ph + e % 4S, and a wave's load is one
  // contiguous run of a row (1 KiB for 4S = 64) instead of 16 rows x 64 bytes
  // in operand shape.  The store puts it at its operand slot (q_slot).  Rows
  // past n_q and columns past Lc are zero.  Loads are unconditional (clamped
  // addresses); the zeroing is a select made when the registers are stored,
  // so that issuing the loads never waits for them.
  uint32_t qmask = 0;
  const int lgC = a.lgS + 2;  // log2 of the 16-byte columns per row and phase (4 S, S a power of two)
  // With NS slices, consecutive runs of a row alternate between the slices:
  // element e is slice (e >> lgC) % NS, row (e >> lgC) / NS.
  auto q_load = [&](int ph, uint4 (&qr)[kQRegs]) __attribute__((always_inline)) {
    qmask = 0;
#pragma unroll
    for (int i = 0; i < kQRegs; ++i) {
      // slots past the P NB fragments (f >= FPS, so p >= P) and masked rows
      // load row q0 of term 0, which every chunk has
      bool ok;
      const int64_t src = score_q_u4<NB, NS, FPS, M::EPL>(a.n_q, a.q0, a.nq_total, a.Lc, a.split_u4,
                                                          tid + kLdsThreads * i, ph, lgC, row_u4, ok);
      qr[i] = Qq[src];
      qmask |= ok ? 1u << i : 0u;
    }
  };
  auto q_store = [&](int ph, const uint4 (&qr)[kQRegs]) __attribute__((always_inline)) {
    uint4* dst = qs + (ph & 1) * kPhaseU4;
#pragma unroll
    for (int i = 0; i < kQRegs; ++i) {
      const bool ok = (qmask >> i) & 1u;
      dst[score_q_slot<U, VPS, SEGC, FPS, NS>(tid + kLdsThreads * i, lgC, a.lgS)] =
          uint4{ok ? qr[i].x : 0u, ok ? qr[i].y : 0u, ok ? qr[i].z : 0u, ok ? qr[i].w : 0u};
    }
  };
  auto barrier_lds = []() __attribute__((always_inline)) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
  };

  bool staged = false;  // an earlier round of this workgroup has used the phase buffers
  // the rounds over tiles [t_begin, t_end) of the current key sequence
  auto rounds = [&](const int t_begin, const int t_end) __attribute__((always_inline)) {
  for (int rb = t_begin; rb < t_end; rb += TW * MB) {
    // this wave's tiles: rb + tw + TW j.  Missing ones repeat tile rb (the
    // first tile of wave 0 in this round): their loads hit the cache and their
    // results are never stored.
    int nmb = 0;
#pragma unroll
    for (int j = 0; j < MB; ++j) nmb += (rb + tw + TW * j < t_end) ? 1 : 0;
    const uint4* kq[MB][VPS];
    const uint4* k16[MB];
#pragma unroll
    for (int j = 0; j < MB; ++j) {
      const int64_t t0 = (int64_t)(j < nmb ? rb + tw + TW * j : rb) * 16;
      const int64_t last = a.n_vis - 1;
#pragma unroll
      for (int q = 0; q < VPS; ++q) kq[j][q] = Kq + score_key_u4<R>(t0, q, lane, last, krow_u4);
      k16[j] = Kq + score_tail_u4(t0, lane, last, krow_u4, 0, true);
    }
    f32x4 acc[MB][NB];
#pragma unroll
    for (int j = 0; j < MB; ++j)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[j][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

    // SOFTMAX passes: close query head hh, whose unscaled dot products are in
    // acc, and start the next one from zero
    f32x4 prob[MB][NB];  // pass 2: sum over the heads closed so far
#pragma unroll
    for (int j = 0; j < MB; ++j)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) prob[j][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    int head = 0, head_seg = 0;
    // pass 1: bit 4 j + r of vmask[nb] set when this lane's accumulator
    // element (tile j, token 4 g4 + r) is a key that block nb's query sees
    uint32_t vmask[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) vmask[nb] = 0;
    if constexpr (BASE == kModeSoftStats) {
#pragma unroll
      for (int j = 0; j < MB; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t tok = (int64_t)(rb + tw + TW * j) * 16 + g4 * 4 + r;
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
            vmask[nb] |= (j < nmb && tok < key_lim[nb]) ? 1u << (4 * j + r) : 0u;
        }
    }
    auto head_close = [&](int hh) __attribute__((always_inline)) {
      if constexpr (BASE == kModeSoftStats) {
        // (m, sum of exp(s - m)) over this wave's valid tokens, per query row,
        // m = 0 or, where the sum against 0 is out of range, the max; a wave
        // without tokens writes (-inf, 0)
        const int64_t slot = ((int64_t)blockIdx.x * kLdsWaves + wave) * a.rounds + (rb - t_begin) / (TW * MB);
        const int64_t row0 = (int64_t)hh * a.nq_total + a.q0;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          // the sum against 0 first (no max); the row's four lane groups hold
          // the same sum, so the exact form below runs for whole rows only,
          // where that sum leaves (2^-64, 2^64) or the row has no valid token
          float z = 0.f;
#pragma unroll
          for (int j = 0; j < MB; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if ((vmask[nb] >> (4 * j + r)) & 1u) z += __builtin_amdgcn_exp2f(acc[j][nb][r] * c2);
          z = sum_x32(sum_x16(z));
          float mx = 0.f;
          if (!(z < 0x1p64f && z > 0x1p-64f)) {
            mx = -INFINITY;
#pragma unroll
            for (int j = 0; j < MB; ++j)
#pragma unroll
              for (int r = 0; r < 4; ++r)
                if ((vmask[nb] >> (4 * j + r)) & 1u) mx = fmaxf(mx, acc[j][nb][r]);
            mx = max_x32(max_x16(mx));
            const float mc = mx * c2;
            z = 0.f;
#pragma unroll
            for (int j = 0; j < MB; ++j)
#pragma unroll
              for (int r = 0; r < 4; ++r)
                if ((vmask[nb] >> (4 * j + r)) & 1u) z += __builtin_amdgcn_exp2f(fmaf(acc[j][nb][r], c2, -mc));
            z = sum_x32(sum_x16(z));
          }
          const int q = nb * 16 + r16;
          if (g4 == 0 && q < a.n_q) {
            const int64_t row = row0 + q;  // 16 lanes: one or two 128-byte runs
            a.stats_part[((row >> 4) * a.nparts + slot) * 16 + (row & 15)] = make_float2(mx * a.soft_scale, z);
          }
        }
      } else if constexpr (BASE == kModeSoftProb) {
        const float2* sth = st_sh + hh * a.n_q;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const int q = nb * 16 + r16;
          const float2 st = sth[q < a.n_q ? q : a.n_q - 1];
#pragma unroll
          for (int j = 0; j < MB; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r) prob[j][nb][r] += __builtin_amdgcn_exp2f(fmaf(acc[j][nb][r], c2, -st.x));
        }
      }
#pragma unroll
      for (int j = 0; j < MB; ++j)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[j][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    };

    // loads of the U virtual steps from ms (U/VPS segments, VPS loads each)
    auto k_load = [&](uint4 (&f)[U][MB], int ms) __attribute__((always_inline)) {
#pragma unroll
      for (int h = 0; h < U / VPS; ++h) {
        int seg = min(ms / VPS + h, a.nseg - 1);
        if constexpr (GQA) seg = seg_map[seg];
#pragma unroll
        for (int q = 0; q < VPS; ++q)
#pragma unroll
          for (int j = 0; j < MB; ++j) {
            // keys are read once: non-temporal loads (1 fps stream 46.0 -> 43.4 us)
            const u32x4v t = __builtin_nontemporal_load(reinterpret_cast<const u32x4v*>(kq[j][q] + SEGC * seg));
            f[VPS * h + q][j] = uint4{t.x, t.y, t.z, t.w};
          }
      }
    };

    uint4 fa[U][MB], fb[U][MB];
    if (a.nseg > 0) k_load(fa, 0);
    if (staged) barrier_lds();  // previous round's readers are done
    staged = true;
    uint4 qr[kQRegs];
    q_load(0, qr);
    q_store(0, qr);
    bool pending = a.nphase > 1;
    if (pending) q_load(1, qr);
    barrier_lds();

    // one batch: prefetch the next batch into `nxt`, multiply `cur`, and at a
    // phase end publish the next phase's fragments
    int ph = 0;
    // SOFTMAX with grouped heads: `nxt` holds the batch two before the one it
    // is about to receive; when both read the same key segments (consecutive
    // query heads of one key head), the keys are already in place
    auto keys_in_place = [&](int X) __attribute__((always_inline)) {
      if constexpr (!GQA) {
        return false;
      } else {
        if (X < 2 * U) return false;
        bool same = true;
#pragma unroll
        for (int h = 0; h < U / VPS; ++h)
          same = same && seg_map[min(X / VPS + h, a.nseg - 1)] == seg_map[min((X - 2 * U) / VPS + h, a.nseg - 1)];
        return same;
      }
    };
    auto batch = [&](int ms, const uint4 (&cur)[U][MB], uint4 (&nxt)[U][MB], bool guard) __attribute__((always_inline)) {
      if (!keys_in_place(ms + U)) k_load(nxt, ms + U);
      if (pending && ms > ph * a.S) {
        q_store(ph + 1, qr);
        pending = false;
      }
      // ms - ph S is a multiple of U; this wave's slice starts S FPS 64 slots further per slice
      const uint4* qb = qs + (ph & 1) * kPhaseU4 + ((slice * a.S + ms - ph * a.S) * FPS) * 64;
#pragma unroll
      for (int h = 0; h < U / VPS; ++h) {
        if (!guard || ms + VPS * h < pfull) {
#pragma unroll
          for (int k = 0; k < VPS; ++k) {
            // operand k: the load ((l%16)/R - k) mod VPS of lane l + R k
            // the register choice: a select of two loaded values, or for 4
            // loads a bit-mask blend (a select chain between array elements
            // would be folded into an indexed stack load)
            uint32_t pick[VPS];
#pragma unroll
            for (int q = 0; q < VPS; ++q) pick[q] = ((qs_lane - k) & (VPS - 1)) == q ? ~0u : 0u;
            uint4 fk[MB];
#pragma unroll
            for (int j = 0; j < MB; ++j) {
              uint4 send = {0u, 0u, 0u, 0u};
              if constexpr (VPS == 2) {
                const uint4 c0 = cur[VPS * h][j], c1 = cur[VPS * h + 1][j];
                send = pick[0] ? c0 : c1;
              } else {
#pragma unroll
                for (int q = 0; q < VPS; ++q) {
                  const uint4 c = cur[VPS * h + q][j];
                  send.x |= c.x & pick[q];
                  send.y |= c.y & pick[q];
                  send.z |= c.z & pick[q];
                  send.w |= c.w & pick[q];
                }
              }
              if constexpr (VPS == 2) {
                fk[j] = k == 0 ? send : row_ror4<8>(send);
              } else {
                fk[j] = k == 0 ? send : (k == 1 ? row_ror4<12>(send) : (k == 2 ? row_ror4<8>(send) : row_ror4<4>(send)));
              }
            }
            uint4 qf[FPS];
#pragma unroll
            for (int f = 0; f < FPS; ++f) qf[f] = qb[((VPS * h + k) * FPS + f) * 64 + lsw[VPS * h + k]];
#pragma unroll
            for (int p = 0; p < P; ++p)
#pragma unroll
              for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int j = 0; j < MB; ++j) M::mac(acc[j][nb], fk[j], qf[p * NB + nb]);
          }
          if constexpr (BASE != kModeLogit) {
            if (++head_seg == a.sph) {
              head_close(head);
              ++head;
              head_seg = 0;
            }
          }
        }
      }
      if (ms + U == (ph + 1) * a.S && ph + 1 < a.nphase) {
        if (pending) {
          q_store(ph + 1, qr);
          pending = false;
        }
        barrier_lds();
        ++ph;
        if (ph + 1 < a.nphase) {
          q_load(ph + 1, qr);
          pending = true;
        }
      }
    };
    // pairs of whole batches (the two register sets alternate without copies),
    // then at most two guarded batches
    int ms = 0;
    for (; ms + 2 * U <= pfull; ms += 2 * U) {
      batch(ms, fa, fb, false);
      batch(ms + U, fb, fa, false);
    }
    if (ms < pfull) {
      batch(ms, fa, fb, true);
      if (ms + U < pfull) batch(ms + U, fb, fa, true);
    }

    // tail steps in plain MFMA shape; lane groups past Lc re-read the previous
    // 32 bytes of their row and contribute zero (the query side is zero too)
    if (pfull < a.ksteps && pending) {  // a last phase holding only the tail
      q_store(ph + 1, qr);
      barrier_lds();
      ++ph;
    }
    for (int v = pfull; v < a.ksteps; ++v) {
      const int col = SEGC * a.nseg + 4 * (v - pfull);  // 16-byte column of lane group 0
      const bool in = (col + g4) * M::EPL < a.Lc;
      const int cph = (col + g4) - (ph << lgC);  // this lane's column within the phase
      const uint4* qb =
          qs + (ph & 1) * kPhaseU4 + (((slice * FPS) << (a.lgS + 6)) + score_q_slot_c<U, VPS, SEGC, FPS>(cph, 0, r16));
      uint4 kf[MB];
#pragma unroll
      for (int j = 0; j < MB; ++j) {
        const uint4 x = k16[j][col + (in ? 0 : -2)];
        kf[j] = in ? x : uint4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int p = 0; p < P; ++p)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const uint4 qf = qb[(p * NB + nb) * 64];
#pragma unroll
          for (int j = 0; j < MB; ++j) M::mac(acc[j][nb], kf[j], qf);
        }
    }

    // the slices' sums: slices 1.. NS-1 publish their accumulators, slice 0
    // adds them in slice order (the buffer lies past the phase buffers in use)
    if constexpr (NS > 1) {
      float* red = reinterpret_cast<float*>(qs + (a.nphase > 1 ? 2 : 1) * kPhaseU4);
      auto red_at = [&](int sl, int j, int nb, int r) __attribute__((always_inline)) {
        return ((((((sl - 1) * TW + tw) * MB + j) * NB + nb) * 4 + r) << 6) + lane;
      };
      if (slice > 0) {
#pragma unroll
        for (int j = 0; j < MB; ++j)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int r = 0; r < 4; ++r) red[red_at(slice, j, nb, r)] = acc[j][nb][r];
      }
      barrier_lds();
      if (slice > 0) continue;  // the next round begins with a barrier of all waves
#pragma unroll
      for (int sl = 1; sl < NS; ++sl)
#pragma unroll
        for (int j = 0; j < MB; ++j)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[j][nb][r] += red[red_at(sl, j, nb, r)];
    }

    if constexpr (BASE == kModeSoftStats) continue;  // the statistics are written
    if constexpr (BASE == kModeSoftProb) {
#pragma unroll
      for (int j = 0; j < MB; ++j)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[j][nb] = prob[j][nb];
    }

    // m_j = scale * max over the query rows: registers over nb, then the 16
    // lanes of a row group; with several queries, one max per query (whole
    // 16-row blocks), max-accumulated when a query began in an earlier chunk
#pragma unroll
    for (int j = 0; j < MB; ++j) {
      if (j < nmb) {
        const int64_t tile = rb + tw + TW * j;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t tok = tile * 16 + g4 * 4 + r;
          if (!SEQ && a.group_rows == 0) {
            float v = -INFINITY;
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
              if (qok[nb]) v = fmaxf(v, acc[j][nb][r]);
#pragma unroll
            for (int o = 8; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 16));
            if (r16 == 0 && tok < a.n_vis) {
              const float x = v * a.scale;
              a.m[tok] = a.accumulate ? fmaxf(a.m[tok], x) : x;
            }
          } else {
            auto store = [&](int g, float v) {
              if (r16 == 0 && tok < a.n_vis) {
                float* dst = a.m + (int64_t)g * a.m_stride + tok;
                const float x = v * a.scale;
                *dst = (int64_t)g * a.group_rows < a.q0 ? fmaxf(*dst, x) : x;
              }
            };
            float vg = -INFINITY;
            int gcur = -1;
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
              // blocks past the chunk's rows belong to no query of it: they
              // are skipped (their g would be a row past m or another
              // sequence's query)
              if (nb * 16 >= a.n_q) break;
              float v = acc[j][nb][r];
#pragma unroll
              for (int o = 8; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 16));
              const int g = (a.q0 + nb * 16) / a.group_rows;
              if (g != gcur) {
                if (gcur >= 0) store(gcur, vg);
                gcur = g;
                vg = v;
              } else {
                vg = fmaxf(vg, v);
              }
            }
            if (gcur >= 0) store(gcur, vg);
          }
        }
      }
    }
  }
  };
  if constexpr (SEQ) {
    // the share, one key sequence at a time
    for (int fb = f_begin; fb < f_end && sidx < a.n_streams;) {
      const QerStreamDesc sd = a.streams[sidx++];
      const int s_end = sd.tile0 + sd.ntiles;
      if (s_end <= fb || sd.ntiles <= 0) continue;
      const int tb = fb - sd.tile0, te = (s_end < f_end ? s_end : f_end) - sd.tile0;
      fb = sd.tile0 + te;
      Kq = K0 + sd.key0 * krow_u4;
      a.n_vis = sd.n_keys;
      a.q0 = sd.q0;
      a.n_q = sd.n_rows;  // whole 16-row blocks (the epilogue skips the others)
      rounds(tb, te);
    }
  } else {
    rounds(f_begin, f_end);
  }
  if constexpr (BASE == kModeSoftStats) {
    // the rounds this workgroup does not run leave empty statistics (a zero
    // sum), which the merge skips
    const int nr = (f_end - f_begin + TW * MB - 1) / (TW * MB);
    for (int rr = nr; rr < a.rounds; ++rr) {
      const int64_t slot = ((int64_t)blockIdx.x * kLdsWaves + wave) * a.rounds + rr;
      for (int i = lane; i < a.H * a.n_q; i += 64) {
        const int hh = i / a.n_q, q = i - hh * a.n_q;
        const int64_t row = (int64_t)hh * a.nq_total + a.q0 + q;
        a.stats_part[((row >> 4) * a.nparts + slot) * 16 + (row & 15)] = make_float2(-INFINITY, 0.f);
      }
    }
  }
}

// ---- several key sequences, up to 128 query rows per chunk: qer_seq_kernel ----------
// The multi-stream workload stacks 4 queries of 32 rows per stream: 128 rows
// per key tile.  There the general score kernel (one tile per wave, query
// fragments restaged through registers with a bank swizzle every round)
// reads 1 KiB of query fragments from LDS per MFMA and stalls at every round
// boundary.  This kernel instead:
//  * takes the query side from a copy in MFMA operand order, written once per
//    call by qer_qop_kernel ([chunk][virtual step][16-row block][lane] x 16 B,
//    rows past the chunk zero), so a phase of query fragments is a contiguous
//    copy, global to registers to LDS, 2 x 16 B per thread and batch, and every
//    fragment read is 1 KiB of consecutive LDS;
//  * gives each wave two tiles of 16 keys (MB = 2): every fragment read from
//    LDS feeds two MFMAs, half the LDS traffic per key byte;
//  * runs one pipeline over all the rounds of the workgroup's share: the key
//    loads of the next round's first batch and the query fragments of its
//    first phase are in flight while the current round finishes, so a round
//    boundary costs only the epilogue.
// Key rows stream in 128-byte segments of 8 rows per load, turned into MFMA
// operands by a lane select and a DPP rotation as in qer_score_kernel.
struct SeqArgs {
  const uint8_t* K;          // [n_vis][Lc] bf16
  const uint4* Qop;          // [chunks][ksteps][8][64] operand-order query fragments
  const QerStreamDesc* seq;  // one per chunk
  int32_t n_seq;
  int32_t tiles;             // over all chunks
  int32_t nwg;
  int32_t xcd_order;
  int32_t nseg;              // segments (1024 / R bytes) per key row: ksteps = (16 / R) nseg, a multiple of kSeqS
  int32_t k_row_u4;          // 16-byte chunks per key row
  float scale;
  float* m;                  // [n_queries][m_stride]
  int64_t m_stride;
  int32_t group_rows;        // rows per query (a multiple of 16)
  int32_t* clear;            // workgroup 0 zeroes clear[0, nclear)
  int32_t nclear;
};

constexpr int kSeqNB = 8;                         // 16-row blocks: 128 query rows
constexpr int kSeqS = 8;                          // virtual steps per phase
constexpr int kSeqPhaseU4 = kSeqS * kSeqNB * 64;  // uint4 per phase (64 KiB)
constexpr int kSeqTab = 64;                       // chunks a workgroup's share may span
constexpr size_t kSeqLds = 2 * (size_t)kSeqPhaseU4 * 16 + kSeqTab * sizeof(QerStreamDesc);

// Key load q of lane `lane` for tile t of a chunk whose keys end at row last:
// 16-byte offset from the chunk's first key row (32-bit: the host keeps a
// sequence's keys under 2^31 16-byte units).  Row R q + lane % R of the tile,
// clamped; chunk VPS (lane / 16) + ((lane % 16) / R - q) mod VPS.
template <int R>
__host__ __device__ __forceinline__ int32_t seq_key_off(int t, int q, int lane, int last, int32_t k_row_u4) {
  constexpr int VPS = 16 / R;
  const int t16 = t * 16 + R * q + lane % R;
  const int tok = t16 < last ? t16 : last;
  return (int32_t)((int64_t)tok * k_row_u4 + VPS * (lane >> 4) + ((((lane & 15) / R) - q) & (VPS - 1)));
}
// Operand-order query copy: element r of a chunk's copy (virtual step v, block
// nb, lane l) holds the 16 bytes of chunk row `row` at 16-byte column `col`.
__host__ __device__ __forceinline__ void qop_source(int64_t r, int R, int& row, int& col) {
  const int vps = 16 / R, segc = 64 / R;
  const int v = (int)(r / (kSeqNB * 64)), nb = (int)((r / 64) % kSeqNB), l = (int)(r & 63);
  row = 16 * nb + (l & 15);
  col = segc * (v / vps) + vps * (l >> 4) + v % vps;
}

// Operand-order copy of the stacked queries: chunk c (rows [q0, q0 + n_rows)
// of the stacked query rows), virtual step v = 2 m + k, block nb, lane l: the
// 16 bytes of row q0 + 16 nb + l % 16 at 16-byte column 8 m + 2 (l / 16) + k
// (zero past n_rows).  With keys read R rows per load (segments of 64 / R
// 16-byte columns, VPS = 16 / R virtual steps each) step v = VPS m + k takes
// column (64 / R) m + VPS (l / 16) + k.
__global__ void qer_qop_kernel(const uint4* Q, int64_t row_u4, const QerStreamDesc* seq, int32_t n_seq,
                               int32_t ksteps, int32_t R, uint4* out) {
  const int64_t per = (int64_t)ksteps * kSeqNB * 64;
  const int64_t total = per * n_seq;
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)(e / per);
    int row, col;
    qop_source(e - c * per, R, row, col);
    const QerStreamDesc sd = seq[c];
    out[e] = row < sd.n_rows ? Q[(int64_t)(sd.q0 + row) * row_u4 + col] : uint4{0u, 0u, 0u, 0u};
  }
}

template <int U, int R>
__global__ __launch_bounds__(kLdsThreads) void qer_seq_kernel(SeqArgs a) {
  constexpr int MB = 2, NB = kSeqNB, TW = kLdsWaves;
  constexpr int VPS = 16 / R, SEGC = 64 / R;  // virtual steps (loads per tile) and 16-byte columns per segment
  constexpr int BPP = kSeqS / U;                    // batches per phase
  constexpr int CP = kSeqPhaseU4 / kLdsThreads / BPP;  // uint4 each thread copies per batch
  static_assert(U % VPS == 0 && kSeqS % U == 0 && CP >= 1, "whole segments per batch, whole batches per phase");
  extern __shared__ uint4 qs[];  // [2][kSeqPhaseU4]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g4 = lane >> 4, own = r16 / R;  // own: the load holding this lane's row
  const int ksteps = VPS * a.nseg, bpr = ksteps / U;  // batches per round
  const int wg = a.xcd_order ? (int)((blockIdx.x & 7) * (a.nwg >> 3) + (blockIdx.x >> 3)) : (int)blockIdx.x;
  const int f_begin = (int)((int64_t)a.tiles * wg / a.nwg);
  const int f_end = (int)((int64_t)a.tiles * (wg + 1) / a.nwg);
  if (blockIdx.x == 0 && a.clear)
    for (int i = tid; i < a.nclear; i += kLdsThreads) a.clear[i] = 0;

  // rounds of the share: RoundDesc of the current and of the next round
  struct Rnd {
    int sidx;      // chunk
    int tb, te;    // first tile of the round, end of the chunk's part of the share (chunk tiles)
    int nmb;       // this wave's valid tiles
  };
  int sidx0 = 0;
  while (sidx0 + 1 < a.n_seq && a.seq[sidx0].tile0 + a.seq[sidx0].ntiles <= f_begin) ++sidx0;
  // the chunks of the share, in LDS past the phase buffers (at most kSeqTab:
  // the host plans shares that span no more), so that a round change reads
  // its descriptors without a memory-counter wait behind the loads in flight
  QerStreamDesc* tab = reinterpret_cast<QerStreamDesc*>(qs + 2 * kSeqPhaseU4);
  for (int i = tid; i < kSeqTab && sidx0 + i < a.n_seq; i += kLdsThreads) tab[i] = a.seq[sidx0 + i];
  __syncthreads();
  const int tab_end = sidx0 + kSeqTab < a.n_seq ? sidx0 + kSeqTab : a.n_seq;
  auto seq_at = [&](int i) __attribute__((always_inline)) { return tab[i - sidx0]; };
  // the round after r (or r.sidx < 0 at the end of the share)
  auto first_of = [&](int si, int from) __attribute__((always_inline)) {
    Rnd r{-1, 0, 0, 0};
    for (; si < tab_end; ++si) {
      const QerStreamDesc sd = seq_at(si);
      const int s_end = sd.tile0 + sd.ntiles;
      if (sd.ntiles <= 0 || s_end <= from) continue;
      if (sd.tile0 >= f_end) break;
      r.sidx = si;
      r.tb = (from > sd.tile0 ? from : sd.tile0) - sd.tile0;
      r.te = (s_end < f_end ? s_end : f_end) - sd.tile0;
      break;
    }
    return r;
  };
  auto next_of = [&](const Rnd& r) __attribute__((always_inline)) {
    if (r.tb + TW * MB < r.te) return Rnd{r.sidx, r.tb + TW * MB, r.te, 0};
    const QerStreamDesc sd = seq_at(r.sidx);
    return first_of(r.sidx + 1, sd.tile0 + r.te);
  };
  auto fill = [&](Rnd& r) __attribute__((always_inline)) {
    int n = 0;
#pragma unroll
    for (int j = 0; j < MB; ++j) n += (r.tb + wave + TW * j < r.te) ? 1 : 0;
    r.nmb = n;
  };
  Rnd cur = first_of(sidx0, f_begin);
  if (cur.sidx < 0) return;
  fill(cur);
  Rnd nxt = next_of(cur);
  if (nxt.sidx >= 0) fill(nxt);

  // key load offsets (16-byte units from the chunk's first key row) of this
  // lane for tile j and load q of a segment: row 8 q + lane % 8 of the tile
  // (clamped to the sequence), chunk 2 g4 + (lane % 16 / 8 - q) mod 2
  const uint4* const K0 = reinterpret_cast<const uint4*>(a.K);
  // key load offsets (16-byte units from the chunk's first key row) of this
  // lane for tile j and load q of a segment: row 8 q + lane % 8 of the tile
  // (clamped to the sequence), chunk 2 g4 + (lane % 16 / 8 - q) mod 2; for
  // the current round (c) and the next (n)
  const uint4* kc_base = K0;
  const uint4* kn_base = K0;
  int32_t kc_off[MB * VPS], kn_off[MB * VPS];
  auto koff = [&](const Rnd& r, const uint4*& base, int32_t (&off)[MB * VPS]) __attribute__((always_inline)) {
    const QerStreamDesc sd = seq_at(r.sidx);
    base = K0 + sd.key0 * a.k_row_u4;
    const int last = sd.n_keys - 1;
#pragma unroll
    for (int j = 0; j < MB; ++j) {
      const int t = j < r.nmb ? r.tb + wave + TW * j : r.tb;  // missing tiles repeat the round's first
#pragma unroll
      for (int q = 0; q < VPS; ++q) off[VPS * j + q] = seq_key_off<R>(t, q, lane, last, a.k_row_u4);
    }
  };
  koff(cur, kc_base, kc_off);
  koff(nxt.sidx >= 0 ? nxt : cur, kn_base, kn_off);  // without a next round: a harmless repeat

  // batch loads: U virtual steps = U / VPS segments, from segment ms / VPS
  auto k_load = [&](uint4 (&f)[U][MB], const uint4* base, const int32_t (&off)[MB * VPS], int ms)
      __attribute__((always_inline)) {
#pragma unroll
    for (int h = 0; h < U / VPS; ++h)
#pragma unroll
      for (int q = 0; q < VPS; ++q)
#pragma unroll
        for (int j = 0; j < MB; ++j) {
          const u32x4v t = __builtin_nontemporal_load(
              reinterpret_cast<const u32x4v*>(base + off[VPS * j + q] + SEGC * (ms / VPS + h)));
          f[VPS * h + q][j] = uint4{t.x, t.y, t.z, t.w};
        }
  };
  // query fragments: phase ph of chunk si is kSeqPhaseU4 contiguous uint4
  auto q_src = [&](int si, int ph) __attribute__((always_inline)) {
    return a.Qop + ((int64_t)si * ksteps + (int64_t)ph * kSeqS) * NB * 64;
  };
  auto barrier_lds = []() __attribute__((always_inline)) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
  };

  // Query fragments move two batches ahead of their store, in two register
  // groups that alternate with the batches: in batch (ph, bp) group bp % 2,
  // loaded two batches before, is stored as slice bp of phase ph + 1, and is
  // loaded again with slice bp + 2 of phase ph + 1 (or slice bp - 2 of phase
  // ph + 2).  (Waiting for a slice then never waits for keys newer than the
  // batch's own.)  Phases count on across rounds: ph + 1 and ph + 2 lie in
  // this round or in the next (a round has at least two phases).
  const int nph = ksteps / kSeqS;
  // (a phase past the share reads the current chunk's data, never used)
  auto phase_src = [&](int pir) __attribute__((always_inline)) {
    const bool next = pir >= nph;
    const int si = next && nxt.sidx >= 0 ? nxt.sidx : cur.sidx;
    return q_src(si, next ? pir - nph : pir);
  };
  // phase 0 of the first round into buffer 0
  {
    const uint4* src = q_src(cur.sidx, 0);
#pragma unroll
    for (int i = 0; i < kSeqPhaseU4 / kLdsThreads; ++i) qs[tid + kLdsThreads * i] = src[tid + kLdsThreads * i];
  }
  // the slices in flight: CP (2 or 4) uint4 per thread and group, in named
  // registers (an array here is placed in scratch memory by the compiler)
  static_assert(CP == 2 || CP == 4, "two or four query uint4 per thread and batch");
  uint4 ca0, ca1, ca2, ca3, cb0, cb1, cb2, cb3;
  auto cp_load = [&](int grp, const uint4* src) __attribute__((always_inline)) {
    uint4 &c0 = grp ? cb0 : ca0, &c1 = grp ? cb1 : ca1, &c2 = grp ? cb2 : ca2, &c3 = grp ? cb3 : ca3;
    c0 = src[0];
    c1 = src[kLdsThreads];
    if constexpr (CP == 4) {
      c2 = src[2 * kLdsThreads];
      c3 = src[3 * kLdsThreads];
    }
  };
  auto cp_store = [&](int grp, uint4* dst) __attribute__((always_inline)) {
    const uint4 &c0 = grp ? cb0 : ca0, &c1 = grp ? cb1 : ca1, &c2 = grp ? cb2 : ca2, &c3 = grp ? cb3 : ca3;
    dst[0] = c0;
    dst[kLdsThreads] = c1;
    if constexpr (CP == 4) {
      dst[2 * kLdsThreads] = c2;
      dst[3 * kLdsThreads] = c3;
    }
  };
  cp_load(0, phase_src(1) + tid);
  cp_load(1, phase_src(1) + CP * kLdsThreads + tid);
  // keys three batches ahead, four register sets rotating with the batches of
  // a phase (BPP = 4): batches 0-2 in flight before the first (a round has at
  // least two phases)
  static_assert(BPP == 4, "four batches per phase: the rotation of the key register sets");
  uint4 fa[U][MB], fb[U][MB], fc[U][MB], fd[U][MB];
  k_load(fa, kc_base, kc_off, 0);
  k_load(fb, kc_base, kc_off, U);
  k_load(fc, kc_base, kc_off, 2 * U);
  barrier_lds();

  f32x4 acc[MB][NB];
#pragma unroll
  for (int j = 0; j < MB; ++j)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[j][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  int gph = 0;  // phases finished (the current phase's buffer is gph & 1)
  // batch bp (a constant after inlining) of phase ph of the current round: the
  // query slice loaded two batches ago stored, the slice two ahead and the keys
  // three batches ahead loaded, this batch's MFMAs
  auto batch = [&](int ph, const int bp, const uint4 (&cur_k)[U][MB], uint4 (&nxt_k)[U][MB])
      __attribute__((always_inline)) {
    // (unconditional, so that the memory-counter waits stay exact: a slice of
    // a phase past the share lands in a buffer no later phase reads)
    cp_store(bp & 1, qs + ((gph + 1) & 1) * kSeqPhaseU4 + bp * CP * kLdsThreads + tid);
    {
      const bool wrap = bp + 2 >= BPP;
      cp_load(bp & 1, phase_src(ph + (wrap ? 2 : 1)) + (wrap ? bp + 2 - BPP : bp + 2) * CP * kLdsThreads + tid);
    }
    // the keys of the batch three ahead: this round's, or one of the next
    // round's first three (unconditional loads: past the last round they
    // repeat its first batches)
    {
      const int ahead = BPP * ph + bp + 3;
      const bool from_next = ahead >= bpr;
      int32_t off[MB * VPS];
#pragma unroll
      for (int i = 0; i < MB * VPS; ++i) off[i] = from_next ? kn_off[i] : kc_off[i];
      k_load(nxt_k, from_next ? kn_base : kc_base, off, (from_next ? ahead - bpr : ahead) * U);
    }
    // keep the loads ahead of this batch's multiplies (the scheduler would
    // otherwise sink them to the batch end, leaving nothing in flight)
    __builtin_amdgcn_sched_barrier(0);
    const uint4* qb = qs + (gph & 1) * kSeqPhaseU4 + (bp * U) * NB * 64 + lane;
#pragma unroll
    for (int v = 0; v < U; ++v) {
      const int h = v / VPS, k = v % VPS;
      uint4 fk[MB];
#pragma unroll
      for (int j = 0; j < MB; ++j) {
        // operand k: load (lane % 16 / R - k) mod VPS of lane + R k within its
        // 16-lane row (a bit-mask blend, then a DPP rotation; a select between
        // the array's elements would be folded into an indexed scratch load)
        uint4 send = uint4{0u, 0u, 0u, 0u};
#pragma unroll
        for (int q = 0; q < VPS; ++q) {
          const uint32_t pick = ((own - k) & (VPS - 1)) == q ? ~0u : 0u;
          const uint4 c = cur_k[VPS * h + q][j];
          send.x |= c.x & pick;
          send.y |= c.y & pick;
          send.z |= c.z & pick;
          send.w |= c.w & pick;
        }
        if constexpr (VPS == 2)
          fk[j] = k == 0 ? send : row_ror4<8>(send);
        else
          fk[j] = k == 0 ? send : (k == 1 ? row_ror4<12>(send) : (k == 2 ? row_ror4<8>(send) : row_ror4<4>(send)));
      }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const uint4 qf = qb[(v * NB + nb) * 64];
#pragma unroll
        for (int j = 0; j < MB; ++j) Mma<bf16_t>::mac(acc[j][nb], fk[j], qf);
      }
    }
  };

  while (cur.sidx >= 0) {
    for (int ph = 0; ph < nph; ++ph) {
      batch(ph, 0, fa, fd);
      batch(ph, 1, fb, fa);
      batch(ph, 2, fc, fb);
      batch(ph, 3, fd, fc);
      barrier_lds();  // phase end: the next phase is in place, this buffer free
      ++gph;
    }
    // m_j = scale * max over each query's rows, for this wave's tiles
    const QerStreamDesc sd = seq_at(cur.sidx);
#pragma unroll
    for (int j = 0; j < MB; ++j) {
      if (j < cur.nmb) {
        const int tile = cur.tb + wave + TW * j;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int tok = tile * 16 + g4 * 4 + r;
          float vg = -INFINITY;
          int gcur = -1;
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) {
            if (nb * 16 >= sd.n_rows) break;
            float v = acc[j][nb][r];
#pragma unroll
            for (int o = 8; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 16));
            const int g = (sd.q0 + nb * 16) / a.group_rows;
            if (g != gcur) {
              if (gcur >= 0 && r16 == 0 && tok < sd.n_keys) a.m[(int64_t)gcur * a.m_stride + tok] = vg * a.scale;
              gcur = g;
              vg = v;
            } else {
              vg = fmaxf(vg, v);
            }
          }
          if (gcur >= 0 && r16 == 0 && tok < sd.n_keys) a.m[(int64_t)gcur * a.m_stride + tok] = vg * a.scale;
        }
      }
    }
#pragma unroll
    for (int j = 0; j < MB; ++j)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[j][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    cur = nxt;
    kc_base = kn_base;
#pragma unroll
    for (int i = 0; i < MB * VPS; ++i) kc_off[i] = kn_off[i];
    if (cur.sidx >= 0) {
      nxt = next_of(cur);
      if (nxt.sidx >= 0) fill(nxt);
      koff(nxt.sidx >= 0 ? nxt : cur, kn_base, kn_off);
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

// Eq. 8: the k frames of largest score (ties to the lower index), written in
// chronological order and padded with -1, by the whole workgroup (blockDim a
// multiple of 64, at least 256).  Up to kTopkCount frames each frame's rank
// is counted against every key.  Beyond, a radix select on the
// order-preserving 32-bit keys finds the k-th largest key (8 bits per pass,
// the digit located by a suffix scan of the 256 digit counts) and how many
// keys equal to it are taken; a scan over the frames in index order then
// writes the selected indices, each thread owning a contiguous chunk of
// frames.
constexpr int kTopkCount = 128;   // up to this many frames: ranks by counting
constexpr int kTopkStage = 8192;  // up to this many frames: keys staged in LDS

__device__ void topk_block(const uint32_t* keys_g, int32_t n_frames, int32_t k_top, int32_t* out_idx) {
  __shared__ __align__(16) uint32_t keys_sh[kTopkStage];
  __shared__ int hist[256];
  __shared__ int wsum[16];
  __shared__ uint32_t sh_prefix;
  __shared__ int sh_need;
  const int tid = threadIdx.x, nthr = blockDim.x, lane = tid & 63, wave = tid >> 6;
  const int k = k_top < n_frames ? k_top : n_frames;
  if (k > 0 && n_frames <= kTopkCount) {
    // rank = frames that beat f; keys are read four at a time (the LDS copy is
    // padded with zero keys, which never beat anything: a key is >= the key
    // of -inf, 0x007FFFFF)
    const int padded = (n_frames + 3) & ~3;
    for (int f = tid; f < padded; f += nthr) keys_sh[f] = f < n_frames ? keys_g[f] : 0u;
    __syncthreads();
    int sel = 0;
    if (tid < n_frames) {
      const uint32_t kf = keys_sh[tid];
      const uint4* k4 = reinterpret_cast<const uint4*>(keys_sh);
      int rank = 0;
#pragma unroll 4
      for (int q = 0; q < padded / 4; ++q) {
        const uint4 v = k4[q];
        const int g = 4 * q;
        rank += (v.x > kf) || (v.x == kf && g < tid);
        rank += (v.y > kf) || (v.y == kf && g + 1 < tid);
        rank += (v.z > kf) || (v.z == kf && g + 2 < tid);
        rank += (v.w > kf) || (v.w == kf && g + 3 < tid);
      }
      sel = rank < k ? 1 : 0;
    }
    int total;
    const int pos = block_exscan(sel, &total, wsum);
    if (sel) out_idx[pos] = tid;
  } else if (k > 0) {
    const bool staged = n_frames <= kTopkStage;
    const uint32_t* keys = staged ? keys_sh : keys_g;
    if (staged) {
      for (int f = tid; f < n_frames; f += nthr) keys_sh[f] = keys_g[f];
    }
    const int chunk = (n_frames + nthr - 1) / nthr;
    const int f_lo = tid * chunk < n_frames ? tid * chunk : n_frames;
    const int f_hi = f_lo + chunk < n_frames ? f_lo + chunk : n_frames;
    uint32_t prefix = 0, mask = 0;
    int need = k;
    for (int shift = 24; shift >= 0; shift -= 8) {
      if (tid < 256) hist[tid] = 0;
      __syncthreads();
      for (int f = f_lo; f < f_hi; ++f) {
        const uint32_t key = keys[f];
        if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1);
      }
      __syncthreads();
      // thread t < 256 takes digit d = 255 - t; an inclusive scan over t gives
      // the count of keys with digit >= d, so exactly one d has
      // (count > d) < need <= (count >= d)
      int ge = 0, cnt = 0;
      if (tid < 256) {
        cnt = hist[255 - tid];
        ge = cnt;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int y = __shfl_up(ge, o);
          if (lane >= o) ge += y;
        }
        if (lane == 63) wsum[wave] = ge;
      }
      __syncthreads();
      if (tid < 256) {
        for (int i = 0; i < wave; ++i) ge += wsum[i];
        const int above = ge - cnt;
        if (above < need && need <= ge) {
          sh_prefix = prefix | ((uint32_t)(255 - tid) << shift);
          sh_need = need - above;
        }
      }
      __syncthreads();
      prefix = sh_prefix;
      need = sh_need;
      mask |= 255u << shift;
    }
    // prefix = the k-th largest key; `need` keys equal to it are taken, the
    // lowest frame indices first
    int n_eq = 0;
    for (int f = f_lo; f < f_hi; ++f) n_eq += keys[f] == prefix ? 1 : 0;
    int total;
    int eq_rank = block_exscan(n_eq, &total, wsum);
    int n_sel = 0;
    for (int f = f_lo; f < f_hi; ++f) {
      const uint32_t key = keys[f];
      const bool eq = key == prefix;
      n_sel += (key > prefix || (eq && eq_rank < need)) ? 1 : 0;
      eq_rank += eq ? 1 : 0;
    }
    int pos = block_exscan(n_sel, &total, wsum);
    eq_rank -= n_eq;
    for (int f = f_lo; f < f_hi; ++f) {
      const uint32_t key = keys[f];
      const bool eq = key == prefix;
      if (key > prefix || (eq && eq_rank < need)) out_idx[pos++] = f;
      eq_rank += eq ? 1 : 0;
    }
  }
  for (int i = k + tid; i < k_top; i += nthr) out_idx[i] = -1;
}

// One query of a launch over several key sequences: its sequence's frames
// are [frame0, frame0 + n_frames) of the launch's CSR, whose key rows start
// at key0 (n_keys rows), and it ranks the first nf of them.
struct QerQueryDesc {
  int64_t key0;
  int32_t n_keys;
  int32_t frame0;
  int32_t n_frames;
  int32_t nf;
};

// Eq. 7: w_f = mean over the frame's visual tokens of m_j; one wave per frame
// (wave w of the grid takes frames w, w + waves, ...), fp64 partial sums in a
// fixed lane order.  Also writes the frame's sort key.
// Several queries (blockIdx.y): query g reads row g of m, covers its first
// nf_q[g] frames (all when nf_q is null) and writes row g of the scores and
// keys; frames past its prefix score -inf.
// trees != null (1024 threads; one zeroed arrival tree of tree_ints ints per
// query): the last workgroup of query g to finish also selects its top k
// (Eq. 8) into row g of out_idx, so the selection needs no launch of its own.
// qd != null (several key sequences): query g takes its frames, key rows and
// prefix from qd[g]; n_vis and n_frames are then only the row strides of m
// and of the scores and keys.
__global__ __launch_bounds__(1024) void qer_frame_mean_kernel(const float* m, int32_t n_vis,
                                                              const int32_t* offs, int32_t n_frames,
                                                              float* out_scores, uint32_t* keys,
                                                              const int32_t* nf_q, int32_t* trees,
                                                              int32_t tree_ints, int32_t tree_stride,
                                                              int32_t k_top, int32_t* out_idx,
                                                              const QerQueryDesc* qd) {
  const int lane = threadIdx.x & 63;
  const int64_t g = blockIdx.y;
  int32_t nf = nf_q ? nf_q[g] : n_frames;
  int32_t nfr = n_frames, nv = n_vis;
  int64_t key0 = 0;
  m += g * n_vis;
  out_scores += g * n_frames;
  keys += g * n_frames;
  if (qd) {
    const QerQueryDesc q = qd[g];
    offs += q.frame0;
    key0 = q.key0;
    nv = q.n_keys;
    nfr = q.n_frames;
    nf = q.nf;
  }
  // every wave takes frames (blockIdx.x * waves + wave) + k * (grid * waves)
  const int64_t fstep = (int64_t)gridDim.x * (blockDim.x >> 6);
  for (int64_t f = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6); f < nfr; f += fstep) {
  if (f >= nf) {
    if (lane == 0) {
      out_scores[f] = -INFINITY;
      st_agent(keys + f, order_key(-INFINITY));
    }
  } else {
    int64_t lo64 = (int64_t)offs[f] - key0, hi64 = (int64_t)offs[f + 1] - key0;
    const int lo = (int)(lo64 < 0 ? 0 : (lo64 > nv ? nv : lo64));
    const int hi = (int)(hi64 < lo ? lo : (hi64 > nv ? nv : hi64));
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
      st_agent(keys + f, order_key(w));
    }
  }
  }
  if (trees) {
    __shared__ int32_t last_sh;
    if (arrive_last(trees + g * tree_ints, tree_stride, (int32_t)blockIdx.x, (int32_t)gridDim.x, &last_sh))
      topk_block(keys, nf, k_top, out_idx + g * k_top);
  }
}

// Several queries: workgroup g ranks the first nf_q[g] keys of row g (stride
// n_stride) and writes row g of out_idx; nf_q null = one query of n_stride keys.
__global__ __launch_bounds__(1024) void qer_topk_kernel(const uint32_t* keys_g, int32_t n_stride,
                                                        int32_t k_top, int32_t* out_idx, const int32_t* nf_q) {
  const int64_t gq = blockIdx.x;
  topk_block(keys_g + gq * n_stride, nf_q ? nf_q[gq] : n_stride, k_top, out_idx + gq * k_top);
}

// ---- top-k of given scores; evidence preservation ----------------------------------
__global__ void order_keys_kernel(const float* w, int32_t n, uint32_t* keys) {
  for (int64_t f = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; f < n; f += (int64_t)gridDim.x * blockDim.x)
    keys[f] = order_key(w[f]);
}

// out[0] = sum of w over the masked frames / sum over all (0 if the total is
// 0); out[1] = share of the top-k frames that are masked.  fp64 sums, one
// workgroup: each thread a contiguous chunk of frames, then a fixed tree.
__global__ __launch_bounds__(1024) void evidence_kernel(const float* w, const uint8_t* mask, int32_t n,
                                                        const int32_t* top, int32_t k, double* out) {
  __shared__ double tot_sh[1024], kept_sh[1024];
  __shared__ int hit_sh[1024];
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int chunk = (n + nthr - 1) / nthr;
  const int lo = tid * chunk < n ? tid * chunk : n, hi = lo + chunk < n ? lo + chunk : n;
  double tot = 0, kept = 0;
  for (int f = lo; f < hi; ++f) {
    const double v = (double)w[f];
    tot += v;
    if (mask[f]) kept += v;
  }
  int hit = 0;
  for (int i = tid; i < k; i += nthr) hit += mask[top[i]] ? 1 : 0;
  tot_sh[tid] = tot;
  kept_sh[tid] = kept;
  hit_sh[tid] = hit;
  __syncthreads();
  for (int o = nthr / 2; o > 0; o >>= 1) {
    if (tid < o) {
      tot_sh[tid] += tot_sh[tid + o];
      kept_sh[tid] += kept_sh[tid + o];
      hit_sh[tid] += hit_sh[tid + o];
    }
    __syncthreads();
  }
  if (tid == 0) {
    out[0] = tot_sh[0] != 0 ? kept_sh[0] / tot_sh[0] : 0.0;
    out[1] = k > 0 ? (double)hit_sh[0] / (double)k : 0.0;
  }
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

// Row statistics from per-part (max, sum of exp) pairs, part b of row r at
// partial[b * ps + r * rs]: one wave per row, parts strided over the lanes;
// the max, then sum_b z_b exp(m_b - max) in fp64, each over the lanes and a
// fixed xor tree.  Parts with a zero sum (no tokens) are skipped.
// stats[r] = (max, sum of exp(s - max)).
__global__ __launch_bounds__(256) void qer_soft_merge_kernel(const float2* partial, int64_t nparts, int64_t ps,
                                                             int64_t rs, int32_t rows, float2* stats) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;  // whole waves; the kernel has no barrier
  const float2* src = partial + r * rs;
  float mx = -INFINITY;
  for (int64_t b = lane; b < nparts; b += 64) {
    const float2 v = src[b * ps];
    if (v.y > 0.f) mx = fmaxf(mx, v.x);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  double z = 0.0;
  for (int64_t b = lane; b < nparts; b += 64) {
    const float2 v = src[b * ps];
    if (v.y > 0.f) z += (double)v.y * (double)__expf(v.x - mx);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) z += __shfl_xor(z, o);
  if (lane == 0) stats[r] = make_float2(mx, (float)z);
}

// The same for the score kernel's pass-1 layout (rows in blocks of 16, part b
// of the block at [b][16]): workgroup per 16 rows, thread t takes row t % 16
// and parts t / 16 + 64 u (each load of the workgroup is 64 consecutive
// parts, 8 KiB), 32 of them in flight at a time: their max, then the sum of
// z exp(m - max) in fp64 from registers, folded into the thread's running
// pair.  The 64 pairs of a row are then combined pairwise in LDS (a fixed
// tree of six levels).
__global__ __launch_bounds__(1024) void qer_soft_merge_blocked_kernel(const float2* partial, int64_t nparts,
                                                                      int32_t rows, float2* stats) {
  __shared__ float mx_sh[64][16];
  __shared__ double z_sh[64][16];
  constexpr int C = 32;
  const int tid = threadIdx.x, r16 = tid & 15, grp = tid >> 4;
  const float2* src = partial + (int64_t)blockIdx.x * nparts * 16 + r16;
  float M = -INFINITY;
  double Z = 0.0;
  for (int64_t b0 = grp; b0 < nparts; b0 += 64 * C) {
    float2 v[C];
#pragma unroll
    for (int u = 0; u < C; ++u) {
      const int64_t b = b0 + 64 * u;
      v[u] = b < nparts ? src[b * 16] : make_float2(-INFINITY, 0.f);
    }
    float m = M;
#pragma unroll
    for (int u = 0; u < C; ++u) m = v[u].y > 0.f ? fmaxf(m, v[u].x) : m;
    double z = Z > 0.0 ? Z * (double)__expf(M - m) : 0.0;
#pragma unroll
    for (int u = 0; u < C; ++u) z += v[u].y > 0.f ? (double)v[u].y * (double)__expf(v[u].x - m) : 0.0;
    M = m;
    Z = z;
  }
  mx_sh[grp][r16] = M;
  z_sh[grp][r16] = Z;
  for (int half = 32; half > 0; half >>= 1) {
    __syncthreads();
    if (grp < half) {
      const float m1 = mx_sh[grp][r16], m2 = mx_sh[grp + half][r16];
      const double z1 = z_sh[grp][r16], z2 = z_sh[grp + half][r16];
      const float m = z1 > 0.0 ? (z2 > 0.0 ? fmaxf(m1, m2) : m1) : m2;
      const double z = (z1 > 0.0 ? z1 * (double)__expf(m1 - m) : 0.0) + (z2 > 0.0 ? z2 * (double)__expf(m2 - m) : 0.0);
      mx_sh[grp][r16] = m;
      z_sh[grp][r16] = z;
    }
  }
  if (tid < 16) {
    const int64_t r = (int64_t)blockIdx.x * 16 + tid;
    if (r < rows) stats[r] = make_float2(mx_sh[0][tid], (float)z_sh[0][tid]);
  }
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
  // SOFTMAX through the LDS-staged score kernel: heads of whole 128-byte
  // segments, the pass-2 statistics and the segment map within the LDS budget
  bool soft_fast;
  bool soft_wide;       // 128 query rows per pass (else 64)
  int64_t soft_nwg;     // workgroups of the score kernel (qer_soft_grp_kernel: pass 1's key ranges)
  int64_t soft_rounds;  // their rounds (qer_soft_grp_kernel: 1)
  // SOFTMAX through qer_soft_grp_kernel (grouped bf16 heads of d = 128, one query)
  bool soft_grp;
};

struct QerScratch {
  float* m;        // [n_queries][n_vis]
  uint32_t* keys;  // [n_queries][n_frames]
  uint8_t* qp;
  float2* partial;
  float2* stats;
  int32_t* nf;     // [n_queries] frames per query (several queries only)
  int32_t* done;   // [n_queries][tree_ints] arrival trees of the frame-mean kernel
};

// Arrival trees of the frame-mean kernel (16 frames per workgroup).
struct QerTrees {
  int32_t nwg, ints, stride;
};
// Grid of the frame-mean kernel (16 waves a workgroup): one frame per wave
// while the queries' workgroups fit one per CU, else each wave strides over
// ceil(workgroups / CUs) frames, so the launch stays one round on the chip
// (fewer, fuller waves and a shallower arrival tree per query).
inline QerTrees qer_trees(int32_t n_frames, int32_t n_queries) {
  QerTrees t;
  const int64_t one = ((int64_t)n_frames + 15) / 16, cus = device_cu_count();
  const int64_t fpw = std::max<int64_t>(1, (one * std::max(n_queries, 1) + cus - 1) / cus);
  t.nwg = (int32_t)(((int64_t)n_frames + 16 * fpw - 1) / (16 * fpw));
  t.stride = arrive_fan(t.nwg) > 0 ? 16 : 1;
  t.ints = (arrive_fan(t.nwg) + 1) * t.stride;
  return t;
}

QerScratch carve_qer(Arena& ar, const cofie_qer_desc& h, const QerPlan& p, int32_t n_queries = 1) {
  QerScratch w;
  w.m = ar.take<float>((size_t)n_queries * (h.n_vis > 0 ? h.n_vis : 1));
  w.keys = ar.take<uint32_t>((size_t)n_queries * (h.n_frames > 0 ? h.n_frames : 1));
  w.qp = p.fold ? ar.take<uint8_t>((size_t)p.P * n_queries * h.n_q * p.Lc * p.esize) : nullptr;
  // (the SOFTMAX partial statistics are carved below)
  w.nf = n_queries > 1 ? ar.take<int32_t>((size_t)n_queries) : nullptr;
  w.done = ar.take<int32_t>((size_t)n_queries * qer_trees(h.n_frames, n_queries).ints);
  if (h.score_mode == COFIE_SCORE_SOFTMAX) {
    // the score kernel's statistics: rows (heads x query rows) in whole blocks
    // of 16, per wave and round
    const size_t rows16 = (size_t)ceil_div((int64_t)h.H_q * h.n_q * n_queries, 16) * 16;
    w.partial = p.soft_grp    ? ar.take<float2>((size_t)p.soft_nwg * rows16)
                : p.soft_fast ? ar.take<float2>((size_t)p.soft_nwg * kLdsWaves * p.soft_rounds * rows16)
                              : ar.take<float2>((size_t)p.nblk_soft * h.H_q * h.n_q);
    w.stats = ar.take<float2>((size_t)h.H_q * h.n_q * n_queries);
  } else {
    w.partial = nullptr;
    w.stats = nullptr;
  }
  return w;
}

void plan_soft(const cofie_qer_desc& h, int32_t n_queries, QerPlan& p);

// n_queries: queries of h.n_q rows each sharing K (cofie_qer_rank_batched)
QerPlan plan_qer(const cofie_qer_desc& h, int32_t n_queries = 1) {
  QerPlan p;
  p.esize = h.dtype == COFIE_BF16 ? 2 : 4;
  p.fold = h.score_mode == COFIE_SCORE_LOGIT && h.H_q != h.H_kv;
  p.Lc = (int64_t)(p.fold ? h.H_kv : h.H_q) * h.d;  // MHA: H_q == H_kv
  p.P = (p.fold && h.dtype == COFIE_BF16) ? 3 : 1;
  p.nblk_soft = (h.n_vis + kMB * 16 - 1) / (kMB * 16);
  plan_soft(h, n_queries, p);
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

// Work split of the LDS-staged score kernel: one workgroup per CU (fewer for
// small inputs), tiles of 16 tokens spread evenly over the workgroups, 1 or 2
// tiles per wave per round, 4-row key segments unless the batch is too short
// to hold one, phases as long as a 64 KiB buffer allows.  Inputs of too few
// tiles to give every wave of the chip a tile split the contraction NS ways
// (NS depends on the tile count, the contraction and the query terms only, not
// on the query rows, so that queries ranked together or alone add in the same
// order).
struct LdsPlan {
  int MB, R, NS, nwg, S, lgS, nphase, nseg, ksteps, split_u4;
  size_t lds;
};

// Slices of the contraction for `tiles` tiles: the largest NS in {4, 2} whose
// tiles still take one round (one tile per wave group on at most every CU:
// each further round restages the whole query side and restarts the key
// pipeline, measured at ~11 us per round for the multi-stream heads, more than
// the split saves), else 1.  Whole segments per slice, no tail steps, one
// query term.
inline int plan_slices(int64_t tiles, int64_t Lc, size_t esize, int P, int cus) {
  const int64_t seg_el = (1024 / lds_rows(1, 1)) / (int64_t)esize;
  if (P != 1 || Lc % seg_el != 0) return 1;
  const int64_t nseg = Lc / seg_el;
  for (int ns = 4; ns > 1; ns /= 2)
    if (nseg % ns == 0 && tiles <= (int64_t)cus * (kLdsWaves / ns)) return ns;
  return 1;
}

LdsPlan plan_score_lds(int64_t n_vis, int64_t Lc, size_t esize, int P, int PNB, int cus, bool split_ok) {
  LdsPlan L;
  const int64_t tiles = ceil_div(n_vis, 16);
  L.NS = split_ok ? plan_slices(tiles, Lc, esize, P, cus) : 1;
  const int tw = kLdsWaves / L.NS;
  L.nwg = (int)std::min<int64_t>(cus, ceil_div(tiles, tw));
  const int64_t tpw = ceil_div(tiles, L.nwg);
  L.MB = (L.NS == 1 && tpw > kLdsWaves) ? 2 : 1;
  L.R = lds_rows(L.MB, PNB);
  const int U = lds_batch(L.MB, PNB, L.R, L.NS);
  const int64_t kps = 64 / (int64_t)esize;             // elements per plain MFMA step
  const int64_t seg_el = (1024 / L.R) / (int64_t)esize;  // elements per segment
  const int64_t Ls = Lc / L.NS;                        // one slice (whole segments when NS > 1)
  L.nseg = (int)(Ls / seg_el);
  L.ksteps = (int)((16 / L.R) * L.nseg + ceil_div(Ls % seg_el, kps));
  L.split_u4 = (int)(Ls * (int64_t)esize / 16);
  const int phase_u4 = lds_q_regs(PNB, L.NS) * kLdsThreads;
  // S: a power of two (>= U), as large as the phase buffer holds (NS slices
  // of S steps), no larger than the contraction needs
  const int64_t cap = (phase_u4 / 64) / PNB / L.NS;
  L.S = U;
  while (2 * L.S <= cap && L.S < L.ksteps) L.S *= 2;
  L.lgS = 0;
  while ((1 << L.lgS) < L.S) ++L.lgS;
  L.nphase = (int)ceil_div(L.ksteps, L.S);
  L.lds = (size_t)(L.nphase > 1 ? 2 : 1) * phase_u4 * sizeof(uint4);
  if (L.NS > 1) L.lds += (size_t)(L.NS - 1) * tw * PNB * 4 * 64 * sizeof(float);
  return L;
}

// ---- address models (dry run) -------------------------------------------------------
// Host walks of the addresses that a kernel's threads touch, computed by the
// index functions the kernel itself uses, each checked against the registered
// buffers or the launch's LDS.  An address affine in a loop counter (the key
// segments of a row) is checked at both ends of the loop, which bounds every
// address between them.  Values that decide an index and lie in device
// memory are read from the host copies of the plan tables (dry_shadow).

template <typename T>
const T* shadow_of(const T* dev, const char* what) {
  const T* p = static_cast<const T*>(dry_shadow(dev));
  if (!p && dev) dry_range(0, 0, 0, what);  // a table no copy wrote: reported as a violation
  return p;
}

// qer_score_kernel with grid `grid` and `lds` bytes of LDS
template <typename T, int MB, int NB, int P, int NS, int MODE>
void model_score(ScoreLdsArgs a, int grid, size_t lds) {
  constexpr int BASE = MODE & 3;
  constexpr bool GQA = (MODE & kModeGqa) != 0;
  constexpr bool SEQ = (MODE & kModeSeq) != 0;
  constexpr int R = lds_rows(MB, P * NB);
  constexpr int VPS = 16 / R, SEGC = 64 / R;
  constexpr int U = score_batch(MB, NB, P, NS, MODE);
  constexpr int FPS = P * NB;
  constexpr int kQRegs = lds_q_regs(FPS, NS);
  constexpr int kPhaseU4 = kQRegs * kLdsThreads;
  constexpr int TW = kLdsWaves / NS;
  const int64_t L = (int64_t)lds;
  const int lgC = a.lgS + 2;
  const int pfull = VPS * a.nseg;
  const int64_t row_u4 = (int64_t)a.Lc * sizeof(T) / 16;
  const int64_t krow_u4 = a.k_row_u4;
  dry_range(grid, a.nwg, a.nwg + 1, "score: grid and planned workgroups differ");
  if (a.xcd_order) dry_range(a.nwg % 8, 0, 1, "score: XCD order needs whole groups of 8 workgroups");
  if (a.clear && a.nclear > 0) dry_access(a.clear, 0, 4 * (int64_t)a.nclear, "score: arrival counters");
  // LDS past the phase buffers
  const int64_t extra = (int64_t)(a.nphase > 1 ? 2 : 1) * kPhaseU4 * 16;
  if constexpr (BASE == kModeSoftProb) dry_lds(extra, (int64_t)a.H * a.n_q * 8, L, "score: row statistics in LDS");
  int seg_lo = 0, seg_hi = a.nseg - 1;  // the key segments read (mapped for grouped heads)
  if constexpr (GQA) {
    dry_lds(extra + (BASE == kModeSoftProb ? (int64_t)a.H * a.n_q * 8 : 0), 4 * (int64_t)a.nseg, L,
            "score: segment map");
    seg_lo = INT32_MAX;
    seg_hi = -1;
    for (int v = 0; v < a.nseg; ++v) {
      const int sm = (v / a.sph / a.G) * a.sph + v % a.sph;
      seg_lo = std::min(seg_lo, sm);
      seg_hi = std::max(seg_hi, sm);
    }
  }
  if constexpr (NS > 1) dry_lds(extra, (int64_t)(NS - 1) * TW * MB * NB * 4 * 64 * 4, L, "score: slice sums");
  if constexpr (BASE == kModeSoftProb)
    if (a.H * a.n_q > 0) {
      dry_access(a.stats, ((int64_t)a.q0) * 8, 8, "score: pass-2 statistics");
      dry_access(a.stats, ((int64_t)(a.H - 1) * a.nq_total + a.q0 + a.n_q - 1) * 8, 8, "score: pass-2 statistics");
    }

  // query fragment stores: slots inside the phase buffer, both buffers
  for (int par = 0; par < (a.nphase > 1 ? 2 : 1); ++par)
    for (int e = 0; e < kPhaseU4; ++e) {
      const int slot = score_q_slot<U, VPS, SEGC, FPS, NS>(e, lgC, a.lgS);
      dry_range(slot, 0, kPhaseU4, "score: query slot outside its phase buffer");
      dry_lds(((int64_t)par * kPhaseU4 + slot) * 16, 16, L, "score: query fragment store");
    }
  // fragment reads of the batches and the tail, following the kernel's phase
  // counter; phase ph's buffer is ph % 2
  for (int slice = 0; slice < NS; ++slice) {
    int ph = 0;
    bool pending = a.nphase > 1;
    for (int ms = 0; ms < pfull; ms += U) {
      if (pending && ms > ph * a.S) pending = false;
      const int64_t qb = ((int64_t)slice * a.S + ms - (int64_t)ph * a.S) * FPS * 64;
      for (int h = 0; h < U / VPS; ++h) {
        if (ms + VPS * h >= pfull) continue;
        for (int k = 0; k < VPS; ++k) {
          const int64_t lo = qb + (int64_t)((VPS * h + k) * FPS) * 64, hi = lo + (int64_t)(FPS - 1) * 64 + 63;
          dry_range(lo, 0, kPhaseU4, "score: batch fragment read outside its phase buffer");
          dry_range(hi, 0, kPhaseU4, "score: batch fragment read outside its phase buffer");
          dry_lds(((ph & 1) * (int64_t)kPhaseU4 + lo) * 16, (hi - lo + 1) * 16, L, "score: batch fragment read");
        }
      }
      if (ms + U == (ph + 1) * a.S && ph + 1 < a.nphase) {
        pending = false;
        ++ph;
        if (ph + 1 < a.nphase) pending = true;
      }
    }
    if (pfull < a.ksteps && pending) ++ph;
    for (int v = pfull; v < a.ksteps; ++v) {
      const int col = SEGC * a.nseg + 4 * (v - pfull);
      for (int lane = 0; lane < 64; ++lane) {
        const int cph = col + (lane >> 4) - (ph << lgC);
        dry_range(cph, 0, 1 << lgC, "score: tail column outside its phase");
        const int64_t slot = ((int64_t)(slice * FPS) << (a.lgS + 6)) + score_q_slot_c<U, VPS, SEGC, FPS>(cph, 0, lane & 15);
        for (int f = 0; f < FPS; ++f) {
          dry_range(slot + f * 64, 0, kPhaseU4, "score: tail fragment read outside its phase buffer");
          dry_lds(((ph & 1) * (int64_t)kPhaseU4 + slot + f * 64) * 16, 16, L, "score: tail fragment read");
        }
      }
    }
  }

  // the chunk's query rows (q0, n_q): every phase's loads
  auto q_loads = [&](int q0, int n_q) {
    for (int ph = 0; ph < a.nphase; ++ph)
      for (int e = 0; e < kPhaseU4; ++e) {
        bool ok;
        const int64_t src = score_q_u4<NB, NS, FPS, Mma<T>::EPL>(n_q, q0, a.nq_total, a.Lc, a.split_u4, e, ph, lgC,
                                                                 row_u4, ok);
        dry_access(a.Qp, src * 16, 16, "score: query load");
      }
  };
  std::vector<std::pair<int, int>> q_done;
  const int32_t* nf_h = nullptr;
  if constexpr (BASE == kModeSoftStats)
    if (a.soft_nf) nf_h = shadow_of(a.soft_nf, "score: per-query frame counts without a host copy");
  // tiles [t_begin, t_end) of one key sequence for workgroup b
  auto share = [&](int b, int t_begin, int t_end, int64_t kbase_u4, int64_t n_vis, int q0, int n_q) {
    if (std::find(q_done.begin(), q_done.end(), std::make_pair(q0, n_q)) == q_done.end()) {
      q_done.push_back({q0, n_q});
      q_loads(q0, n_q);
    }
    if constexpr (BASE == kModeSoftStats) {
      if (a.soft_nf)
        for (int nb = 0; nb < NB; ++nb)
          if (nb * 16 < n_q) {
            const int gi = (q0 + nb * 16) / a.group_rows;
            dry_access(a.soft_nf, 4 * (int64_t)gi, 4, "score: per-query frame count");
            if (nf_h) dry_access(a.soft_offs, 4 * (int64_t)nf_h[gi], 4, "score: the query's key limit");
          }
    }
    const int64_t last = n_vis - 1;
    for (int rb = t_begin; rb < t_end; rb += TW * MB) {
      const int rr = (rb - t_begin) / (TW * MB);
      if constexpr (BASE == kModeSoftStats) dry_range(rr, 0, a.rounds, "score: round past the statistics slots");
      for (int tw = 0; tw < TW; ++tw) {
        int nmb = 0;
        for (int j = 0; j < MB; ++j) nmb += (rb + tw + TW * j < t_end) ? 1 : 0;
        for (int slice = 0; slice < NS; ++slice) {
          const int64_t k0 = kbase_u4 + (NS > 1 ? (int64_t)slice * a.split_u4 : 0);
          for (int j = 0; j < MB; ++j) {
            const int64_t t0 = (int64_t)(j < nmb ? rb + tw + TW * j : rb) * 16;
            for (int lane = 0; lane < 64; ++lane) {
              if (a.nseg > 0)
                for (int q = 0; q < VPS; ++q) {
                  const int64_t off = k0 + score_key_u4<R>(t0, q, lane, last, krow_u4);
                  dry_access(a.K, (off + (int64_t)SEGC * seg_lo) * 16, 16, "score: key load");
                  dry_access(a.K, (off + (int64_t)SEGC * seg_hi) * 16, 16, "score: key load");
                }
              for (int v = pfull; v < a.ksteps; ++v) {
                const int col = SEGC * a.nseg + 4 * (v - pfull);
                const bool in = (col + (lane >> 4)) * Mma<T>::EPL < a.Lc;
                dry_access(a.K, (k0 + score_tail_u4(t0, lane, last, krow_u4, col, in)) * 16, 16, "score: key tail load");
              }
            }
          }
        }
        if constexpr (BASE == kModeSoftStats) {
          // (max, sum) of every head and query row of this wave and round
          const int heads = a.sph > 0 ? a.nseg / a.sph : 0;
          const int64_t slot = ((int64_t)b * kLdsWaves + tw) * a.rounds + rr;
          if (heads > 0 && n_q > 0)
            for (int64_t row : {(int64_t)q0, (int64_t)(heads - 1) * a.nq_total + q0 + n_q - 1})
              dry_access(a.stats_part, (((row >> 4) * a.nparts + slot) * 16 + (row & 15)) * 8, 8,
                         "score: pass-1 statistics");
          continue;
        }
        // the maxima of this wave's tiles (slice 0 of the wave group)
        for (int j = 0; j < nmb; ++j) {
          const int64_t tile = rb + tw + TW * j;
          for (int64_t tok : {tile * 16, std::min(tile * 16 + 15, n_vis - 1)}) {
            if (tok < tile * 16 || tok >= n_vis) continue;
            if (!SEQ && a.group_rows == 0) {
              dry_access(a.m, tok * 4, 4, "score: m");
              continue;
            }
            dry_range(tok, 0, a.m_stride, "score: token past the row of m");
            for (int nb = 0; nb < NB; ++nb) {
              if (nb * 16 >= n_q) break;
              const int64_t g = (q0 + nb * 16) / a.group_rows;
              dry_access(a.m, (g * a.m_stride + tok) * 4, 4, "score: m of a query");
            }
          }
        }
      }
    }
  };
  const QerStreamDesc* sd_h = nullptr;
  if constexpr (SEQ) sd_h = shadow_of(a.streams, "score: sequence table without a host copy");
  for (int blk = 0; blk < grid; ++blk) {
    const int wg = a.xcd_order ? (blk & 7) * (a.nwg >> 3) + (blk >> 3) : blk;
    dry_range(wg, 0, a.nwg, "score: workgroup share");
    const int f_begin = (int)((int64_t)a.tiles * wg / a.nwg);
    const int f_end = (int)((int64_t)a.tiles * (wg + 1) / a.nwg);
    int nr = 0;  // rounds run (pass 1: the rest are filled with empty statistics)
    if constexpr (SEQ) {
      if (!sd_h) return;
      int sidx = 0;
      while (sidx + 1 < a.n_streams && sd_h[sidx].tile0 + sd_h[sidx].ntiles <= f_begin) ++sidx;
      for (int fb = f_begin; fb < f_end && sidx < a.n_streams;) {
        dry_access(a.streams, (int64_t)sidx * sizeof(QerStreamDesc), sizeof(QerStreamDesc), "score: sequence table");
        const QerStreamDesc sd = sd_h[sidx++];
        const int s_end = sd.tile0 + sd.ntiles;
        if (s_end <= fb || sd.ntiles <= 0) continue;
        const int tb = fb - sd.tile0, te = (s_end < f_end ? s_end : f_end) - sd.tile0;
        fb = sd.tile0 + te;
        share(blk, tb, te, sd.key0 * krow_u4, sd.n_keys, sd.q0, sd.n_rows);
      }
    } else {
      share(blk, f_begin, f_end, 0, a.n_vis, a.q0, a.n_q);
      nr = (f_end - f_begin + TW * MB - 1) / (TW * MB);
    }
    if constexpr (BASE == kModeSoftStats) {
      for (int tw = 0; tw < kLdsWaves; ++tw)
        for (int rr = nr; rr < a.rounds; ++rr) {
          const int64_t slot = ((int64_t)blk * kLdsWaves + tw) * a.rounds + rr;
          if (a.H * a.n_q > 0)
            for (int64_t row : {(int64_t)a.q0, (int64_t)(a.H - 1) * a.nq_total + a.q0 + a.n_q - 1})
              dry_access(a.stats_part, (((row >> 4) * a.nparts + slot) * 16 + (row & 15)) * 8, 8,
                         "score: empty pass-1 statistics");
        }
    }
  }
}

// Address model of qer_frame_mean_kernel (grid x gy workgroups of `threads`)
void model_frame_mean(int gx, int gy, int threads, const float* m, int32_t n_vis, const int32_t* offs,
                      int32_t n_frames, const float* out_scores, const uint32_t* keys, const int32_t* nf_q,
                      const int32_t* trees, int32_t tree_ints, int32_t tree_stride, int32_t k_top,
                      const int32_t* out_idx, const QerQueryDesc* qd) {
  const int32_t* nf_h = nf_q ? shadow_of(nf_q, "frame mean: per-query frame counts without a host copy") : nullptr;
  const QerQueryDesc* qd_h = qd ? shadow_of(qd, "frame mean: query table without a host copy") : nullptr;
  if ((nf_q && !nf_h) || (qd && !qd_h)) return;
  const int64_t nfw = (int64_t)gx * (threads / 64);  // frames the grid covers
  for (int64_t g = 0; g < gy; ++g) {
    int32_t nf = nf_q ? nf_h[g] : n_frames, nfr = n_frames, nv = n_vis, frame0 = 0;
    if (nf_q) dry_access(nf_q, 4 * g, 4, "frame mean: frame count");
    if (qd) {
      dry_access(qd, g * (int64_t)sizeof(QerQueryDesc), sizeof(QerQueryDesc), "frame mean: query table");
      frame0 = qd_h[g].frame0;
      nv = qd_h[g].n_keys;
      nfr = qd_h[g].n_frames;
      nf = qd_h[g].nf;
    }
    dry_range(nv, 0, (int64_t)n_vis + 1, "frame mean: keys past the row of m");
    dry_range(nfr, 0, (int64_t)n_frames + 1, "frame mean: frames past the row of scores");
    dry_range(nf, 0, (int64_t)nfr + 1, "frame mean: prefix past the frames");
    (void)nfw;  // the waves loop over the frames with the grid's stride: every frame is covered
    const int32_t fr = nfr;
    if (fr > 0) {
      dry_access(out_scores, (g * n_frames) * 4, 4 * (int64_t)fr, "frame mean: scores");
      dry_access(keys, (g * n_frames) * 4, 4 * (int64_t)fr, "frame mean: sort keys");
    }
    const int32_t nread = std::min(nf, fr);  // frames whose tokens are read
    if (nread > 0) {
      dry_access(offs, 4 * (int64_t)frame0, 4 * ((int64_t)nread + 1), "frame mean: frame offsets");
      if (nv > 0) dry_access(m, (g * n_vis) * 4, 4 * (int64_t)nv, "frame mean: m");
    }
    if (k_top > 0 && nf > 0) dry_access(keys, (g * n_frames) * 4, 4 * (int64_t)std::min(nf, fr), "frame mean: top-k keys");
    if (trees) {
      const int32_t G = arrive_fan(gx);
      dry_range((int64_t)G * tree_stride, 0, tree_ints, "frame mean: arrival tree");
      dry_access(trees, (g * tree_ints) * 4, ((int64_t)G * tree_stride + 1) * 4, "frame mean: arrival tree");
      if (k_top > 0) dry_access(out_idx, (g * k_top) * 4, 4 * (int64_t)k_top, "frame mean: top-k");
    }
  }
}

// qer_frame_mean_kernel on grid (gx, gy) of `threads` (its model in a dry run)
int launch_frame_mean(int gx, int gy, int threads, hipStream_t s, const float* m, int32_t n_vis, const int32_t* offs,
                      int32_t n_frames, float* out_scores, uint32_t* keys, const int32_t* nf_q, int32_t* trees,
                      int32_t tree_ints, int32_t tree_stride, int32_t k_top, int32_t* out_idx, const QerQueryDesc* qd) {
  if (dry_run()) {
    if (gx > 0 && gy > 0)
      model_frame_mean(gx, gy, threads, m, n_vis, offs, n_frames, out_scores, keys, nf_q, trees, tree_ints,
                       tree_stride, k_top, out_idx, qd);
    return COFIE_OK;
  }
  return launch("qer_frame_mean", qer_frame_mean_kernel, dim3((unsigned)gx, (unsigned)gy), dim3((unsigned)threads), 0,
                s, m, n_vis, offs, n_frames, out_scores, keys, nf_q, trees, tree_ints, tree_stride, k_top, out_idx, qd);
}

template <typename T, int MB, int NB, int P, int NS, int MODE>
int launch_lds_t(const ScoreLdsArgs& sa, const LdsPlan& L, size_t lds, hipStream_t s) {
  auto k = qer_score_kernel<T, MB, NB, P, NS, MODE>;
  int rc = allow_lds(k, lds);
  if (rc) return rc;
  if (dry_run()) {
    dry_range((int64_t)lds, 0, 160 * 1024 + 1, "score: LDS beyond a CU's 160 KiB");
    if (L.nwg > 0) model_score<T, MB, NB, P, NS, MODE>(sa, L.nwg, lds);
    return COFIE_OK;
  }
  const int base = MODE & 3;
  const char* name = base == kModeLogit ? "qer_score" : (base == kModeSoftStats ? "qer_soft_stats" : "qer_soft_score");
  return launch(name, k, dim3((unsigned)L.nwg), dim3(kLdsThreads), lds, s, sa);
}

template <typename T, int MB, int P, int NS, int MODE>
int launch_lds_nb(const ScoreLdsArgs& sa, const LdsPlan& L, int NB, size_t lds, hipStream_t s) {
  // 128 query rows in one pass: one query term, one tile per wave (two
  // spill), no contraction split (LOGIT, and both SOFTMAX passes)
  if constexpr (MB == 1 && P == 1 && NS == 1) {
    if (NB == 8) return launch_lds_t<T, 1, 8, 1, NS, MODE>(sa, L, lds, s);
  }
  switch (NB) {
    case 1: return launch_lds_t<T, MB, 1, P, NS, MODE>(sa, L, lds, s);
    case 2: return launch_lds_t<T, MB, 2, P, NS, MODE>(sa, L, lds, s);
    case 3: return launch_lds_t<T, MB, 3, P, NS, MODE>(sa, L, lds, s);
    default: return launch_lds_t<T, MB, 4, P, NS, MODE>(sa, L, lds, s);
  }
}

// lds = 0: the plan's (the phase buffers and the slices' accumulators)
template <typename T, int P, int MODE = kModeLogit>
int launch_lds(const ScoreLdsArgs& sa, const LdsPlan& L, int NB, hipStream_t s, size_t lds = 0) {
  if (!lds) lds = L.lds;
  if constexpr (P == 1 && MODE == kModeLogit) {
    if (L.NS == 4) return launch_lds_nb<T, 1, P, 4, MODE>(sa, L, NB, lds, s);
    if (L.NS == 2) return launch_lds_nb<T, 1, P, 2, MODE>(sa, L, NB, lds, s);
  }
  return L.MB == 1 ? launch_lds_nb<T, 1, P, 1, MODE>(sa, L, NB, lds, s)
                   : launch_lds_nb<T, 2, P, 1, MODE>(sa, L, NB, lds, s);
}

// SOFTMAX through the score kernel: the LDS of a pass (phase buffers, pass 2's
// statistics [H][nq] of its query chunk, the segment map for grouped heads)
// and the pass-1 statistics per row (one per wave and round).
size_t soft_lds(const LdsPlan& L, int mode, int H, int nq_chunk, int G, int64_t nseg) {
  size_t b = L.lds;
  if (mode == kModeSoftProb) b += (size_t)H * nq_chunk * sizeof(float2);
  if (G > 1) b += (size_t)nseg * sizeof(int32_t);
  return b;
}
int64_t soft_rounds(const LdsPlan& L, int64_t n_vis) {
  const int64_t tiles = ceil_div(n_vis, 16);
  return ceil_div(ceil_div(tiles, L.nwg), (int64_t)kLdsWaves * L.MB);
}
constexpr size_t kLdsMax = 160 * 1024;

// SOFTMAX through qer_soft_grp_kernel: bf16 grouped heads of d = 128 with an
// instance for their shape, one query
bool soft_grp_ok(const cofie_qer_desc& h, int32_t n_queries) {
  return h.score_mode == COFIE_SCORE_SOFTMAX && h.dtype == COFIE_BF16 && h.d == 128 && n_queries == 1 &&
         h.n_vis > 0 && h.H_q % h.H_kv == 0 && grp_has_instance(h.H_kv, h.H_q / h.H_kv);
}
int grp_blocks(int32_t n_q) { return (n_q + 15) / 16; }
// key ranges of a pass whose workgroups are `per` per range: a multiple of 8
// (whole XCD groups), at most one workgroup per CU
int grp_ranges(int per, int cus) { return 8 * std::max(1, cus / (8 * per)); }
// pass 1: per range, one workgroup per key head and set of row blocks
int grp_ranges1(const cofie_qer_desc& h, int cus) {
  const int nb = grp_blocks(h.n_q), nbw = grp_nbw(h.H_q / h.H_kv, nb);
  return grp_ranges(h.H_kv * ((nb + nbw - 1) / nbw), cus);
}

// Whether SOFTMAX takes the score kernel (each head whole 128-byte segments
// of a key row, the widest query chunk's LDS within the CU's), and its
// pass-1 statistics count.
void plan_soft(const cofie_qer_desc& h, int32_t n_queries, QerPlan& p) {
  p.soft_fast = p.soft_wide = p.soft_grp = false;
  p.soft_nwg = p.soft_rounds = 0;
  if (h.score_mode != COFIE_SCORE_SOFTMAX || h.n_vis <= 0) return;
  if (soft_grp_ok(h, n_queries)) {
    p.soft_grp = true;
    p.soft_nwg = grp_ranges1(h, device_cu_count());  // pass 1's key ranges: the partial statistics
    p.soft_rounds = 1;
    return;
  }
  const int64_t seg_el = (1024 / lds_rows(1, 1)) / (int64_t)p.esize;
  if (h.d % seg_el != 0) return;
  const int cus = device_cu_count();
  const int64_t rows = (int64_t)h.n_q * n_queries;
  // 128 query rows per pass (K read twice for up to 128 stacked rows) where
  // the plan takes one tile per wave and the LDS holds the pass-2 statistics
  // of 128 rows; else 64
  p.soft_wide = false;
  if (rows > 64) {
    const LdsPlan W = plan_score_lds(h.n_vis, p.Lc, p.esize, 1, 8, cus, false);
    p.soft_wide = W.MB == 1 && soft_lds(W, kModeSoftProb, h.H_q, 128, h.H_q / h.H_kv, p.Lc / seg_el) <= kLdsMax;
  }
  const int nq = (int)std::min<int64_t>(p.soft_wide ? 128 : 64, rows), NB = nq > 64 ? 8 : (nq + 15) / 16;
  const LdsPlan L = plan_score_lds(h.n_vis, p.Lc, p.esize, 1, NB, cus, false);
  if (soft_lds(L, kModeSoftProb, h.H_q, nq, h.H_q / h.H_kv, p.Lc / seg_el) > kLdsMax) return;
  p.soft_fast = true;
  p.soft_nwg = L.nwg;
  p.soft_rounds = soft_rounds(L, h.n_vis);
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

// QER for n_queries queries of h.n_q rows each sharing K (one query: the
// single-query path); query g covers its first nf_host[g] frames.
int rank_impl(const void* Q, const void* K, const int32_t* frame_offsets, const cofie_qer_desc& h,
              int32_t n_queries, const int32_t* nf_host, int32_t k_top, float* out_scores, int32_t* out_idx,
              hipStream_t s) {
  int rc;
  const bool multi = n_queries > 1;
  const int32_t R = n_queries * h.n_q;  // query rows
  const QerPlan p = plan_qer(h, n_queries);
  Arena plan;
  carve_qer(plan, h, p, n_queries);
  Scratch scratch;
  rc = scratch.acquire(h.workspace, h.workspace_bytes, plan.bytes(), s);
  if (rc) return rc;
  Arena ar;
  ar.base = scratch.ptr();
  QerScratch w = carve_qer(ar, h, p, n_queries);
  if (multi) {
    rc = copy_to_device(w.nf, nf_host, n_queries * sizeof(int32_t), s, "the per-query frame counts");
    if (rc) return rc;
  }
  const bool bf16 = h.dtype == COFIE_BF16;
  const float base_scale = h.scale > 0.f ? h.scale : (float)(1.0 / std::sqrt((double)h.d));
  // the top-k runs in the frame-mean kernel's last workgroup when the score
  // kernel (launched first) clears its arrival counters
  const bool fused_tail =
      (h.score_mode == COFIE_SCORE_LOGIT || p.soft_fast || p.soft_grp) && h.n_vis > 0 && h.n_frames > 0 && k_top > 0;

  if (h.n_vis > 0) {
    if (h.score_mode == COFIE_SCORE_LOGIT) {
      const uint8_t* qp = static_cast<const uint8_t*>(Q);
      if (p.fold) {
        const int64_t total = (int64_t)R * p.Lc;
        const unsigned grid = (unsigned)std::min<int64_t>(ceil_div(total, 256), 8192);
        rc = bf16 ? launch("qer_fold", qer_fold_kernel<bf16_t>, dim3(grid), dim3(256), 0, s,
                           static_cast<const bf16_t*>(Q), R, h.H_q, h.H_kv, h.d, (void*)w.qp)
                  : launch("qer_fold", qer_fold_kernel<float>, dim3(grid), dim3(256), 0, s,
                           static_cast<const float*>(Q), R, h.H_q, h.H_kv, h.d, (void*)w.qp);
        if (rc) return rc;
        qp = w.qp;
      }
      ScoreLdsArgs sa{};
      sa.K = static_cast<const uint8_t*>(K);
      sa.Qp = qp;
      sa.n_vis = h.n_vis;
      sa.nq_total = R;
      sa.group_rows = multi ? h.n_q : 0;
      sa.m_stride = h.n_vis;
      sa.Lc = (int32_t)p.Lc;
      sa.tiles = (int32_t)ceil_div(h.n_vis, 16);
      sa.scale = (float)((double)base_scale / (double)h.H_q);
      sa.m = w.m;
      sa.nclear = n_queries * qer_trees(h.n_frames, n_queries).ints;
      const int cus = device_cu_count();
      // query rows per pass over K: 64, or 128 (eight 16-row blocks) where the
      // plan gives one tile per wave, no contraction split (its LDS would not
      // fit; the split, which decides the summation order, stays a function of
      // the keys alone) and one query term, so that K is read once for up to
      // 128 rows (several queries of a stream)
      const LdsPlan probe = plan_score_lds(h.n_vis, p.Lc, p.esize, p.P, 4, cus, true);
      const bool wide = p.P == 1 && R > 64 && probe.MB == 1 && probe.NS == 1;
      const int chunk = wide ? 128 : 64;
      for (int q0 = 0; q0 < R; q0 += chunk) {
        sa.clear = (q0 == 0 && fused_tail) ? w.done : nullptr;
        sa.q0 = q0;
        sa.n_q = std::min(chunk, R - q0);
        sa.accumulate = q0 > 0;
        const int NB = sa.n_q > 64 ? 8 : (sa.n_q + 15) / 16;
        const LdsPlan L = plan_score_lds(h.n_vis, p.Lc, p.esize, p.P, p.P * NB, cus, true);
        sa.nseg = L.nseg;
        sa.ksteps = L.ksteps;
        sa.S = L.S;
        sa.lgS = L.lgS;
        sa.nphase = L.nphase;
        sa.nwg = L.nwg;
        sa.split_u4 = L.split_u4;
        sa.k_row_u4 = (int32_t)(p.Lc * (int64_t)p.esize / 16);
        if (bf16)
          rc = p.P == 3 ? launch_lds<bf16_t, 3>(sa, L, NB, s) : launch_lds<bf16_t, 1>(sa, L, NB, s);
        else
          rc = launch_lds<float, 1>(sa, L, NB, s);
        if (rc) return rc;
      }
    } else if (p.soft_grp) {
      // grouped heads: per-head statistics, their merge over the key ranges,
      // then the probabilities
      SoftGrpArgs ga{};
      ga.K = static_cast<const uint4*>(K);
      ga.Q = static_cast<const uint4*>(Q);
      ga.n_vis = h.n_vis;
      ga.n_q = h.n_q;
      ga.tiles = ceil_div(h.n_vis, 16);
      ga.nb = grp_blocks(h.n_q);
      ga.ranges = grp_ranges(ga.nb, device_cu_count());
      ga.ranges1 = (int32_t)p.soft_nwg;
      ga.nbw = grp_nbw(h.H_q / h.H_kv, ga.nb);
      ga.nbs = (ga.nb + ga.nbw - 1) / ga.nbw;
      ga.c2 = (float)((double)base_scale * 1.4426950408889634);
      ga.inv_h = 1.0f / (float)h.H_q;
      ga.stats_part = w.partial;
      ga.stats = w.stats;
      ga.m = w.m;
      ga.clear = fused_tail ? w.done : nullptr;
      ga.nclear = qer_trees(h.n_frames, 1).ints;
      ga.q_gstride = (h.H_q / h.H_kv) * 256;
      rc = launch_grp(ga, h.H_kv, h.H_q / h.H_kv, 1, s);
      if (rc) return rc;
      const int32_t rows = h.H_q * h.n_q;
      rc = launch("qer_soft_merge", qer_soft_merge_blocked_kernel, dim3((unsigned)ceil_div(rows, 16)), dim3(1024), 0,
                  s, (const float2*)w.partial, p.soft_nwg, rows, w.stats);
      if (rc) return rc;
      rc = launch_grp(ga, h.H_kv, h.H_q / h.H_kv, 2, s);
      if (rc) return rc;
    } else if (p.soft_fast) {
      // two passes of the score kernel over K (per-head statistics, then the
      // probabilities), the statistics merged in between
      ScoreLdsArgs sa{};
      sa.K = static_cast<const uint8_t*>(K);
      sa.Qp = static_cast<const uint8_t*>(Q);
      sa.n_vis = h.n_vis;
      sa.nq_total = R;  // several queries: their rows stacked, statistics per row
      sa.group_rows = multi ? h.n_q : 0;
      sa.soft_offs = multi ? frame_offsets : nullptr;
      sa.soft_nf = multi ? w.nf : nullptr;
      sa.m_stride = h.n_vis;
      sa.Lc = (int32_t)p.Lc;
      sa.tiles = (int32_t)ceil_div(h.n_vis, 16);
      sa.m = w.m;
      sa.k_row_u4 = (int32_t)((int64_t)h.H_kv * h.d * (int64_t)p.esize / 16);
      const int64_t seg_el = (1024 / lds_rows(1, 1)) / (int64_t)p.esize;
      sa.sph = (int32_t)(h.d / seg_el);
      sa.H = h.H_q;
      sa.G = h.H_q / h.H_kv;
      sa.soft_scale = base_scale;
      sa.stats_part = w.partial;
      sa.stats = w.stats;
      sa.nclear = n_queries * qer_trees(h.n_frames, n_queries).ints;
      const int cus = device_cu_count();
      const int chunk = p.soft_wide ? 128 : 64;
      for (int pass = 1; pass <= 2; ++pass) {
        for (int q0 = 0; q0 < R; q0 += chunk) {
          sa.q0 = q0;
          sa.n_q = std::min(chunk, R - q0);
          sa.accumulate = pass == 2 && q0 > 0;
          sa.clear = (pass == 2 && q0 == 0 && fused_tail) ? w.done : nullptr;
          sa.scale = 1.0f / (float)h.H_q;  // pass 2: the head mean
          const int NB = sa.n_q > 64 ? 8 : (sa.n_q + 15) / 16;
          const LdsPlan L = plan_score_lds(h.n_vis, p.Lc, p.esize, 1, NB, cus, false);
          sa.nseg = L.nseg;
          sa.ksteps = L.ksteps;
          sa.S = L.S;
          sa.lgS = L.lgS;
          sa.nphase = L.nphase;
          sa.nwg = L.nwg;
          sa.split_u4 = L.split_u4;
          sa.rounds = (int32_t)soft_rounds(L, h.n_vis);
          sa.nparts = (int32_t)(p.soft_nwg * kLdsWaves * p.soft_rounds);
          if (L.nwg != p.soft_nwg || sa.rounds != p.soft_rounds)  // the scratch was sized for that plan
            return set_error(COFIE_EHIP, "SOFTMAX plan mismatch (%d x %d against %lld x %lld)", L.nwg, sa.rounds,
                             (long long)p.soft_nwg, (long long)p.soft_rounds);
          const int mode = pass == 1 ? kModeSoftStats : kModeSoftProb;
          const size_t lds = soft_lds(L, mode, h.H_q, sa.n_q, sa.G, L.nseg);
          const bool gqa = sa.G > 1;
          if (pass == 1 && !gqa)
            rc = bf16 ? launch_lds<bf16_t, 1, kModeSoftStats>(sa, L, NB, s, lds)
                      : launch_lds<float, 1, kModeSoftStats>(sa, L, NB, s, lds);
          else if (pass == 1)
            rc = bf16 ? launch_lds<bf16_t, 1, kModeSoftStats | kModeGqa>(sa, L, NB, s, lds)
                      : launch_lds<float, 1, kModeSoftStats | kModeGqa>(sa, L, NB, s, lds);
          else if (!gqa)
            rc = bf16 ? launch_lds<bf16_t, 1, kModeSoftProb>(sa, L, NB, s, lds)
                      : launch_lds<float, 1, kModeSoftProb>(sa, L, NB, s, lds);
          else
            rc = bf16 ? launch_lds<bf16_t, 1, kModeSoftProb | kModeGqa>(sa, L, NB, s, lds)
                      : launch_lds<float, 1, kModeSoftProb | kModeGqa>(sa, L, NB, s, lds);
          if (rc) return rc;
        }
        if (pass == 1) {
          const int32_t rows = h.H_q * R;
          rc = launch("qer_soft_merge", qer_soft_merge_blocked_kernel, dim3((unsigned)ceil_div(rows, 16)),
                      dim3(1024), 0, s, (const float2*)w.partial, p.soft_nwg * kLdsWaves * p.soft_rounds, rows,
                      w.stats);
          if (rc) return rc;
        }
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
      rc = launch("qer_soft_merge", qer_soft_merge_kernel, dim3((unsigned)ceil_div(rows, 4)), dim3(256), 0, s,
                  (const float2*)w.partial, p.nblk_soft, (int64_t)rows, (int64_t)1, rows, w.stats);
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
  if (fused_tail) {
    const QerTrees tr = qer_trees(h.n_frames, n_queries);
    return launch_frame_mean(tr.nwg, n_queries, 1024, s,
                  (const float*)w.m, h.n_vis, frame_offsets, h.n_frames, out_scores, w.keys, (const int32_t*)w.nf,
                  w.done, tr.ints, tr.stride, k_top, out_idx, (const QerQueryDesc*)nullptr);
  }
  if (h.n_frames > 0) {
    rc = launch_frame_mean(ceil_div(h.n_frames, 4), n_queries, 256, s, (const float*)w.m, h.n_vis, frame_offsets,
                           h.n_frames, out_scores, w.keys, (const int32_t*)w.nf, (int32_t*)nullptr, 0, 0, k_top,
                           out_idx, (const QerQueryDesc*)nullptr);
    if (rc) return rc;
  }
  if (k_top == 0) return COFIE_OK;
  return launch("qer_topk", qer_topk_kernel, dim3(n_queries), dim3(1024), 0, s, (const uint32_t*)w.keys,
                h.n_frames, k_top, out_idx, (const int32_t*)w.nf);
}

// ---- several key sequences in one launch (cofie_qer_rank_streams) -------------------
// The sequences' stacked query rows are cut into chunks of whole queries, at
// most 128 rows (64 with the three query terms of a folded grouped-query
// contraction), each chunk a QerStreamDesc that reads its sequence's keys;
// every query gets a QerQueryDesc for the frame means.  Both tables are
// copied to the device with one copy per call.
struct StreamsPlan {
  std::vector<QerStreamDesc> seq;
  std::vector<QerQueryDesc> qry;
  int64_t max_keys = 0;    // row stride of m
  int32_t max_frames = 0;  // row stride of the scores and their sort keys
  int64_t tiles = 0;       // over all chunks
  int NB = 1;              // 16-row blocks of the widest chunk (1-4, or 8)
  int32_t n_queries = 0;
};

int plan_streams(const cofie_qer_desc& h, const QerPlan& p, int32_t n_streams, const int64_t* stream_keys,
                 const int32_t* stream_frames, const int32_t* stream_queries, const int32_t* nf, StreamsPlan& sp) {
  if (n_streams < 1) return set_error(COFIE_EINVAL, "n_streams = %d must be >= 1", n_streams);
  if (!stream_keys || !stream_frames || !stream_queries)
    return set_error(COFIE_EINVAL, "stream_keys, stream_frames and stream_queries must not be NULL");
  if (stream_keys[0] != 0 || stream_frames[0] != 0 || stream_queries[0] != 0)
    return set_error(COFIE_EINVAL, "stream_keys, stream_frames and stream_queries must start at 0");
  if (stream_keys[n_streams] != h.n_vis || stream_frames[n_streams] != h.n_frames)
    return set_error(COFIE_EINVAL, "stream_keys[n_streams] = %lld and stream_frames[n_streams] = %d must equal "
                     "n_vis = %d and n_frames = %d", (long long)stream_keys[n_streams], stream_frames[n_streams],
                     h.n_vis, h.n_frames);
  if (h.score_mode != COFIE_SCORE_LOGIT)
    return set_error(COFIE_EUNSUPPORTED, "several key sequences are ranked in LOGIT mode only");
  const int rows_max = p.P == 1 ? 128 : 64;
  if (h.n_q % 16 != 0 || h.n_q > rows_max)
    return set_error(COFIE_EUNSUPPORTED, "several key sequences need n_q (%d) a multiple of 16 and at most %d",
                     h.n_q, rows_max);
  const int32_t nq = stream_queries[n_streams];
  if (nq < 1) return set_error(COFIE_EINVAL, "no queries");
  if (!nf) return set_error(COFIE_EINVAL, "n_frames_per_query is NULL");
  if ((int64_t)nq * h.n_q * h.H_q * h.d >= (int64_t(1) << 31)) return set_error(COFIE_EUNSUPPORTED, "queries too large");
  const int32_t per_chunk = rows_max / h.n_q;  // queries per chunk
  sp = StreamsPlan();
  sp.n_queries = nq;
  int widest = 0;
  for (int32_t st = 0; st < n_streams; ++st) {
    const int64_t k0 = stream_keys[st], nk = stream_keys[st + 1] - k0;
    const int32_t f0 = stream_frames[st], nfr = stream_frames[st + 1] - f0;
    const int32_t g0 = stream_queries[st], ng = stream_queries[st + 1] - g0;
    if (nk < 0 || nfr < 0 || ng < 0) return set_error(COFIE_EINVAL, "sequence %d: decreasing stream arrays", st);
    if (nk >= (int64_t(1) << 31) - 16) return set_error(COFIE_EUNSUPPORTED, "sequence %d: too many keys", st);
    sp.max_keys = std::max(sp.max_keys, nk);
    sp.max_frames = std::max(sp.max_frames, nfr);
    for (int32_t g = g0; g < g0 + ng; ++g) {
      if (nf[g] < 0 || nf[g] > nfr)
        return set_error(COFIE_EINVAL, "query %d: %d frames outside [0, %d] (its sequence's frames)", g, nf[g], nfr);
      sp.qry.push_back(QerQueryDesc{k0, (int32_t)nk, f0, nfr, nf[g]});
    }
    const int32_t nt = (int32_t)ceil_div(nk, 16);
    for (int32_t c = 0; c < ng && nt > 0; c += per_chunk) {
      const int32_t cg = std::min(per_chunk, ng - c);
      if (sp.tiles + nt >= (int64_t(1) << 31)) return set_error(COFIE_EUNSUPPORTED, "too many tiles");
      sp.seq.push_back(QerStreamDesc{k0, (int32_t)nk, (int32_t)sp.tiles, nt, (g0 + c) * h.n_q, cg * h.n_q, 0});
      sp.tiles += nt;
      widest = std::max(widest, cg * h.n_q);
    }
  }
  const int nb = (widest + 15) / 16;
  sp.NB = nb > 4 ? 8 : (nb < 1 ? 1 : nb);
  return COFIE_OK;
}

// qer_seq_kernel's shape: virtual steps per batch, key rows per load
constexpr int kSeqU = 2;
constexpr int kSeqR = 8;
constexpr int kSeqSegBytes = 1024 / kSeqR;  // a segment of a key row (16 / kSeqR virtual steps)

// Whether the chunks take qer_seq_kernel: bf16 heads of one query term, a
// chunk wider than 64 rows, key rows of whole segments, at least two phases
// per round.
bool seq_fast(const cofie_qer_desc& h, const QerPlan& p, const StreamsPlan& sp) {
  const int64_t row_bytes = p.Lc * (int64_t)p.esize, ksteps = row_bytes / 64;
  return h.dtype == COFIE_BF16 && p.P == 1 && sp.NB == 8 && row_bytes % kSeqSegBytes == 0 &&
         ksteps % kSeqS == 0 && ksteps >= 2 * kSeqS &&
         sp.max_keys * (row_bytes / 16) < (int64_t(1) << 31);  // 32-bit key offsets within a sequence
}

// qer_seq_kernel's workgroups: one per CU (whole XCD groups), at most one per
// round of 16 tiles
int seq_nwg(const StreamsPlan& sp, int cus) {
  int n = (int)std::min<int64_t>(cus, ceil_div(sp.tiles, (int64_t)kLdsWaves * 2));
  if (n >= 8) n &= ~7;
  return std::max(n, 1);
}
// the most chunks one workgroup's share of the tiles reaches
int seq_span(const StreamsPlan& sp, int nwg) {
  int worst = 0;
  size_t c = 0;
  for (int b = 0; b < nwg; ++b) {
    const int64_t fb = sp.tiles * b / nwg, fe = sp.tiles * (b + 1) / nwg;
    while (c + 1 < sp.seq.size() && sp.seq[c].tile0 + sp.seq[c].ntiles <= fb) ++c;
    size_t e = c;
    while (e < sp.seq.size() && sp.seq[e].tile0 < fe) ++e;
    worst = std::max(worst, (int)(e - c));
  }
  return worst;
}

struct StreamsScratch {
  float* m;           // [n_queries][max_keys]
  uint32_t* keys;     // [n_queries][max_frames]
  uint8_t* qp;        // folded queries (grouped heads)
  uint4* qop;         // operand-order query fragments of each chunk (qer_seq_kernel)
  uint8_t* meta;      // QerStreamDesc[seq] then QerQueryDesc[n_queries]
  int32_t* done;      // [n_queries][tree ints] arrival trees of the frame-mean kernel
};

size_t meta_bytes(const StreamsPlan& sp) {
  return sp.seq.size() * sizeof(QerStreamDesc) + sp.qry.size() * sizeof(QerQueryDesc);
}

StreamsScratch carve_streams(Arena& ar, const cofie_qer_desc& h, const QerPlan& p, const StreamsPlan& sp) {
  StreamsScratch w;
  w.m = ar.take<float>((size_t)sp.n_queries * std::max<int64_t>(sp.max_keys, 1));
  w.keys = ar.take<uint32_t>((size_t)sp.n_queries * std::max(sp.max_frames, 1));
  w.qp = p.fold ? ar.take<uint8_t>((size_t)p.P * sp.n_queries * h.n_q * p.Lc * p.esize) : nullptr;
  w.qop = seq_fast(h, p, sp) ? ar.take<uint4>(sp.seq.size() * (size_t)(p.Lc * p.esize / 64) * kSeqNB * 64) : nullptr;
  w.meta = ar.take<uint8_t>(meta_bytes(sp));
  w.done = ar.take<int32_t>((size_t)sp.n_queries * qer_trees(std::max(sp.max_frames, 1), sp.n_queries).ints);
  return w;
}

constexpr int kSeqLogit = kModeLogit | kModeSeq;

// Address model of qer_qop_kernel: every element of the copy
void model_qop(const uint4* Q, int64_t row_u4, const QerStreamDesc* seq, int32_t n_seq, int32_t ksteps, int32_t R,
               const uint4* out) {
  const QerStreamDesc* sd_h = shadow_of(seq, "qop: sequence table without a host copy");
  if (!sd_h) return;
  const int64_t per = (int64_t)ksteps * kSeqNB * 64;
  for (int32_t c = 0; c < n_seq; ++c) {
    dry_access(seq, (int64_t)c * sizeof(QerStreamDesc), sizeof(QerStreamDesc), "qop: sequence table");
    dry_access(out, (int64_t)c * per * 16, per * 16, "qop: copy");
    for (int64_t r = 0; r < per; ++r) {
      int row, col;
      qop_source(r, R, row, col);
      dry_range(col, 0, row_u4, "qop: column past the query row");
      if (row < sd_h[c].n_rows) dry_access(Q, ((int64_t)(sd_h[c].q0 + row) * row_u4 + col) * 16, 16, "qop: query load");
    }
  }
}

// Address model of qer_seq_kernel<U, R> (grid a.nwg, `lds` bytes of LDS): the
// round sequence of every workgroup as the kernel walks it, its key loads at
// both ends of each round's segments, its query-fragment copies and LDS
// traffic, and its stores of m.
template <int U, int R>
void model_seq(const SeqArgs& a, size_t lds) {
  constexpr int MB = 2, NB = kSeqNB, TW = kLdsWaves;
  constexpr int VPS = 16 / R, SEGC = 64 / R;
  constexpr int BPP = kSeqS / U;
  constexpr int CP = kSeqPhaseU4 / kLdsThreads / BPP;
  const int64_t L = (int64_t)lds;
  const int ksteps = VPS * a.nseg, bpr = ksteps / U, nph = ksteps / kSeqS;
  dry_range(nph, 2, INT32_MAX, "seq: a round needs two phases");
  dry_range(ksteps % kSeqS, 0, 1, "seq: whole phases per round");
  if (a.xcd_order) dry_range(a.nwg % 8, 0, 1, "seq: XCD order needs whole groups of 8 workgroups");
  if (a.clear && a.nclear > 0) dry_access(a.clear, 0, 4 * (int64_t)a.nclear, "seq: arrival counters");
  const QerStreamDesc* seq = shadow_of(a.seq, "seq: sequence table without a host copy");
  if (!seq) return;
  // LDS: the two phase buffers, then the table
  for (int bp = 0; bp < BPP; ++bp) {
    const int64_t hi = (int64_t)bp * CP * kLdsThreads + (CP - 1) * kLdsThreads + kLdsThreads - 1;
    dry_range(hi, 0, kSeqPhaseU4, "seq: query slice past its phase buffer");
    const int64_t rd = (int64_t)bp * U * NB * 64 + ((U - 1) * NB + NB - 1) * 64 + 63;
    dry_range(rd, 0, kSeqPhaseU4, "seq: fragment read past its phase buffer");
    dry_lds((kSeqPhaseU4 + rd) * 16, 16, L, "seq: fragment read");
  }
  dry_lds(2 * (int64_t)kSeqPhaseU4 * 16, kSeqTab * (int64_t)sizeof(QerStreamDesc), L, "seq: chunk table");
  auto q_src = [&](int si, int ph) { return ((int64_t)si * ksteps + (int64_t)ph * kSeqS) * NB * 64; };
  struct Rnd {
    int sidx, tb, te;
  };
  for (int blk = 0; blk < a.nwg; ++blk) {
    const int wg = a.xcd_order ? (blk & 7) * (a.nwg >> 3) + (blk >> 3) : blk;
    const int f_begin = (int)((int64_t)a.tiles * wg / a.nwg);
    const int f_end = (int)((int64_t)a.tiles * (wg + 1) / a.nwg);
    int sidx0 = 0;
    while (sidx0 + 1 < a.n_seq && seq[sidx0].tile0 + seq[sidx0].ntiles <= f_begin) ++sidx0;
    const int tab_end = std::min(sidx0 + kSeqTab, a.n_seq);
    dry_access(a.seq, (int64_t)sidx0 * sizeof(QerStreamDesc), (int64_t)(tab_end - sidx0) * sizeof(QerStreamDesc),
               "seq: chunk table load");
    auto first_of = [&](int si, int from) {
      Rnd r{-1, 0, 0};
      for (; si < tab_end; ++si) {
        const QerStreamDesc sd = seq[si];
        const int s_end = sd.tile0 + sd.ntiles;
        if (sd.ntiles <= 0 || s_end <= from) continue;
        if (sd.tile0 >= f_end) break;
        r = Rnd{si, std::max(from, sd.tile0) - sd.tile0, std::min(s_end, f_end) - sd.tile0};
        break;
      }
      return r;
    };
    auto next_of = [&](const Rnd& r) {
      if (r.tb + TW * MB < r.te) return Rnd{r.sidx, r.tb + TW * MB, r.te};
      return first_of(r.sidx + 1, seq[r.sidx].tile0 + r.te);
    };
    // a round's key offsets, lane by lane, at its first and last segment
    auto keys = [&](const Rnd& r) {
      const QerStreamDesc sd = seq[r.sidx];
      const int64_t base = sd.key0 * a.k_row_u4;
      for (int wave = 0; wave < TW; ++wave) {
        int nmb = 0;
        for (int j = 0; j < MB; ++j) nmb += (r.tb + wave + TW * j < r.te) ? 1 : 0;
        for (int j = 0; j < MB; ++j) {
          const int t = j < nmb ? r.tb + wave + TW * j : r.tb;
          for (int lane = 0; lane < 64; ++lane)
            for (int q = 0; q < VPS; ++q) {
              const int32_t off = seq_key_off<R>(t, q, lane, sd.n_keys - 1, a.k_row_u4);
              dry_range(off, 0, (int64_t)sd.n_keys * a.k_row_u4, "seq: key offset outside its sequence");
              dry_access(a.K, (base + off) * 16, 16, "seq: key load");
              dry_access(a.K, (base + off + (int64_t)SEGC * (a.nseg - 1)) * 16, 16, "seq: key load");
            }
        }
      }
    };
    Rnd cur = first_of(sidx0, f_begin);
    if (cur.sidx < 0) continue;
    Rnd nxt = next_of(cur);
    keys(cur);
    dry_access(a.Qop, q_src(cur.sidx, 0) * 16, (int64_t)kSeqPhaseU4 * 16, "seq: first phase");
    auto phase_src = [&](int pir) {
      const bool next = pir >= nph;
      const int si = next && nxt.sidx >= 0 ? nxt.sidx : cur.sidx;
      dry_range(next ? pir - nph : pir, 0, nph, "seq: phase past its chunk");
      return q_src(si, next ? pir - nph : pir);
    };
    dry_access(a.Qop, phase_src(1) * 16, 2 * (int64_t)CP * kLdsThreads * 16, "seq: query slices");
    while (cur.sidx >= 0) {
      dry_range(cur.sidx - sidx0, 0, kSeqTab, "seq: chunk past the LDS table");
      for (int ph = 0; ph < nph; ++ph)
        for (int bp = 0; bp < BPP; ++bp) {
          const bool wrap = bp + 2 >= BPP;
          const int64_t src = phase_src(ph + (wrap ? 2 : 1)) + (int64_t)(wrap ? bp + 2 - BPP : bp + 2) * CP * kLdsThreads;
          dry_access(a.Qop, src * 16, (int64_t)CP * kLdsThreads * 16, "seq: query slice");
          const int ahead = BPP * ph + bp + 3;
          const int ms = (ahead >= bpr ? ahead - bpr : ahead) * U;
          dry_range(ms / VPS, 0, a.nseg, "seq: key segment");
          dry_range(ms / VPS + U / VPS - 1, 0, a.nseg, "seq: key segment");
        }
      const QerStreamDesc sd = seq[cur.sidx];
      for (int wave = 0; wave < TW; ++wave)
        for (int j = 0; j < MB; ++j) {
          const int tile = cur.tb + wave + TW * j;
          if (tile >= cur.te) continue;
          for (int tok : {tile * 16, std::min(tile * 16 + 15, sd.n_keys - 1)}) {
            if (tok < tile * 16 || tok >= sd.n_keys) continue;
            dry_range(tok, 0, a.m_stride, "seq: token past the row of m");
            for (int nb = 0; nb < NB && nb * 16 < sd.n_rows; ++nb) {
              const int64_t g = (sd.q0 + nb * 16) / a.group_rows;
              dry_access(a.m, (g * a.m_stride + tok) * 4, 4, "seq: m of a query");
            }
          }
        }
      cur = nxt;
      if (cur.sidx >= 0) {
        keys(cur);
        nxt = next_of(cur);
      }
    }
  }
}



int rank_streams_impl(const void* Q, const void* K, const int32_t* frame_offsets, const cofie_qer_desc& h,
                      const QerPlan& p, const StreamsPlan& sp, int32_t k_top, float* out_scores, int32_t* out_idx,
                      hipStream_t s) {
  Arena plan;
  carve_streams(plan, h, p, sp);
  Scratch scratch;
  int rc = scratch.acquire(h.workspace, h.workspace_bytes, plan.bytes(), s);
  if (rc) return rc;
  Arena ar;
  ar.base = scratch.ptr();
  const StreamsScratch w = carve_streams(ar, h, p, sp);
  std::vector<uint8_t> meta(meta_bytes(sp));
  std::memcpy(meta.data(), sp.seq.data(), sp.seq.size() * sizeof(QerStreamDesc));
  std::memcpy(meta.data() + sp.seq.size() * sizeof(QerStreamDesc), sp.qry.data(),
              sp.qry.size() * sizeof(QerQueryDesc));
  rc = copy_to_device(w.meta, meta.data(), meta.size(), s, "the sequence tables");
  if (rc) return rc;
  const auto* seq_d = reinterpret_cast<const QerStreamDesc*>(w.meta);
  const auto* qry_d = reinterpret_cast<const QerQueryDesc*>(w.meta + sp.seq.size() * sizeof(QerStreamDesc));
  const bool bf16 = h.dtype == COFIE_BF16;
  const int32_t R = sp.n_queries * h.n_q;
  const uint8_t* qp = static_cast<const uint8_t*>(Q);
  if (p.fold) {
    const int64_t total = (int64_t)R * p.Lc;
    const unsigned grid = (unsigned)std::min<int64_t>(ceil_div(total, 256), 8192);
    rc = bf16 ? launch("qer_fold", qer_fold_kernel<bf16_t>, dim3(grid), dim3(256), 0, s,
                       static_cast<const bf16_t*>(Q), R, h.H_q, h.H_kv, h.d, (void*)w.qp)
              : launch("qer_fold", qer_fold_kernel<float>, dim3(grid), dim3(256), 0, s,
                       static_cast<const float*>(Q), R, h.H_q, h.H_kv, h.d, (void*)w.qp);
    if (rc) return rc;
    qp = w.qp;
  }
  const QerTrees tr = qer_trees(std::max(sp.max_frames, 1), sp.n_queries);
  const float base_scale = h.scale > 0.f ? h.scale : (float)(1.0 / std::sqrt((double)h.d));
  const int cus = device_cu_count();
  if (w.qop && sp.tiles > 0 && seq_span(sp, seq_nwg(sp, cus)) <= kSeqTab) {
    // the query side in operand order, then qer_seq_kernel
    const int32_t ksteps = (int32_t)(p.Lc * p.esize / 64);
    const int64_t total = (int64_t)sp.seq.size() * ksteps * kSeqNB * 64;
    if (dry_run())
      model_qop(static_cast<const uint4*>(Q), (int64_t)(p.Lc * p.esize / 16), seq_d, (int32_t)sp.seq.size(), ksteps,
                (int32_t)kSeqR, w.qop);
    rc = launch("qer_qop", qer_qop_kernel, dim3((unsigned)std::min<int64_t>(ceil_div(total, 256), 8192)), dim3(256),
                0, s, static_cast<const uint4*>(Q), (int64_t)(p.Lc * p.esize / 16), seq_d, (int32_t)sp.seq.size(),
                ksteps, (int32_t)kSeqR, w.qop);
    if (rc) return rc;
    SeqArgs qa{};
    qa.K = static_cast<const uint8_t*>(K);
    qa.Qop = w.qop;
    qa.seq = seq_d;
    qa.n_seq = (int32_t)sp.seq.size();
    qa.tiles = (int32_t)sp.tiles;
    qa.nwg = seq_nwg(sp, cus);
    qa.xcd_order = qa.nwg % 8 == 0 ? 1 : 0;
    qa.nseg = (int32_t)(p.Lc * p.esize / kSeqSegBytes);
    qa.k_row_u4 = (int32_t)(p.Lc * p.esize / 16);
    qa.scale = (float)((double)base_scale / (double)h.H_q);
    qa.m = w.m;
    qa.m_stride = std::max<int64_t>(sp.max_keys, 1);
    qa.group_rows = h.n_q;
    qa.clear = w.done;
    qa.nclear = sp.n_queries * tr.ints;
    auto kern = qer_seq_kernel<kSeqU, kSeqR>;
    const size_t lds = kSeqLds;
    rc = allow_lds(kern, lds);
    if (rc) return rc;
    if (dry_run()) model_seq<kSeqU, kSeqR>(qa, lds);
    rc = launch("qer_score", kern, dim3((unsigned)qa.nwg), dim3(kLdsThreads), lds, s, qa);
    if (rc) return rc;
    return launch_frame_mean(tr.nwg, sp.n_queries, 1024, s,
                  (const float*)w.m, (int32_t)qa.m_stride, frame_offsets, std::max(sp.max_frames, 1), out_scores,
                  w.keys, (const int32_t*)nullptr, w.done, tr.ints, tr.stride, k_top, out_idx, qry_d);
  }
  // the score kernel: one launch over every chunk's tiles (its workgroup 0
  // clears the frame-mean kernel's arrival trees, so it runs even without keys)
  LdsPlan L = plan_score_lds(std::max<int64_t>(sp.tiles, 1) * 16, p.Lc, p.esize, p.P, p.P * sp.NB, cus, false);
  if (sp.NB == 8 && L.MB != 1) {  // eight blocks take one tile per wave (two spill)
    L = plan_score_lds(std::min<int64_t>(sp.tiles, (int64_t)cus * kLdsWaves) * 16, p.Lc, p.esize, p.P,
                       p.P * sp.NB, cus, false);
  }
  ScoreLdsArgs sa{};
  sa.K = static_cast<const uint8_t*>(K);
  sa.Qp = qp;
  sa.n_vis = 0;  // per sequence
  sa.nq_total = R;
  sa.group_rows = h.n_q;
  sa.m_stride = std::max<int64_t>(sp.max_keys, 1);
  sa.Lc = (int32_t)p.Lc;
  sa.tiles = (int32_t)sp.tiles;
  sa.scale = (float)((double)base_scale / (double)h.H_q);
  sa.m = w.m;
  sa.clear = w.done;
  sa.nclear = sp.n_queries * tr.ints;
  sa.accumulate = 0;
  sa.nseg = L.nseg;
  sa.ksteps = L.ksteps;
  sa.S = L.S;
  sa.lgS = L.lgS;
  sa.nphase = L.nphase;
  sa.nwg = std::max(1, (L.nwg >= 8 ? L.nwg & ~7 : L.nwg));
  sa.xcd_order = sa.nwg % 8 == 0 ? 1 : 0;
  sa.split_u4 = L.split_u4;
  sa.k_row_u4 = (int32_t)(p.Lc * (int64_t)p.esize / 16);
  sa.streams = seq_d;
  sa.n_streams = (int32_t)sp.seq.size();
  L.nwg = sa.nwg;
  if (bf16) {
    if (sp.NB == 8)
      rc = launch_lds_t<bf16_t, 1, 8, 1, 1, kSeqLogit>(sa, L, L.lds, s);
    else if (p.P == 3)
      rc = L.MB == 1 ? launch_lds_nb<bf16_t, 1, 3, 1, kSeqLogit>(sa, L, sp.NB, L.lds, s)
                     : launch_lds_nb<bf16_t, 2, 3, 1, kSeqLogit>(sa, L, sp.NB, L.lds, s);
    else
      rc = L.MB == 1 ? launch_lds_nb<bf16_t, 1, 1, 1, kSeqLogit>(sa, L, sp.NB, L.lds, s)
                     : launch_lds_nb<bf16_t, 2, 1, 1, kSeqLogit>(sa, L, sp.NB, L.lds, s);
  } else {
    if (sp.NB == 8)
      rc = launch_lds_t<float, 1, 8, 1, 1, kSeqLogit>(sa, L, L.lds, s);
    else
      rc = L.MB == 1 ? launch_lds_nb<float, 1, 1, 1, kSeqLogit>(sa, L, sp.NB, L.lds, s)
                     : launch_lds_nb<float, 2, 1, 1, kSeqLogit>(sa, L, sp.NB, L.lds, s);
  }
  if (rc) return rc;
  return launch_frame_mean(tr.nwg, sp.n_queries, 1024, s,
                (const float*)w.m, (int32_t)sa.m_stride, frame_offsets, std::max(sp.max_frames, 1), out_scores,
                w.keys, (const int32_t*)nullptr, w.done, tr.ints, tr.stride, k_top, out_idx, qry_d);
}

}  // namespace

// Eqs. 7-8 from a finished m (one query): w_f and its top-k.  keys: scratch
// of n_frames words.  Shared with the fused attention path.
int qer_rank_from_m(const float* m, int32_t n_vis, const int32_t* offs, int32_t n_frames, int32_t k_top,
                    float* out_scores, uint32_t* keys, int32_t* out_idx, hipStream_t s) {
  if (n_frames > 0) {
    int rc = launch_frame_mean(ceil_div(n_frames, 4), 1, 256, s, m, n_vis, offs, n_frames, out_scores, keys,
                               (const int32_t*)nullptr, (int32_t*)nullptr, 0, 0, k_top, out_idx,
                               (const QerQueryDesc*)nullptr);
    if (rc) return rc;
  }
  if (k_top == 0) return COFIE_OK;
  return launch("qer_topk", qer_topk_kernel, dim3(1), dim3(1024), 0, s, (const uint32_t*)keys, n_frames, k_top,
                out_idx, (const int32_t*)nullptr);
}

}  // namespace cofie

// ---- scratch of the entry point that allocates nothing ------------------------------
// cofie_qer_rank_noalloc's scratch: a file-scope device array, one copy per
// device the library runs on, held until the process ends.  Host code never
// passes the array's name to a kernel or a copy (on the host it is only a
// stand-in for the symbol): it uses the device address hipGetSymbolAddress
// returns, taken once per device with that device current.
static __device__ __align__(256) unsigned char scratch[COFIE_QER_NOALLOC_SCRATCH_BYTES];

namespace cofie {
namespace {

// Device address of `scratch` on the current device (looked up on the first
// call on each device, then cached).
int noalloc_scratch(void** out) {
  static std::mutex mu;
  static void* addr[64] = {};
  if (dry_run()) {  // a fake address of the array's size, checked like the caller's buffers
    static const uintptr_t kDryScratch = uintptr_t(0x7e) << 40;
    *out = reinterpret_cast<void*>(kDryScratch);
    return cofie_debug_buffer(*out, COFIE_QER_NOALLOC_SCRATCH_BYTES, "static scratch");
  }
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return set_error(COFIE_EHIP, "hipGetDevice failed");
  if (dev < 0 || dev >= 64) return set_error(COFIE_EUNSUPPORTED, "device ordinal %d beyond 63", dev);
  std::lock_guard<std::mutex> lk(mu);
  if (!addr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return set_error(COFIE_EHIP, "hipGetSymbolAddress of the static scratch failed on device %d: %s", dev,
                       hipGetErrorString(e));
    addr[dev] = ptr;
  }
  *out = addr[dev];
  return COFIE_OK;
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
  return rank_impl(Q, K, frame_offsets, *heads, 1, nullptr, k_top, out_scores, out_idx,
                   static_cast<hipStream_t>(stream));
}

int cofie_qer_rank_noalloc(const void* Q, const void* K, const int32_t* frame_offsets,
                           const cofie_qer_desc* heads, int32_t k_top, float* out_scores,
                           int32_t* out_idx, void* stream) {
  clear_error();
  int rc = validate_qer(Q, K, frame_offsets, heads, k_top, out_scores, out_idx);
  if (rc) return rc;
  if (heads->workspace)
    return set_error(COFIE_EINVAL, "heads->workspace must be NULL: this call uses the library's static scratch");
  Arena ar;
  carve_qer(ar, *heads, plan_qer(*heads));
  if (ar.bytes() > (size_t)COFIE_QER_NOALLOC_SCRATCH_BYTES)
    return set_error(COFIE_EUNSUPPORTED, "needs %zu bytes of scratch, more than the static %zu", ar.bytes(),
                     (size_t)COFIE_QER_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  rc = noalloc_scratch(&ws);
  if (rc) return rc;
  cofie_qer_desc h = *heads;
  h.workspace = ws;
  h.workspace_bytes = COFIE_QER_NOALLOC_SCRATCH_BYTES;
  return rank_impl(Q, K, frame_offsets, h, 1, nullptr, k_top, out_scores, out_idx,
                   static_cast<hipStream_t>(stream));
}

size_t cofie_qer_batched_workspace_bytes(const cofie_qer_desc* heads, int32_t n_queries, int32_t k_top) {
  static const uint64_t dummy[4] = {0, 0, 0, 0};
  static const int32_t doffs = 0;
  float dscore;
  int32_t didx;
  if (n_queries < 1 || validate_qer(dummy, dummy, &doffs, heads, k_top, &dscore, &didx)) return 0;
  Arena ar;
  carve_qer(ar, *heads, plan_qer(*heads, n_queries), n_queries);
  return ar.bytes();
}

int cofie_qer_rank_batched(const void* Q, const void* K, const int32_t* frame_offsets,
                           const cofie_qer_desc* heads, int32_t n_queries, const int32_t* n_frames_per_query,
                           int32_t k_top, float* out_scores, int32_t* out_idx, void* stream) {
  clear_error();
  int rc = validate_qer(Q, K, frame_offsets, heads, k_top, out_scores, out_idx);
  if (rc) return rc;
  const cofie_qer_desc& h = *heads;
  if (n_queries < 1) return set_error(COFIE_EINVAL, "n_queries = %d must be >= 1", n_queries);
  if (!n_frames_per_query) return set_error(COFIE_EINVAL, "n_frames_per_query is NULL");
  for (int32_t g = 0; g < n_queries; ++g)
    if (n_frames_per_query[g] < 0 || n_frames_per_query[g] > h.n_frames)
      return set_error(COFIE_EINVAL, "query %d: %d frames outside [0, n_frames = %d]", g, n_frames_per_query[g],
                       h.n_frames);
  if (n_queries > 1 && h.n_q % 16 != 0)
    return set_error(COFIE_EUNSUPPORTED, "several queries need n_q (%d) a multiple of 16", h.n_q);
  if (n_queries > 1 && h.score_mode != COFIE_SCORE_LOGIT && !plan_qer(h, n_queries).soft_fast)
    return set_error(COFIE_EUNSUPPORTED,
                     "several queries in SOFTMAX mode need heads of whole 128-byte key segments "
                     "(d a multiple of %d elements)", h.dtype == COFIE_BF16 ? 64 : 32);
  if ((int64_t)n_queries * h.n_q * h.H_q * h.d >= (int64_t(1) << 31))
    return set_error(COFIE_EUNSUPPORTED, "queries too large");
  return rank_impl(Q, K, frame_offsets, h, n_queries, n_frames_per_query, k_top, out_scores, out_idx,
                   static_cast<hipStream_t>(stream));
}

size_t cofie_qer_streams_workspace_bytes(const cofie_qer_desc* heads, int32_t n_streams, const int64_t* stream_keys,
                                         const int32_t* stream_frames, const int32_t* stream_queries,
                                         const int32_t* n_frames_per_query, int32_t k_top) {
  static const uint64_t dummy[4] = {0, 0, 0, 0};
  static const int32_t doffs = 0;
  float dscore;
  int32_t didx;
  if (validate_qer(dummy, dummy, &doffs, heads, k_top, &dscore, &didx)) return 0;
  const QerPlan p = plan_qer(*heads);
  StreamsPlan sp;
  if (plan_streams(*heads, p, n_streams, stream_keys, stream_frames, stream_queries, n_frames_per_query, sp)) return 0;
  Arena ar;
  carve_streams(ar, *heads, p, sp);
  return ar.bytes();
}

int cofie_qer_rank_streams(const void* Q, const void* K, const int32_t* frame_offsets, const cofie_qer_desc* heads,
                           int32_t n_streams, const int64_t* stream_keys, const int32_t* stream_frames,
                           const int32_t* stream_queries, const int32_t* n_frames_per_query, int32_t k_top,
                           float* out_scores, int32_t* out_idx, void* stream) {
  clear_error();
  int rc = validate_qer(Q, K, frame_offsets, heads, k_top, out_scores, out_idx);
  if (rc) return rc;
  if (!out_scores) return set_error(COFIE_EINVAL, "out_scores is NULL");
  const QerPlan p = plan_qer(*heads);
  StreamsPlan sp;
  rc = plan_streams(*heads, p, n_streams, stream_keys, stream_frames, stream_queries, n_frames_per_query, sp);
  if (rc) return rc;
  return rank_streams_impl(Q, K, frame_offsets, *heads, p, sp, k_top, out_scores, out_idx,
                           static_cast<hipStream_t>(stream));
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


int cofie_topk(const float* w, int32_t n, int32_t k_top, int32_t* out_idx, void* stream) {
  clear_error();
  if (n < 0 || k_top < 0) return set_error(COFIE_EINVAL, "negative n or k_top");
  if (k_top > 0 && !out_idx) return set_error(COFIE_EINVAL, "out_idx is NULL");
  if (n > 0 && !w) return set_error(COFIE_EINVAL, "w is NULL");
  if (k_top == 0) return COFIE_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  Scratch scratch;
  int rc = scratch.acquire(nullptr, 0, (size_t)(n > 0 ? n : 1) * sizeof(uint32_t), s);
  if (rc) return rc;
  uint32_t* keys = reinterpret_cast<uint32_t*>(scratch.ptr());
  if (n > 0) {
    rc = launch("qer_order_keys", order_keys_kernel, dim3((unsigned)std::min<int64_t>(ceil_div(n, 256), 4096)),
                dim3(256), 0, s, w, n, keys);
    if (rc) return rc;
  }
  return launch("qer_topk", qer_topk_kernel, dim3(1), dim3(1024), 0, s, (const uint32_t*)keys, n, k_top, out_idx,
                (const int32_t*)nullptr);
}

int cofie_evidence_preservation(const float* w, const uint8_t* mask, int32_t n, double top_frac, double* out,
                                void* stream) {
  clear_error();
  if (n < 0) return set_error(COFIE_EINVAL, "n is negative");
  if (!out) return set_error(COFIE_EINVAL, "out is NULL");
  if (n > 0 && (!w || !mask)) return set_error(COFIE_EINVAL, "w or mask is NULL");
  if (!(top_frac >= 0)) return set_error(COFIE_EINVAL, "top_frac must be a non-negative number");
  hipStream_t s = static_cast<hipStream_t>(stream);
  int64_t k = n > 0 ? cofie_qer_k_from_ratio(top_frac, n) : 0;
  if (k > n) k = n;
  Scratch scratch;
  int rc = scratch.acquire(nullptr, 0, (size_t)(k > 0 ? k : 1) * sizeof(int32_t), s);
  if (rc) return rc;
  int32_t* top = reinterpret_cast<int32_t*>(scratch.ptr());
  if (k > 0) {
    rc = cofie_topk(w, n, (int32_t)k, top, stream);
    if (rc) return rc;
  }
  return launch("qer_evidence", evidence_kernel, dim3(1), dim3(1024), 0, s, w, mask, n, (const int32_t*)top,
                (int32_t)k, out);
}

}  // extern "C"

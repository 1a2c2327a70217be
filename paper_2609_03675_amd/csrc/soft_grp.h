// SOFTMAX-mode QER for grouped query heads (Sec. 3.3, Eqs. 6-7 in the
// per-head softmax reading): the two passes of qer_soft_grp_kernel, launched
// by the QER driver between which the partial statistics are merged.
#pragma once

#include "common.h"

namespace cofie {

struct SoftGrpArgs {
  const uint4* K;         // [n_vis][H_kv][128] bf16: 16 uint4 per key head row
  const uint4* Q;         // [n_q][H_q][128] bf16
  int32_t n_vis, n_q;
  int32_t tiles;          // ceil(n_vis / 16)
  int32_t nb;             // 16-row blocks of the query rows
  int32_t ranges;         // pass 2: key ranges (a multiple of 8), one workgroup per range and row block
  int32_t ranges1;        // pass 1: key ranges (a multiple of 8), one workgroup per range, key head
  int32_t nbw;            //   and set of nbw row blocks
  int32_t nbs;            //   (nbs sets: ceil(nb / nbw))
  float c2;               // scale * log2(e)
  float inv_h;            // 1 / H_q
  float2* stats_part;     // pass 1: [(H_q n_q + 15) / 16][ranges1][16], row h n_q + q
  const float2* stats;    // pass 2: the merged (max * scale, sum of exp) of every row
  float* m;               // [n_vis]: max over the rows of the head mean of the probabilities
  int32_t* clear;         // pass 1 zeroes clear[0, nclear) (the frame-mean arrival trees)
  int32_t nclear;
  int32_t q_gstride;      // query-fragment slots (uint4) per key head in LDS: G * 256
};

// Whether an instance exists for hkv key heads with g query heads each.
bool grp_has_instance(int hkv, int g);
// Row blocks a pass-1 workgroup holds (the fragments of g query heads for each
// take 4 KiB per head in LDS), at most 4.
int grp_nbw(int g, int nb);
// Pass 1 (statistics; hkv * a.nbs * a.ranges1 workgroups) or 2
// (probabilities; a.nb * a.ranges workgroups); in a dry run, the address
// model instead.
int launch_grp(const SoftGrpArgs& a, int hkv, int g, int pass, hipStream_t s);

}  // namespace cofie

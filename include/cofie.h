/*
 * cofie.h -- C ABI of libcofie: CoFiE evidence selection on AMD Instinct
 * MI355X (gfx950).
 *
 * CoFiE selects evidence frames for a video LLM in two stages:
 *   NGFF  Novelty-Guided Frame Filtering (Sec. 3.2): per-frame histograms of
 *         raw uint8 frames, a total-variation novelty score against the
 *         previous frame and the last kept frame, and a gap-aware keep rule,
 *         run before any vision encoder.
 *   QER   Query-Specific Evidence Refinement (Sec. 3.3): head-averaged
 *         text-to-visual scaled dot products at prefill, max over text tokens,
 *         mean over each frame's visual tokens, top-k frames.
 *
 * Conventions shared by every entry point
 *   - Return value: COFIE_OK (0) or a negative COFIE_E* status.  On error,
 *     cofie_last_error() returns a message for the calling thread.  Nothing
 *     throws across this boundary.
 *   - "device" pointers are HIP device memory (for example from PyTorch on
 *     ROCm); "host" pointers are read during the call only.  The library never
 *     keeps a pointer past the call and never frees caller memory.
 *   - Every argument is validated on the host before any work is enqueued;
 *     a rejected call enqueues nothing.
 *   - `stream` is a hipStream_t (NULL = the null stream).  All work is
 *     enqueued on it asynchronously; outputs are valid once the caller has
 *     synchronised the stream.
 *   - Scratch memory: a caller may pass a device workspace of at least the
 *     size the matching *_workspace_bytes() function reports.  With a NULL
 *     workspace the library allocates and frees scratch with stream-ordered
 *     hipMallocAsync / hipFreeAsync on `stream`.
 *   - Results are deterministic: the same inputs give the same output bits.
 */
#ifndef COFIE_H_
#define COFIE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------- */
#define COFIE_OK 0
#define COFIE_EINVAL (-1)       /* invalid argument (null pointer, bad size or enum) */
#define COFIE_EUNSUPPORTED (-2) /* valid but outside what the library implements */
#define COFIE_EHIP (-3)         /* a HIP runtime call or kernel launch failed */
#define COFIE_ENOMEM (-4)       /* scratch allocation failed or workspace too small */

/* ---- enums -------------------------------------------------------------- */
/* Histogram of a frame (Sec. 3.2).  B = `bins` (a power of two).  Intensity v
 * falls in bin floor(v * B / 256), i.e. B equal bins over the normalised range.
 *   GRAY         B bins of the BT.601 luma (299 R + 587 G + 114 B + 500) div 1000
 *                (C = 3) or of the single channel (C = 1).  The paper's default
 *                (32 bins).  Mass M = H*W.
 *   PER_CHANNEL  3B bins: R, G and B histograms side by side.  Mass M = 3*H*W;
 *                the total-variation distance is then the mean of the three
 *                per-channel distances.  C = 3.
 *   JOINT3D      B^3 bins indexed (bin(R)*B + bin(G))*B + bin(B).  Mass M = H*W.
 *                C = 3, B^3 <= 4096.                                          */
/* The novelty signal can also be one of the alternative pre-encoder signals
 * of the paper's filtering-signal ablation (Table 5, defined there only by
 * citation; readings):
 *   FRAMEDIFF    low-resolution frame difference: the luma image (BT.601 in
 *                integers as for GRAY; the value itself when C = 1) box-
 *                averaged on a G x G grid, G = `bins` (a power of two in
 *                [2, 64], G <= H and G <= W), each cell mean rounded half up;
 *                row = the G^2 means; distance = L1 / (255 G^2) (2M = 255 G^2).
 *   DHASH        difference hash: luma box means on 8 rows x 9 columns (H >= 8,
 *                W >= 9; `bins` unused); row = 64 entries, 1 where cell
 *                (r, c+1) is brighter than cell (r, c); distance = Hamming / 64.
 * Row y belongs to grid row (y * rows) div H, column x to (x * cols) div W.
 * W <= 16384.  The keep rule, calibration and histogram outputs work on these
 * rows unchanged; the online state (cofie_ngff_stream_*) does not take them. */
enum cofie_hist_mode {
  COFIE_HIST_GRAY = 0,
  COFIE_HIST_PER_CHANNEL = 1,
  COFIE_HIST_JOINT3D = 2,
  COFIE_SIGNAL_FRAMEDIFF = 3,
  COFIE_SIGNAL_DHASH = 4
};

/* Element type of Q and K. */
enum cofie_dtype { COFIE_F32 = 0, COFIE_BF16 = 1 };

/* Text-to-visual association a_ij aggregated by QER.
 *   LOGIT    the paper's Eq. 6: head mean of scaled dot products.
 *   SOFTMAX  head mean of softmax-normalised scaled dot products, each softmax
 *            taken over all n_vis visual keys passed in (not over the model's
 *            full key set).                                                  */
enum cofie_score_mode { COFIE_SCORE_LOGIT = 0, COFIE_SCORE_SOFTMAX = 1 };

/* ---- NGFF --------------------------------------------------------------- */

/* Keep rule of NGFF (Sec. 3.2, Eqs. 3-5 and the gap-aware safeguards).
 * For each independent stream of T frames:
 *   s_t = max(d(h_t, h_{t-1}), d(h_t, h_{r(t)})), d = total variation of the
 *         normalised histograms, computed as the exact integer L1 distance D of
 *         the counts divided once, in IEEE fp32, by 2M; s_0 = 1.
 *   r(t) = the most recent frame kept by the rule below (top-up frames excluded).
 *   Frame 0 and frame T-1 are kept; frame 0 < t < T-1 is kept when
 *   s_t >= tau or (L_max > 0 and t - r(t) >= L_max).  If fewer than M_min
 *   frames are kept (M_min >= 2), the frames floor(i (T-1) / (M_min-1)),
 *   i = 0..M_min-1, are added.                                                 */
typedef struct cofie_keep_rule {
  int32_t hist_mode;             /* enum cofie_hist_mode (paper default: GRAY)      */
  float tau_h;                   /* novelty threshold tau (paper default 0.30);      */
                                 /*   any non-NaN value: < 0 keeps every frame,     */
                                 /*   > 1 keeps only the forced frames              */
  const float* tau_per_segment;  /* optional device [n_segments]: one tau per       */
                                 /*   stream, overrides tau_h (e.g. the output of   */
                                 /*   cofie_ngff_calibrate)                         */
  int32_t L_max;                 /* forced-retention gap in frames (default 30);    */
                                 /*   <= 0 disables the gap rule                    */
  int32_t M_min;                 /* minimum kept frames per stream (default 4)      */
  int64_t segment_len;           /* frames per independent stream; 0 = the whole   */
                                 /*   batch is one stream; the last may be shorter  */
  uint32_t* out_hist;            /* optional device [n][nbins] histogram counts     */
  int32_t* out_count;            /* optional device [n_segments] kept frames         */
  void* workspace;               /* optional device scratch (see header comment)    */
  size_t workspace_bytes;
} cofie_keep_rule;

/* Fill *rule with the paper's defaults: GRAY histogram, tau_h = 0.30,
 * L_max = 30, M_min = 4 (Sec. 3.2; Table 7's middle row), one stream, no
 * optional outputs, library-managed scratch. */
void cofie_keep_rule_default(cofie_keep_rule* rule);

/* Number of histogram bins (row entries) for a mode and `bins` (B, 3B, B^3;
 * G^2 for FRAMEDIFF, 64 for DHASH); 0 if invalid. */
int64_t cofie_ngff_nbins(int32_t hist_mode, int32_t bins);

/* Bytes of device scratch cofie_ngff_filter / cofie_ngff_calibrate need for
 * these arguments (0 for invalid arguments). */
size_t cofie_ngff_workspace_bytes(int64_t n, int32_t H, int32_t W, int32_t C, int32_t bins,
                                  const cofie_keep_rule* rule);

/* Per-frame histogram counts of NGFF (Sec. 3.2, the normalised B-bin
 * histogram h_t = counts / M).
 *   frames    device uint8 [n][H][W][C], C-order, channels interleaved (RGB)
 *   n         frames (n = 0: nothing to do)
 *   H, W, C   frame shape; C = 3, or C = 1 with GRAY
 *   bins      B, a power of two in [2, 256]
 *   out_hist  device uint32 [n][nbins], fully overwritten
 * Errors: EINVAL for null pointers, negative/zero sizes, bad enums or C;
 * EUNSUPPORTED for B not a power of two, B^3 > 4096, or 2M >= 2^31.       */
int cofie_ngff_histogram(const uint8_t* frames, int64_t n, int32_t H, int32_t W, int32_t C,
                         int32_t bins, int32_t hist_mode, uint32_t* out_hist, void* stream);

/* NGFF end to end (Sec. 3.2, Eqs. 2-5 and safeguards): histograms, novelty
 * scores and the keep rule of `keep_rule` (host struct).
 *   out_scores  device float [n]: s_t (s = 1 for each stream's first frame)
 *   out_mask    device uint8 [n]: 1 = frame is a candidate (in S_c), else 0
 * Same frame arguments and errors as cofie_ngff_histogram; also EINVAL for
 * a NULL keep_rule, a NaN tau_h, M_min < 0 or segment_len < 0; ENOMEM if the
 * caller's workspace is smaller than cofie_ngff_workspace_bytes(). */
int cofie_ngff_filter(const uint8_t* frames, int64_t n, int32_t H, int32_t W, int32_t C,
                      int32_t bins, const cofie_keep_rule* keep_rule, float* out_scores,
                      uint8_t* out_mask, void* stream);

/* NGFF's keep rule on histograms computed earlier (for example by
 * cofie_ngff_histogram on another stream, so that independent work can run
 * beside the rule): everything cofie_ngff_filter does after its histogram
 * (Sec. 3.2, Eqs. 2-5 and safeguards), with the same scores and mask.
 *   hist      device uint32 [n][nbins] counts as cofie_ngff_histogram writes
 *             them for frames of shape H x W x C and `bins` (they fix M and
 *             nbins); read only
 * Other arguments, outputs and errors as cofie_ngff_filter;
 * keep_rule->out_hist is ignored. */
int cofie_ngff_filter_hist(const uint32_t* hist, int64_t n, int32_t H, int32_t W, int32_t C, int32_t bins,
                           const cofie_keep_rule* keep_rule, float* out_scores, uint8_t* out_mask,
                           void* stream);

/* Threshold calibration for a retention target (the paper fixes tau_h; a
 * target kept count per stream is an extension).  Per stream, among the
 * candidate integer thresholds theta in {0, 2M+1} and every distance
 * D(t, t-k), 1 <= k <= L_max, the smallest one whose keep rule (with
 * tau = fl32(theta)/fl32(2M), top-up included) keeps at most
 * `target_per_segment` frames; 2M+1 if none does.  Writes that tau to
 * out_tau (device float [n_segments]), ready for tau_per_segment.  Uses
 * hist_mode, L_max (>= 1 required, else EUNSUPPORTED), M_min, segment_len and
 * the workspace of keep_rule; tau_h, tau_per_segment, out_hist and out_count
 * are ignored. */
int cofie_ngff_calibrate(const uint8_t* frames, int64_t n, int32_t H, int32_t W, int32_t C,
                         int32_t bins, const cofie_keep_rule* keep_rule,
                         int64_t target_per_segment, float* out_tau, void* stream);

/* ---- NGFF as frames arrive ---------------------------------------------- */
/* The keep rule applied online (Sec. 3.1: the model sees the current video
 * prefix; Sec. 3.2): each frame is decided when it is pushed, by the rule
 * above without its two end-of-stream safeguards (frame T-1 kept, the M_min
 * top-up), which cofie_ngff_stream_finish applies once the streams end.
 * Pushing a stream's frames in any batches and finishing gives exactly the
 * scores and mask of one cofie_ngff_filter call over the whole stream.  The
 * state holds, per stream, the histograms of the last L_max frames, the last
 * kept frame and the kept count; it lives on the device current at creation
 * and is used from one stream at a time. */
typedef struct cofie_ngff_stream cofie_ngff_stream;

/* New state for n_streams streams of H x W x C frames (as cofie_ngff_histogram).
 * From `rule` (host, read during the call): hist_mode, tau_h or
 * tau_per_segment (device [n_streams], copied), L_max (>= 1 required, else
 * EUNSUPPORTED: the rule then compares against a kept frame that can be
 * arbitrarily old) and M_min; segment_len, out_hist, out_count and the
 * workspace are ignored.  Allocates device memory (synchronous).  Errors as
 * cofie_ngff_filter, plus ENOMEM. */
int cofie_ngff_stream_create(int32_t n_streams, int32_t H, int32_t W, int32_t C, int32_t bins,
                             const cofie_keep_rule* rule, cofie_ngff_stream** out_state);

/* Push b >= 0 new frames of every stream.
 *   frames      device uint8: frame j of stream s at frames + (s*frames_ld + j)
 *               * H*W*C, frames_ld >= b (b for a packed [n_streams][b] batch;
 *               T with frames pointing at column t0 of a [n_streams][T] array)
 *   out_scores  device float: s_t of stream s's new frame j at out_scores[s*ld + j]
 *   out_mask    device uint8, same layout: 1 = kept by the rule so far
 *   ld          row stride of the outputs (>= b); pointing the outputs at
 *               column t0 of [n_streams][T] arrays collects whole streams
 * Scratch is allocated stream-ordered.  Errors: EINVAL for NULL pointers,
 * b < 0, ld or frames_ld < b, a finished state or another current device. */
int cofie_ngff_stream_push(cofie_ngff_stream* state, const uint8_t* frames, int64_t frames_ld, int32_t b,
                           float* out_scores, uint8_t* out_mask, int64_t ld, void* stream);

/* End of the streams: in mask_all (device uint8 [n_streams][ld], frames
 * 0..T-1 of every stream as pushed) frame T-1 is kept and, where fewer than
 * M_min frames are kept, the top-up frames are added.  out_added (optional,
 * device int32 [n_streams][M_min+1]) receives the frames this adds,
 * increasing and -1 padded; out_count (optional, device int32 [n_streams])
 * the kept counts.  The state accepts no push afterwards. */
int cofie_ngff_stream_finish(cofie_ngff_stream* state, uint8_t* mask_all, int64_t ld, int32_t* out_added,
                             int32_t* out_count, void* stream);

/* Frames pushed per stream so far (-1 for NULL). */
int64_t cofie_ngff_stream_frames(const cofie_ngff_stream* state);

/* Checkpoint and resume of the streams (the keep rule of Sec. 3.2 needs only
 * the last L_max histograms, r and the kept count of every stream).
 * cofie_ngff_stream_state_bytes: size of a saved state (0 for NULL).
 * cofie_ngff_stream_save writes it to host memory `buf` (bytes >= that size)
 * once the work enqueued before it on `stream` has run; it returns after the
 * copy (synchronises `stream`).  cofie_ngff_stream_restore loads such a blob
 * into a state created with the same n_streams, frame shape, bins and keep
 * rule (thresholds compared bit for bit), on the state's device; the next
 * push continues where the saved streams stopped, with the same results as
 * an uninterrupted run.  The caller keeps the masks of the frames already
 * pushed (cofie_ngff_stream_finish needs them).  Errors: EINVAL for NULL,
 * a short buffer, another device, a blob of another format, shape or rule. */
size_t cofie_ngff_stream_state_bytes(const cofie_ngff_stream* state);
int cofie_ngff_stream_save(const cofie_ngff_stream* state, void* buf, size_t bytes, void* stream);
int cofie_ngff_stream_restore(cofie_ngff_stream* state, const void* buf, size_t bytes, void* stream);

/* Release the state (NULL is accepted).  Frees device memory: call it after
 * the work enqueued with the state has completed. */
int cofie_ngff_stream_destroy(cofie_ngff_stream* state);

/* ---- QER ---------------------------------------------------------------- */

typedef struct cofie_qer_desc {
  int32_t n_q;        /* text (query) tokens used for scoring, >= 1                 */
  int32_t n_vis;      /* visual tokens (rows of K), >= 0                            */
  int32_t n_frames;   /* frames (CSR segments of the visual tokens), >= 0           */
  int32_t H_q;        /* query heads                                                */
  int32_t H_kv;       /* key heads; H_q % H_kv == 0; query head h reads key head    */
                      /*   h / (H_q / H_kv) (contiguous groups)                     */
  int32_t d;          /* head dimension, a multiple of 16                           */
  int32_t dtype;      /* enum cofie_dtype of Q and K                                */
  int32_t score_mode; /* enum cofie_score_mode                                      */
  float scale;        /* dot-product scale; <= 0 selects 1/sqrt(d)                  */
  void* workspace;    /* optional device scratch (see header comment)               */
  size_t workspace_bytes;
} cofie_qer_desc;

/* Bytes of device scratch cofie_qer_rank needs (0 for invalid arguments). */
size_t cofie_qer_workspace_bytes(const cofie_qer_desc* heads, int32_t k_top);

/* QER frame ranking (Sec. 3.3, Eqs. 6-8):
 *   a_ij = (1/H_q) sum_h scale * <q_i^h, k_j^h>          (LOGIT; Eq. 6)
 *   w_f  = (1/|V_f|) sum_{j in V_f} max_i a_ij           (Eq. 7; -inf if V_f empty)
 *   S_e  = the k_top frames of largest w_f               (Eq. 8)
 *   Q              device [n_q][H_q][d] of dtype, row-major (post-RoPE queries)
 *   K              device [n_vis][H_kv][d] of dtype, row-major (post-RoPE keys)
 *   frame_offsets  device int32 [n_frames+1], CSR: V_f = [off[f], off[f+1]);
 *                  values are clamped to [0, n_vis] and an inverted range is an
 *                  empty frame, so malformed offsets never read out of bounds
 *   heads          host descriptor
 *   k_top          frames to keep (>= 0); more than n_frames keeps all
 *   out_scores     device float [n_frames]: w_f
 *   out_idx        device int32 [k_top] (may be NULL if k_top == 0): the winners
 *                  ordered by score descending, ties to the lower frame index,
 *                  NaN ranked as -inf, returned in ascending (chronological)
 *                  frame order and padded with -1.
 * bf16 inputs are multiplied on MFMA with fp32 accumulation; fp32 inputs use
 * the fp32 MFMA.  Errors: EINVAL for null pointers, sizes or enums out of
 * range or H_q % H_kv != 0; EUNSUPPORTED for d % 16 != 0; ENOMEM for a short
 * workspace. */
int cofie_qer_rank(const void* Q, const void* K, const int32_t* frame_offsets,
                   const cofie_qer_desc* heads, int32_t k_top, float* out_scores,
                   int32_t* out_idx, void* stream);

/* cofie_qer_rank for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same arguments, kernels and results, but the scratch is a static
 * device array of the library (COFIE_QER_NOALLOC_SCRATCH_BYTES, one copy per
 * device, held until the process ends) instead of a workspace or an
 * allocation; the call makes no hipMalloc/hipFree and no allocating library
 * call.  heads->workspace must be NULL (EINVAL).  A call needing more scratch
 * than the array (cofie_qer_workspace_bytes() above the maximum) returns
 * EUNSUPPORTED before anything is enqueued.  Every call on a device shares
 * that device's array: calls that overlap on one device (two streams, or two
 * host threads) race and must be serialised by the caller; calls in one
 * stream order are safe.  The array keeps the last call's contents; everything
 * a call reads is written or cleared by that call's own kernels first. */
#define COFIE_QER_NOALLOC_SCRATCH_BYTES (32u << 20)
int cofie_qer_rank_noalloc(const void* Q, const void* K, const int32_t* frame_offsets,
                           const cofie_qer_desc* heads, int32_t k_top, float* out_scores,
                           int32_t* out_idx, void* stream);

/* Several queries sharing one key sequence, K read once for all of them
 * (the multi-stream workload: a stream's queries rank prefixes of its
 * candidates).  Query g has heads->n_q rows of Q (device
 * [n_queries][n_q][H_q][d]) and ranks the first n_frames_per_query[g] frames
 * of frame_offsets (host int32 [n_queries], each in [0, n_frames]) exactly as
 * cofie_qer_rank would: out_scores row g (device float [n_queries][n_frames])
 * holds its w_f (-inf past its prefix), out_idx row g (device int32
 * [n_queries][k_top]) its top-k.  With n_queries > 1: n_q a multiple of 16,
 * and in SOFTMAX mode head rows of whole 128-byte key segments (d a multiple
 * of 64 bf16 or 32 fp32 elements), else EUNSUPPORTED; query g's softmax then
 * normalises over the keys of its own prefix, as a call given only those keys
 * would (equal to rounding: the work split, which orders the sums, follows the
 * key count).  Workspace: the descriptor's, of
 * cofie_qer_batched_workspace_bytes() bytes. */
size_t cofie_qer_batched_workspace_bytes(const cofie_qer_desc* heads, int32_t n_queries, int32_t k_top);
int cofie_qer_rank_batched(const void* Q, const void* K, const int32_t* frame_offsets,
                           const cofie_qer_desc* heads, int32_t n_queries, const int32_t* n_frames_per_query,
                           int32_t k_top, float* out_scores, int32_t* out_idx, void* stream);

/* Several independent key sequences ranked in one launch (the multi-stream
 * workload: every stream's queries rank prefixes of that stream's
 * candidates, Sec. 3.1's streaming setting, Eqs. 6-8 per query).
 *   K              device [n_vis][H_kv][d]: the sequences' keys one after the
 *                  other; sequence s owns rows [stream_keys[s], stream_keys[s+1])
 *   frame_offsets  device int32 [n_frames+1], one CSR over all sequences'
 *                  frames (absolute key rows); sequence s owns frames
 *                  [stream_frames[s], stream_frames[s+1]), whose key ranges are
 *                  clamped to its own rows
 *   Q              device [n_queries][n_q][H_q][d]; queries are grouped by
 *                  sequence: sequence s owns queries [stream_queries[s],
 *                  stream_queries[s+1]), n_queries = stream_queries[n_streams]
 *   stream_keys    host int64 [n_streams+1], stream_frames and stream_queries
 *                  host int32 [n_streams+1]: non-decreasing, starting at 0,
 *                  ending at heads->n_vis, heads->n_frames and n_queries
 *   n_frames_per_query  host int32 [n_queries]: query g ranks the first
 *                  n_frames_per_query[g] frames of its sequence
 *   out_scores     device float [n_queries][F], F = max(1, the largest
 *                  sequence's frame count): row g holds w_f of its sequence's
 *                  frames (-inf past its prefix)
 *   out_idx        device int32 [n_queries][k_top]: each query's top-k as in
 *                  cofie_qer_rank, as frame indices within its sequence.
 * Each query's scores equal cofie_qer_rank given its sequence's keys and the
 * CSR of its prefix, to rounding (the contraction order is the same; only
 * the fp32 additions' grouping follows the work split).  LOGIT mode only,
 * n_q a multiple of 16 and at most 128 (64 with grouped-query heads), else
 * EUNSUPPORTED.  A sequence's queries are scored in chunks of at most 128
 * rows (64 grouped), each chunk reading the sequence's keys once; the keys of
 * all sequences stream in one score-kernel launch and the frame means and
 * top-k of all queries in one more.  Workspace: the descriptor's, of
 * cofie_qer_streams_workspace_bytes() bytes (0 for invalid arguments). */
size_t cofie_qer_streams_workspace_bytes(const cofie_qer_desc* heads, int32_t n_streams, const int64_t* stream_keys,
                                         const int32_t* stream_frames, const int32_t* stream_queries,
                                         const int32_t* n_frames_per_query, int32_t k_top);
int cofie_qer_rank_streams(const void* Q, const void* K, const int32_t* frame_offsets, const cofie_qer_desc* heads,
                           int32_t n_streams, const int64_t* stream_keys, const int32_t* stream_frames,
                           const int32_t* stream_queries, const int32_t* n_frames_per_query, int32_t k_top,
                           float* out_scores, int32_t* out_idx, void* stream);

/* ---- last-layer prefill attention with QER from its QK^T tiles ------------ */

typedef struct cofie_attn_desc {
  int32_t L;          /* prefill tokens (rows of Q, K, V), >= 1                      */
  int32_t H_q, H_kv;  /* heads; H_q % H_kv == 0, query head h reads key/value head   */
                      /*   h / (H_q / H_kv)                                         */
  int32_t d;          /* head dimension: 128 (others EUNSUPPORTED)                   */
  int32_t vis_begin;  /* visual tokens are [vis_begin, vis_end); every other token   */
  int32_t vis_end;    /*   is text (the scoring set of Sec. 3.3), at least one       */
  int32_t n_frames;   /* frames of the visual tokens, >= 0                           */
  float scale;        /* softmax and QER scale; <= 0 selects 1/sqrt(d)               */
  void* workspace;    /* optional device scratch of                                  */
  size_t workspace_bytes; /* cofie_attn_qer_workspace_bytes(); else allocated        */
} cofie_attn_desc;

/* Bytes of device scratch cofie_attn_qer needs (0 for an invalid descriptor). */
size_t cofie_attn_qer_workspace_bytes(const cofie_attn_desc* desc);

/* The causal softmax attention of the last prefill layer, with QER (Sec. 3.3,
 * Eqs. 6-8) taken from the same QK^T tiles instead of a pass of its own:
 *   out[i][h]  = sum_{j<=i} softmax_j(scale <q_i^h, k_j^g>) v_j^g  (bf16)
 *   out_scores = w_f and out_idx = S_e exactly as cofie_qer_rank in LOGIT
 *                mode for Q = the text rows (in sequence order) and K = the
 *                visual rows, frame_offsets relative to vis_begin
 *   Q            device bf16 [L][H_q][128]; K, V device bf16 [L][H_kv][128]
 *   out          device bf16 [L][H_q][128]
 *   frame_offsets device int32 [n_frames+1] (clamped as in cofie_qer_rank)
 * 16-byte aligned tensors.  Errors: EINVAL for NULL pointers or an invalid
 * descriptor (no text token included), EUNSUPPORTED for d != 128, ENOMEM for
 * a short workspace. */
int cofie_attn_qer(const void* Q, const void* K, const void* V, const int32_t* frame_offsets,
                   const cofie_attn_desc* desc, int32_t k_top, void* out, float* out_scores, int32_t* out_idx,
                   void* stream);

/* ---- coarse-to-fine glue ------------------------------------------------ */

/* The NGFF candidate set S_c as frame indices (Sec. 3.1-3.2: the candidates
 * are the frames the visual encoder runs on).
 *   mask           device uint8 [n]; nonzero = candidate (e.g. the out_mask of
 *                  cofie_ngff_filter)
 *   n              frames, 0 <= n < 2^31
 *   segment_len    frames per stream as in cofie_keep_rule (0 = one stream;
 *                  n_segments = ceil(n / segment_len), the last may be shorter)
 *   out_idx        device int32 [n] (may be NULL if n == 0): the candidate
 *                  indices in increasing (chronological) order; entries past
 *                  the candidate count are left untouched
 *   out_seg_start  device int32 [n_segments + 1]: candidates in the streams
 *                  before each stream; the last entry is the candidate count
 * Errors: EINVAL for a NULL pointer, n out of range or segment_len < 0. */
int cofie_mask_compact(const uint8_t* mask, int64_t n, int64_t segment_len, int32_t* out_idx,
                       int32_t* out_seg_start, void* stream);

/* Frame refinement (Sec. 3.3): the frames outside S_e are removed from a token
 * sequence (hidden states, cached keys or values, positions) and the kept
 * frames stay in chronological order.
 *   src                device [n_rows][row_bytes] bytes (any row type)
 *   frame_offsets      device int32 [n_frames+1], CSR of the frames' rows,
 *                      clamped as in cofie_qer_rank (an inverted range is empty)
 *   sel, k             device int32 [k]: the frames to keep, in output order
 *                      (the out_idx of cofie_qer_rank is chronological); entries
 *                      outside [0, n_frames), such as its -1 padding, keep nothing
 *   dst                device [dst_capacity_rows][row_bytes]: the kept rows,
 *                      appended frame by frame; rows beyond the capacity are not
 *                      written
 *   out_offsets        device int32 [k+1]: CSR of the kept rows per entry of
 *                      sel, counted in full (out_offsets[k] > capacity reports
 *                      a short dst); a running count past 2^31 - 1 (sel may
 *                      repeat frames) is stored as 2^31 - 1, and the frames
 *                      from there on are not copied
 *   out_rows           optional device int32 [dst_capacity_rows]: the source
 *                      row of every written dst row (e.g. to gather positions)
 * 16-byte accesses when src, dst and row_bytes are 16-byte aligned.  Errors:
 * EINVAL for NULL pointers, n_rows outside [0, 2^31), row_bytes <= 0, a
 * negative n_frames or k, or a capacity outside [0, 2^31). */
int cofie_gather_frames(const void* src, int64_t n_rows, int64_t row_bytes, const int32_t* frame_offsets,
                        int32_t n_frames, const int32_t* sel, int32_t k, void* dst,
                        int64_t dst_capacity_rows, int32_t* out_offsets, int32_t* out_rows,
                        void* stream);

/* Eq. 8's selection on given scores: the k_top frames of largest w (device
 * float [n]), ties to the lower index, NaN ranked as -inf, in chronological
 * order and -1 padded, to out_idx (device int32 [k_top]).  Errors: EINVAL for
 * NULL pointers or negative sizes. */
int cofie_topk(const float* w, int32_t n, int32_t k_top, int32_t* out_idx, void* stream);

/* Evidence preservation of a coarse filter (appendix, "Preservation of
 * Answer-Relevant Evidence"), with w the QER scores of the full, unfiltered
 * video used as attention mass (device float [n], e.g. the SOFTMAX mode) and
 * mask the frames the filter retains (device uint8 [n]):
 *   out[0]  Attention Preservation Ratio = sum of w over retained frames /
 *           sum of w (0 when that sum is 0)
 *   out[1]  Top-Evidence Recall = share of the top k = max(1, round(top_frac n))
 *           frames (as cofie_topk) that are retained; the paper uses 20 %
 * out: device double [2]; sums in fp64.  Errors: EINVAL for NULL pointers,
 * n < 0 or a negative or NaN top_frac. */
int cofie_evidence_preservation(const float* w, const uint8_t* mask, int32_t n, double top_frac, double* out,
                                void* stream);

/* ---- host helpers ------------------------------------------------------- */

/* k = max(1, round(rho * n_candidates)) (Eq. 8), rounding half to even;
 * 0 if n_candidates <= 0; -1 if rho is NaN or negative. */
int64_t cofie_qer_k_from_ratio(double rho, int64_t n_candidates);

/* Total drop ratio of the two stages, 1 - (1 - d_ngff)(1 - d_qer) (Sec. 4.1, Eq. 9). */
double cofie_drop_total(double d_ngff, double d_qer);

/* Message describing the calling thread's last error ("" if none). */
const char* cofie_last_error(void);

/* Library version string. */
const char* cofie_version(void);

/* ---- measurement -------------------------------------------------------- */

/* Kernel timing: when enabled, every kernel the library enqueues carries a
 * start/stop HIP event pair in its own dispatch (hipExtLaunchKernel), so
 * per-kernel durations are the kernels' own, on the GPU's clock.  cofie_profiler_read synchronises those events and
 * returns, for kernels whose name contains `name_substr`, the summed duration
 * (ms) and the number of launches.  Process-wide state; not for concurrent
 * use from several host threads. */
int cofie_profiler_enable(int on);
int cofie_profiler_reset(void);
int cofie_profiler_read(const char* name_substr, double* total_ms, int64_t* launches);

/* Host-side address check, for tests without a GPU.  cofie_debug_dry_run(1)
 * (per host thread; it also clears earlier results and buffers) makes the
 * entry points validate and plan as usual but launch nothing and make no HIP
 * call; instead every kernel with an address model walks each global and LDS
 * address its threads would touch, computed by the kernel's own index
 * functions, and checks it against the buffers registered with
 * cofie_debug_buffer (fake device addresses and their sizes: the caller's
 * inputs, outputs and workspace; the library allocates nothing in a dry run
 * when a workspace is given) and the launch's LDS.  Kernels with a model:
 * the QER score kernels (every mode), the operand-order query copy, the frame
 * means, the NGFF histograms and the frame gather; other launches are
 * skipped unchecked.
 * cofie_debug_dry_run_result returns the number of violations, the number of
 * accesses checked, and a description of the first violation.
 * cofie_debug_dry_run(0) ends the dry run. */
int cofie_debug_dry_run(int on);
int cofie_debug_buffer(const void* base, size_t bytes, const char* name);
/* As cofie_debug_buffer, for an input whose values decide addresses (frame
 * indices, frame offsets): `data` (host, `bytes` long, copied) is what the
 * fake buffer holds for the address models. */
int cofie_debug_buffer_data(const void* base, const void* data, size_t bytes, const char* name);
int64_t cofie_debug_dry_run_result(int64_t* checked, char* msg, size_t msg_bytes);

/* Streaming copy of `bytes` device bytes (16-byte aligned pointers): a plain
 * HBM read+write kernel used as a bandwidth and hardware-counter reference
 * for the measurement of the kernels above. */
int cofie_diag_stream_copy(const void* src, void* dst, size_t bytes, void* stream);

/* Streaming read of `bytes` device bytes (16-byte aligned): the attainable
 * read bandwidth, the ceiling of the read-dominated kernels above.  `sink`
 * (device, sink_words >= 256 words) receives per-thread XORs of the data. */
int cofie_diag_stream_read(const void* src, size_t bytes, uint32_t* sink, size_t sink_words,
                           void* stream);

#ifdef __cplusplus
}
#endif

#endif /* COFIE_H_ */

/*
 * CPU oracle for CoFiE's evidence-selection path (NGFF and QER).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or
 * load this file; only the test-suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no code, header, table or helper with
 * the HIP implementation.
 *
 * Every function is the plain definition (or, for the recursive keep rule,
 * the algorithm's steps in the paper's order), written as loops, in integer
 * arithmetic for NGFF and in fp64 for QER.  OpenMP only splits independent
 * outer loops (frames, visual tokens, candidate thresholds); it never changes
 * the arithmetic.
 *
 * Paper notation used below:
 *   h_t            normalised B-bin histogram of frame t      (Sec. 3.2)
 *   d(h_i,h_j)     total-variation distance 1/2 ||h_i-h_j||_1  (Sec. 3.2, Eq. 2)
 *   s_adj, s_ref   novelty terms against t-1 and r(t)          (Sec. 3.2, Eq. 3)
 *   s_NGFF         max of the two                              (Sec. 3.2, Eq. 4)
 *   r(t)           most recent candidate (kept) frame before t
 *   tau_h, L_max   keep rule thresholds                        (Sec. 3.2, Eq. 5)
 *   M_min          minimum-candidate safeguard                 (Sec. 3.2, gap-aware retention)
 *   a_ij           head-mean scaled dot product                (Sec. 3.3, Eq. 6)
 *   w_f            max-over-text, mean-over-frame score        (Sec. 3.3, Eq. 7)
 *   S_e            TopK of w_f                                 (Sec. 3.3, Eq. 8)
 *   o_i^h          causal softmax attention of the last layer, whose QK^T
 *                  tiles QER reads                            (Sec. 3.3)
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORC_GRAY = 0, ORC_PER_CHANNEL = 1, ORC_JOINT3D = 2 };
enum { ORC_F32 = 0, ORC_BF16 = 1 };
enum { ORC_LOGIT = 0, ORC_SOFTMAX = 1 };

int orc_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Threads of the parallel loops that follow (n >= 1); timing only. */
void orc_set_num_threads(int n) {
#ifdef _OPENMP
  if (n >= 1) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* ------------------------------------------------------------------------ */
/* NGFF: histograms (Sec. 3.2, "Lightweight histogram-based novelty")       */
/* ------------------------------------------------------------------------ */

/* Bin of an intensity v in [0,255] among B equal bins over the normalised
 * range [0,1]: the bin holding v/255, the value 1.0 folded into the last bin. */
static int bin_of(int v, int B) {
  int b = (v * B) / 255;
  return b < B - 1 ? b : B - 1;
}

/* Grayscale intensity of an RGB pixel: ITU-R BT.601 luma weights
 * 0.299/0.587/0.114, rounded to the nearest integer, in exact integers. */
static int gray_of(int r, int g, int b) { return (299 * r + 587 * g + 114 * b + 500) / 1000; }

int64_t orc_nbins(int32_t mode, int32_t B) {
  if (mode == ORC_GRAY) return B;
  if (mode == ORC_PER_CHANNEL) return 3 * (int64_t)B;
  return (int64_t)B * B * B;
}

/* Histogram mass M: the count total that normalises h_t to sum 1. */
int64_t orc_mass(int32_t mode, int32_t H, int32_t W) {
  int64_t N = (int64_t)H * W;
  return mode == ORC_PER_CHANNEL ? 3 * N : N;
}

/* counts[t][b] for n frames of layout [n][H][W][C] uint8 (C = 1 or 3).
 *   GRAY:        one B-bin histogram of the luma (C = 3) or of the value (C = 1)
 *   PER_CHANNEL: R, G, B histograms side by side: index c*B + bin(v_c)
 *   JOINT3D:     index (bin(r)*B + bin(g))*B + bin(b)                        */
int orc_histogram(const uint8_t* frames, int64_t n, int32_t H, int32_t W, int32_t C, int32_t B,
                  int32_t mode, uint32_t* counts) {
  const int64_t npix = (int64_t)H * W;
  const int64_t nb = orc_nbins(mode, B);
  if (C != 1 && C != 3) return -1;
  if (C == 1 && mode != ORC_GRAY) return -1;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t t = 0; t < n; ++t) {
    uint32_t* h = counts + t * nb;
    const uint8_t* f = frames + t * npix * C;
    memset(h, 0, (size_t)nb * sizeof(uint32_t));
    for (int64_t p = 0; p < npix; ++p) {
      const uint8_t* px = f + p * C;
      if (mode == ORC_GRAY) {
        int y = (C == 3) ? gray_of(px[0], px[1], px[2]) : px[0];
        h[bin_of(y, B)] += 1;
      } else if (mode == ORC_PER_CHANNEL) {
        for (int c = 0; c < 3; ++c) h[c * B + bin_of(px[c], B)] += 1;
      } else {
        int br = bin_of(px[0], B), bg = bin_of(px[1], B), bb = bin_of(px[2], B);
        h[((int64_t)br * B + bg) * B + bb] += 1;
      }
    }
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Alternative pre-encoder signals (Table 5, filtering-signal ablation)      */
/* ------------------------------------------------------------------------ */
/* The paper names them by citation only; the readings taken here:
 *   low-res frame difference: the luma image (gray_of, or the value for C = 1)
 *     box-averaged to a G x G grid, each cell's mean rounded half up to an
 *     integer in [0, 255]; the distance of two frames is the sum of the
 *     cells' absolute differences over 255 G^2 (the mean absolute difference
 *     of the low-resolution images, normalised to [0, 1]);
 *   dHash: the luma image box-averaged to 8 rows x 9 columns the same way;
 *     bit (r, c), c < 8, is set when cell (r, c + 1) is brighter than cell
 *     (r, c); the distance is the Hamming distance over 64.
 * Row y of an H-row image belongs to grid row (y * gh) div H (column x to
 * grid column (x * gw) div W), so the cells tile the image without overlap.
 * Each signal is written as a row of small integers whose L1 distance is the
 * numerator above (cell means for the frame difference, one 0/1 entry per
 * hash bit), so the keep rule of Eqs. 3-5 runs on them unchanged with
 * 2M = 255 G^2 or 64. */
enum { ORC_SIG_FRAMEDIFF = 3, ORC_SIG_DHASH = 4 };

/* Cell means (rounded half up) of the luma image on a gh x gw grid. */
static void cell_means(const uint8_t* f, int32_t H, int32_t W, int32_t C, int32_t gh, int32_t gw,
                       uint32_t* sum, uint32_t* area, uint32_t* mean) {
  for (int32_t i = 0; i < gh * gw; ++i) {
    sum[i] = 0;
    area[i] = 0;
  }
  for (int32_t y = 0; y < H; ++y) {
    const int32_t cy = (int32_t)(((int64_t)y * gh) / H);
    for (int32_t x = 0; x < W; ++x) {
      const int32_t cx = (int32_t)(((int64_t)x * gw) / W);
      const uint8_t* px = f + ((int64_t)y * W + x) * C;
      const int v = (C == 3) ? gray_of(px[0], px[1], px[2]) : px[0];
      sum[cy * gw + cx] += (uint32_t)v;
      area[cy * gw + cx] += 1;
    }
  }
  for (int32_t i = 0; i < gh * gw; ++i) mean[i] = (sum[i] + area[i] / 2) / area[i];
}

/* Signal rows [n][nsig] of n frames [n][H][W][C]: G^2 cell means (frame
 * difference, grid G) or 64 hash bits (dHash).  Returns nsig, or -1 for
 * shapes the signal does not define (a grid finer than the image). */
int64_t orc_signature(const uint8_t* frames, int64_t n, int32_t H, int32_t W, int32_t C, int32_t kind,
                      int32_t G, uint32_t* out) {
  if (C != 1 && C != 3) return -1;
  int32_t gh, gw;
  int64_t nsig;
  if (kind == ORC_SIG_FRAMEDIFF) {
    if (G < 1 || G > H || G > W) return -1;
    gh = gw = G;
    nsig = (int64_t)G * G;
  } else if (kind == ORC_SIG_DHASH) {
    if (H < 8 || W < 9) return -1;
    gh = 8;
    gw = 9;
    nsig = 64;
  } else {
    return -1;
  }
  const int64_t fb = (int64_t)H * W * C;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t t = 0; t < n; ++t) {
    uint32_t sum[4096], area[4096], mean[4096];
    cell_means(frames + t * fb, H, W, C, gh, gw, sum, area, mean);
    uint32_t* o = out + t * nsig;
    if (kind == ORC_SIG_FRAMEDIFF) {
      for (int64_t i = 0; i < nsig; ++i) o[i] = mean[i];
    } else {
      for (int r = 0; r < 8; ++r)
        for (int c = 0; c < 8; ++c) o[r * 8 + c] = mean[r * 9 + c + 1] > mean[r * 9 + c] ? 1u : 0u;
    }
  }
  return nsig;
}

/* The normaliser 2M of a signal's L1 distance: 255 G^2 or 64. */
int64_t orc_signal_two_m(int32_t kind, int32_t G) {
  return kind == ORC_SIG_FRAMEDIFF ? 255 * (int64_t)G * G : 64;
}

/* 2M * d(h_i,h_j) = sum_b |c_i[b] - c_j[b]| : the exact integer numerator of the
 * total-variation distance between two normalised histograms (Eq. 2). */
int64_t orc_l1(const uint32_t* ci, const uint32_t* cj, int64_t nbins) {
  int64_t D = 0;
  for (int64_t b = 0; b < nbins; ++b) {
    int64_t x = (int64_t)ci[b] - (int64_t)cj[b];
    D += x < 0 ? -x : x;
  }
  return D;
}

/* d = D / (2M), the exact quotient rounded once to the nearest fp32 (ties to
 * even).  Written from that definition in integers: with 2^-k <= D/N < 2^(1-k)
 * (N = 2M; D <= N + 1 and N < 2^31, so 0 <= k <= 31) the 24-bit significand
 * is floor(D 2^(23+k) / N), rounded up when twice the remainder exceeds N (or
 * equals it and the significand is odd).  While N < 2^24 this is what one IEEE
 * single division of the (then exact) operands returns. */
static float tv_q(int64_t D, int64_t N) {
  if (D <= 0) return 0.0f;
  int k = 0;
  while (((__int128)D << k) < N) ++k;
  const __int128 num = (__int128)D << (23 + k);
  int64_t m = (int64_t)(num / N);
  const __int128 twice_rem = 2 * (num - (__int128)m * N);
  if (twice_rem > N || (twice_rem == N && (m & 1))) ++m;
  if (m == (int64_t)1 << 24) {
    m >>= 1;
    --k;
  }
  return ldexpf((float)m, -(23 + k));
}
static float tv_of(int64_t D, int64_t mass) { return tv_q(D, 2 * mass); }

/* D / N correctly rounded to fp32 (for the pins of the rounding above). */
float orc_score(int64_t D, int64_t N) { return tv_q(D, N); }

/* ------------------------------------------------------------------------ */
/* NGFF: novelty score and gap-aware retention (Sec. 3.2, Eqs. 3-5)         */
/* ------------------------------------------------------------------------ */

/* One stream of T frames whose counts start at h.  Dtab, when non-NULL, holds
 * D(t, t-k) at Dtab[t*kmax + k-1] for 1 <= k <= kmax (kmax >= every gap the
 * scan can query); otherwise distances are computed from the histograms.
 *
 *   frame 0 is kept, s_0 := 1 (no predecessor), r := 0
 *   for t = 1 .. T-1:
 *       s_adj = d(h_t, h_{t-1});  s_ref = d(h_t, h_{r(t)});  s = max(s_adj, s_ref)
 *       keep t if t = T-1 (last frame), or s >= tau_h, or (L_max > 0 and t - r >= L_max)
 *       on keep (by this rule) r := t
 *   if fewer than M_min frames are kept (M_min >= 2), keep the M_min uniformly
 *   spaced frames floor(i (T-1) / (M_min-1)), i = 0 .. M_min-1.
 * Returns the number of kept frames.                                         */
static int64_t scan_stream(const uint32_t* h, const int64_t* Dtab, int64_t kmax, int64_t T,
                           int64_t nbins, int64_t mass, float tau_h, int32_t L_max, int32_t M_min,
                           float* scores, uint8_t* keep) {
  if (T <= 0) return 0;
  int64_t r = 0, kept = 1;
  keep[0] = 1;
  if (scores) scores[0] = 1.0f;
  for (int64_t t = 1; t < T; ++t) {
    int64_t Dadj, Dref;
    if (Dtab) {
      Dadj = Dtab[t * kmax + 0];
      Dref = Dtab[t * kmax + (t - r) - 1];
    } else {
      Dadj = orc_l1(h + t * nbins, h + (t - 1) * nbins, nbins);
      Dref = orc_l1(h + t * nbins, h + r * nbins, nbins);
    }
    float s_adj = tv_of(Dadj, mass);
    float s_ref = tv_of(Dref, mass);
    float s = s_adj > s_ref ? s_adj : s_ref;
    if (scores) scores[t] = s;
    int k = (t == T - 1) || (s >= tau_h) || (L_max > 0 && t - r >= L_max);
    keep[t] = (uint8_t)k;
    if (k) {
      r = t;
      ++kept;
    }
  }
  if (M_min >= 2 && kept < M_min) {
    for (int64_t i = 0; i < M_min; ++i) {
      int64_t u = (i * (T - 1)) / (M_min - 1);
      if (!keep[u]) {
        keep[u] = 1;
        ++kept;
      }
    }
  }
  return kept;
}

/* Band of exact distances for one stream: Dtab[t*kmax + k-1] = D(t, t-k). */
static int64_t* band_of(const uint32_t* h, int64_t T, int64_t nbins, int64_t kmax) {
  int64_t* Dtab = (int64_t*)calloc((size_t)(T > 0 ? T : 1) * (size_t)(kmax > 0 ? kmax : 1), sizeof(int64_t));
  if (!Dtab) return NULL;
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < T; ++t)
    for (int64_t k = 1; k <= kmax && k <= t; ++k)
      Dtab[t * kmax + k - 1] = orc_l1(h + t * nbins, h + (t - k) * nbins, nbins);
  return Dtab;
}

/* Keep rule over n frames cut into independent streams of seg_len frames
 * (seg_len <= 0: a single stream; the last stream may be shorter).  tau holds
 * one threshold per stream (n_tau = number of streams) or one for all
 * (n_tau = 1).  counts_out (optional) receives the kept count per stream.   */
int orc_ngff_select(const uint32_t* counts, int64_t n, int64_t nbins, int64_t mass, const float* tau,
                    int64_t n_tau, int32_t L_max, int32_t M_min, int64_t seg_len, float* scores,
                    uint8_t* mask, int64_t* counts_out) {
  if (seg_len <= 0 || seg_len > n) seg_len = n;
  if (n <= 0) return 0;
  int64_t nseg = (n + seg_len - 1) / seg_len;
  for (int64_t s = 0; s < nseg; ++s) {
    int64_t t0 = s * seg_len, T = (n - t0 < seg_len) ? n - t0 : seg_len;
    float tau_s = tau[n_tau > 1 ? s : 0];
    int64_t k = scan_stream(counts + t0 * nbins, NULL, 0, T, nbins, mass, tau_s, L_max, M_min,
                            scores + t0, mask + t0);
    if (counts_out) counts_out[s] = k;
  }
  return 0;
}

static int cmp_i64(const void* a, const void* b) {
  int64_t x = *(const int64_t*)a, y = *(const int64_t*)b;
  return (x > y) - (x < y);
}

/* Threshold calibration for a retention target (not in the paper, which takes
 * tau_h as given): per stream, the smallest integer threshold theta in
 *   Theta = {0} u {D(t,t-k) : 1 <= k <= L_max} u {2M+1}
 * whose keep rule, run with tau = fl32(theta)/fl32(2M), keeps at most `target`
 * frames, M_min top-up included.  The kept count is not monotone in theta
 * (r(t) depends on earlier decisions), so every candidate is evaluated.
 * Requires L_max >= 1.  theta_out / tau_out: one entry per stream.          */
int orc_ngff_calibrate(const uint32_t* counts, int64_t n, int64_t nbins, int64_t mass, int32_t L_max,
                       int32_t M_min, int64_t seg_len, int64_t target, int64_t* theta_out,
                       float* tau_out) {
  if (L_max < 1) return -1;
  if (seg_len <= 0 || seg_len > n) seg_len = n;
  if (n <= 0) return 0;
  int64_t nseg = (n + seg_len - 1) / seg_len;
  for (int64_t s = 0; s < nseg; ++s) {
    int64_t t0 = s * seg_len, T = (n - t0 < seg_len) ? n - t0 : seg_len;
    const uint32_t* h = counts + t0 * nbins;
    int64_t kmax = L_max;
    int64_t* Dtab = band_of(h, T, nbins, kmax);
    if (!Dtab) return -2;
    int64_t ncand = T * kmax + 2;
    int64_t* cand = (int64_t*)malloc((size_t)ncand * sizeof(int64_t));
    if (!cand) {
      free(Dtab);
      return -2;
    }
    int64_t m = 0;
    cand[m++] = 0;
    cand[m++] = 2 * mass + 1;
    for (int64_t t = 1; t < T; ++t)
      for (int64_t k = 1; k <= kmax && k <= t; ++k) cand[m++] = Dtab[t * kmax + k - 1];
    qsort(cand, (size_t)m, sizeof(int64_t), cmp_i64);
    int64_t u = 0;
    for (int64_t i = 0; i < m; ++i)
      if (u == 0 || cand[i] != cand[u - 1]) cand[u++] = cand[i];
    /* Evaluate every candidate (independently), then take the smallest that
     * meets the target; candidates are sorted ascending. */
    uint8_t* ok = (uint8_t*)calloc((size_t)u, 1);
    if (!ok) {
      free(cand);
      free(Dtab);
      return -2;
    }
#pragma omp parallel
    {
      uint8_t* keep = (uint8_t*)malloc((size_t)T);
#pragma omp for schedule(dynamic, 16)
      for (int64_t i = 0; i < u; ++i) {
        float tau = tv_of(cand[i], mass);
        int64_t kept = scan_stream(h, Dtab, kmax, T, nbins, mass, tau, L_max, M_min, NULL, keep);
        ok[i] = kept <= target;
      }
      free(keep);
    }
    /* 2M+1 leaves only the forced frames; if even they exceed the target the
     * answer is 2M+1. */
    int64_t theta = 2 * mass + 1;
    for (int64_t i = 0; i < u; ++i)
      if (ok[i]) {
        theta = cand[i];
        break;
      }
    free(ok);
    theta_out[s] = theta;
    tau_out[s] = tv_of(theta, mass);
    free(cand);
    free(Dtab);
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* QER: text-to-visual scores, frame aggregation, top-k (Sec. 3.3)           */
/* ------------------------------------------------------------------------ */

static double val_of(const void* base, int32_t dtype, int64_t i) {
  if (dtype == ORC_F32) return (double)((const float*)base)[i];
  uint32_t bits = (uint32_t)((const uint16_t*)base)[i] << 16; /* bf16 = top half of an fp32 */
  float f;
  memcpy(&f, &bits, sizeof f);
  return (double)f;
}

/* w[f] for frames given by CSR offsets (visual-token index set V_f =
 * [offs[f], offs[f+1])).  Q: [n_q][H_q][d], K: [n_vis][H_kv][d]; query head h
 * reads key head g(h) = floor(h * H_kv / H_q) (contiguous groups).
 *   LOGIT   a_ij = (1/H_q) sum_h scale * <q_i^h, k_j^g(h)>                (Eq. 6)
 *   SOFTMAX a_ij = (1/H_q) sum_h softmax_j'(scale * <q_i^h, k_j'^g(h)>)_j
 *           (normalised over all n_vis visual keys passed in)
 *   m_j = max_i a_ij;  w_f = (1/|V_f|) sum_{j in V_f} m_j, -inf if V_f empty (Eq. 7)
 * scale <= 0 selects 1/sqrt(d).                                              */
int orc_qer_scores(const void* Q, const void* K, int32_t dtype, const int32_t* offs, int32_t n_frames,
                   int32_t n_q, int32_t n_vis, int32_t H_q, int32_t H_kv, int32_t d, int32_t mode,
                   double scale, double* w) {
  if (scale <= 0) scale = 1.0 / sqrt((double)d);
  const int64_t qstride = (int64_t)H_q * d, kstride = (int64_t)H_kv * d;
  double* q = (double*)malloc((size_t)n_q * qstride * sizeof(double));
  double* m = (double*)malloc((size_t)(n_vis > 0 ? n_vis : 1) * sizeof(double));
  if (!q || !m) {
    free(q);
    free(m);
    return -2;
  }
  for (int64_t i = 0; i < (int64_t)n_q * qstride; ++i) q[i] = val_of(Q, dtype, i);

  double* rowmax = NULL; /* SOFTMAX: per (h,i) max and sum of exp over all j */
  double* rowsum = NULL;
  if (mode == ORC_SOFTMAX) {
    rowmax = (double*)malloc((size_t)H_q * n_q * sizeof(double));
    rowsum = (double*)malloc((size_t)H_q * n_q * sizeof(double));
    if (!rowmax || !rowsum) {
      free(q); free(m); free(rowmax); free(rowsum);
      return -2;
    }
#pragma omp parallel for collapse(2) schedule(static)
    for (int h = 0; h < H_q; ++h)
      for (int i = 0; i < n_q; ++i) {
        int g = (int)(((int64_t)h * H_kv) / H_q);
        double mx = -INFINITY;
        for (int j = 0; j < n_vis; ++j) {
          double s = 0;
          for (int x = 0; x < d; ++x)
            s += q[(int64_t)i * qstride + (int64_t)h * d + x] * val_of(K, dtype, (int64_t)j * kstride + (int64_t)g * d + x);
          s *= scale;
          if (s > mx) mx = s;
        }
        double z = 0;
        for (int j = 0; j < n_vis; ++j) {
          double s = 0;
          for (int x = 0; x < d; ++x)
            s += q[(int64_t)i * qstride + (int64_t)h * d + x] * val_of(K, dtype, (int64_t)j * kstride + (int64_t)g * d + x);
          z += exp(s * scale - mx);
        }
        rowmax[h * n_q + i] = mx;
        rowsum[h * n_q + i] = z;
      }
  }

#pragma omp parallel
  {
    double* k = (double*)malloc((size_t)kstride * sizeof(double));
#pragma omp for schedule(static)
    for (int j = 0; j < n_vis; ++j) {
      for (int64_t x = 0; x < kstride; ++x) k[x] = val_of(K, dtype, (int64_t)j * kstride + x);
      double mj = -INFINITY;
      for (int i = 0; i < n_q; ++i) {
        double a = 0;
        for (int h = 0; h < H_q; ++h) {
          int g = (int)(((int64_t)h * H_kv) / H_q);
          double dot = 0;
          for (int x = 0; x < d; ++x) dot += q[(int64_t)i * qstride + (int64_t)h * d + x] * k[(int64_t)g * d + x];
          if (mode == ORC_SOFTMAX)
            a += exp(dot * scale - rowmax[h * n_q + i]) / rowsum[h * n_q + i];
          else
            a += dot * scale;
        }
        a /= H_q;
        if (a > mj) mj = a;
      }
      m[j] = mj;
    }
    free(k);
  }

  for (int f = 0; f < n_frames; ++f) {
    int32_t lo = offs[f], hi = offs[f + 1];
    if (hi <= lo) {
      w[f] = -INFINITY;
      continue;
    }
    double s = 0;
    for (int32_t j = lo; j < hi; ++j) s += m[j];
    w[f] = s / (double)(hi - lo);
  }
  free(q);
  free(m);
  free(rowmax);
  free(rowsum);
  return 0;
}

/* S_e = TopK(w, k) (Eq. 8): order by score descending, ties by lower frame
 * index, NaN ranked as -inf; the k winners are returned in chronological
 * (ascending) order, the tail of idx (k_top > n) padded with -1.            */
int orc_topk(const double* w, int32_t n, int32_t k_top, int32_t* idx) {
  int32_t k = k_top < n ? k_top : n;
  uint8_t* taken = (uint8_t*)calloc((size_t)(n > 0 ? n : 1), 1);
  if (!taken) return -2;
  for (int32_t r = 0; r < k; ++r) {
    int32_t best = -1;
    double bv = 0;
    for (int32_t f = 0; f < n; ++f) {
      if (taken[f]) continue;
      double v = isnan(w[f]) ? -INFINITY : w[f];
      if (best < 0 || v > bv) {
        best = f;
        bv = v;
      }
    }
    taken[best] = 1;
  }
  int32_t o = 0;
  for (int32_t f = 0; f < n; ++f)
    if (taken[f]) idx[o++] = f;
  for (; o < k_top; ++o) idx[o] = -1;
  free(taken);
  return 0;
}

/* ---- coarse-to-fine glue ------------------------------------------------- */

/* The candidate set S_c that NGFF hands to the visual encoder (Sec. 3.1,
 * Sec. 3.2): the indices of the nonzero entries of mask[n], in increasing
 * (chronological) order, written to idx; and for each stream segment of
 * seg_len frames (seg_len = 0: one segment; the last may be shorter), the
 * number of candidates in the segments before it, seg_start[0..nseg], with
 * seg_start[nseg] the total.  Returns the total.                            */
int64_t orc_mask_compact(const uint8_t* mask, int64_t n, int64_t seg_len, int32_t* idx,
                         int32_t* seg_start) {
  const int64_t nseg = seg_len > 0 ? (n + seg_len - 1) / seg_len : 1;
  int64_t c = 0;
  for (int64_t s = 0; s < nseg; ++s) {
    seg_start[s] = (int32_t)c;
    const int64_t lo = seg_len > 0 ? s * seg_len : 0;
    const int64_t hi = seg_len > 0 && lo + seg_len < n ? lo + seg_len : n;
    for (int64_t t = lo; t < hi; ++t)
      if (mask[t]) idx[c++] = (int32_t)t;
  }
  seg_start[nseg] = (int32_t)c;
  return c;
}

/* Frame refinement (Sec. 3.3): frames outside S_e are removed from the token
 * sequence (hidden states, cached keys/values, positions) and the kept frames
 * stay in chronological order.  src holds n_rows rows of row_bytes bytes;
 * frame f owns rows [lo, hi) with lo = clamp(offs[f], 0, n_rows) and
 * hi = max(lo, clamp(offs[f+1], 0, n_rows)).  For i = 0..k-1 the rows of frame
 * sel[i] (none when sel[i] is outside [0, n_frames), e.g. the -1 padding of a
 * top-k) are appended to dst, at most dst_capacity rows being written;
 * out_offs[0..k] is the CSR of the appended rows (counted in full, so a total
 * beyond the capacity shows the shortfall) and out_rows[r] the source row of
 * dst row r (r < capacity).  Returns the total row count.                   */
int64_t orc_gather_frames(const uint8_t* src, int64_t n_rows, int64_t row_bytes, const int32_t* offs,
                          int32_t n_frames, const int32_t* sel, int32_t k, uint8_t* dst,
                          int64_t dst_capacity, int32_t* out_offs, int32_t* out_rows) {
  int64_t pos = 0;
  out_offs[0] = 0;
  for (int32_t i = 0; i < k; ++i) {
    const int32_t f = sel[i];
    if (f >= 0 && f < n_frames) {
      int64_t lo = offs[f], hi = offs[f + 1];
      lo = lo < 0 ? 0 : (lo > n_rows ? n_rows : lo);
      hi = hi < 0 ? 0 : (hi > n_rows ? n_rows : hi);
      if (hi < lo) hi = lo;
      for (int64_t r = lo; r < hi; ++r, ++pos) {
        if (pos < dst_capacity) {
          memcpy(dst + pos * row_bytes, src + r * row_bytes, (size_t)row_bytes);
          out_rows[pos] = (int32_t)r;
        }
      }
    }
    out_offs[i + 1] = (int32_t)pos;
  }
  return pos;
}

/* ---- NGFF as frames arrive ---------------------------------------------- */

/* The keep rule applied online (a reading of Sec. 3.2 for the streaming
 * setting of Sec. 3.1, where the video prefix grows): each frame is decided
 * when it arrives, by the rule of scan_stream except its two end-of-stream
 * safeguards (keep the last frame, the M_min top-up), which need the stream's
 * end and are applied by orc_ngff_finish.  One stream of T frames so far.
 * Returns the kept count; *r_out = the last kept frame.                     */
int64_t orc_ngff_scan_open(const uint32_t* h, int64_t T, int64_t nbins, int64_t mass, float tau_h,
                           int32_t L_max, float* scores, uint8_t* keep, int64_t* r_out) {
  int64_t r = 0, kept = 0;
  for (int64_t t = 0; t < T; ++t) {
    int k;
    if (t == 0) {
      scores[0] = 1.0f;
      k = 1;
    } else {
      const float s_adj = tv_of(orc_l1(h + t * nbins, h + (t - 1) * nbins, nbins), mass);
      const float s_ref = tv_of(orc_l1(h + t * nbins, h + r * nbins, nbins), mass);
      const float s = s_adj > s_ref ? s_adj : s_ref;
      scores[t] = s;
      k = (s >= tau_h) || (L_max > 0 && t - r >= L_max);
    }
    keep[t] = (uint8_t)k;
    if (k) {
      r = t;
      ++kept;
    }
  }
  if (r_out) *r_out = r;
  return kept;
}

/* End of a stream of T frames decided by orc_ngff_scan_open: the last frame
 * is kept, then, if fewer than M_min frames are kept (M_min >= 2), the frames
 * floor(i (T-1) / (M_min-1)) are added.  The frames this adds are written to
 * added[0..M_min] in increasing order, -1 padded.  Returns the kept count.  */
int64_t orc_ngff_finish(uint8_t* keep, int64_t T, int32_t M_min, int32_t* added) {
  const int32_t cap = (M_min > 0 ? M_min : 0) + 1;
  for (int32_t i = 0; i < cap; ++i) added[i] = -1;
  if (T <= 0) return 0;
  uint8_t* before = (uint8_t*)malloc((size_t)T);
  if (!before) return -1;
  memcpy(before, keep, (size_t)T);
  int64_t kept = 0;
  keep[T - 1] = 1;
  for (int64_t t = 0; t < T; ++t) kept += keep[t];
  if (M_min >= 2 && kept < M_min) {
    for (int64_t i = 0; i < M_min; ++i) {
      const int64_t u = (i * (T - 1)) / (M_min - 1);
      if (!keep[u]) {
        keep[u] = 1;
        ++kept;
      }
    }
  }
  int32_t a = 0;
  for (int64_t t = 0; t < T; ++t)
    if (keep[t] && !before[t]) added[a++] = (int32_t)t;
  free(before);
  return kept;
}

/* ---- evidence preservation (App., "Preservation of Answer-Relevant
 * Evidence") ------------------------------------------------------------- */

/* With w the QER scores of the full, unfiltered video (as an attention mass:
 * non-negative, e.g. the SOFTMAX mode) and mask the frames NGFF retains:
 *   APR      = sum of w over the retained frames / sum of w over all frames
 *              (0 when the total is 0)
 *   Recall@p = |TopK(w, k) intersected with the retained frames| / k, with
 *              k = max(1, round(p n)) (half to even), TopK as Eq. 8.
 * Sums in fp64 in frame order.                                              */
int orc_evidence_preservation(const double* w, const uint8_t* mask, int32_t n, double p, double* apr,
                              double* recall) {
  double tot = 0, kept = 0;
  for (int32_t f = 0; f < n; ++f) {
    tot += w[f];
    if (mask[f]) kept += w[f];
  }
  *apr = tot != 0 ? kept / tot : 0;
  *recall = 0;
  if (n <= 0) return 0;
  const double x = p * (double)n;
  int64_t k = (int64_t)nearbyint(x);
  if (k < 1) k = 1;
  if (k > n) k = n;
  int32_t* idx = (int32_t*)malloc((size_t)k * sizeof(int32_t));
  if (!idx) return -2;
  orc_topk(w, n, (int32_t)k, idx);
  int64_t hit = 0;
  for (int64_t i = 0; i < k; ++i) hit += mask[idx[i]] ? 1 : 0;
  *recall = (double)hit / (double)k;
  free(idx);
  return 0;
}

/* ---- last-layer prefill attention (the attention whose QK^T tiles QER
 * reads, Sec. 3.3) ------------------------------------------------------- */

/* Causal softmax attention of the listed query rows, every head, in fp64:
 *   s_ij = scale * <q_i^h, k_j^g(h)>            for j <= i (positions)
 *   o_i^h = sum_{j<=i} exp(s_ij - max_j s_ij) v_j^g(h) / sum_{j<=i} exp(...)
 * Q [L][H_q][d], K and V [L][H_kv][d] (dtype as orc_qer_scores); query head
 * h reads key/value head g(h) = floor(h * H_kv / H_q).  O receives
 * [n_rows][H_q][d] for the rows given (each in [0, L)).  scale <= 0 selects
 * 1/sqrt(d).                                                                */
int orc_attention_rows(const void* Q, const void* K, const void* V, int32_t dtype, int32_t L, int32_t H_q,
                       int32_t H_kv, int32_t d, double scale, const int32_t* rows, int32_t n_rows, double* O) {
  if (scale <= 0) scale = 1.0 / sqrt((double)d);
  const int64_t qstride = (int64_t)H_q * d, kstride = (int64_t)H_kv * d;
  for (int32_t r = 0; r < n_rows; ++r)
    if (rows[r] < 0 || rows[r] >= L) return -1;
  int rc = 0;
#pragma omp parallel
  {
    double* s = (double*)malloc((size_t)(L > 0 ? L : 1) * sizeof(double));
    if (!s) {
#pragma omp atomic write
      rc = -2;
    }
#pragma omp for collapse(2) schedule(dynamic, 1)
    for (int32_t r = 0; r < n_rows; ++r)
      for (int h = 0; h < H_q; ++h) {
        if (!s) continue;
        const int64_t i = rows[r];
        const int g = (int)(((int64_t)h * H_kv) / H_q);
        double mx = -INFINITY;
        for (int64_t j = 0; j <= i; ++j) {
          double dot = 0;
          for (int x = 0; x < d; ++x)
            dot += val_of(Q, dtype, i * qstride + (int64_t)h * d + x) * val_of(K, dtype, j * kstride + (int64_t)g * d + x);
          s[j] = dot * scale;
          if (s[j] > mx) mx = s[j];
        }
        double z = 0;
        for (int64_t j = 0; j <= i; ++j) {
          s[j] = exp(s[j] - mx);
          z += s[j];
        }
        double* o = O + ((int64_t)r * H_q + h) * d;
        for (int x = 0; x < d; ++x) {
          double acc = 0;
          for (int64_t j = 0; j <= i; ++j) acc += s[j] * val_of(V, dtype, j * kstride + (int64_t)g * d + x);
          o[x] = acc / z;
        }
      }
    free(s);
  }
  return rc;
}

/* vxo.c -- plain CPU fp64 oracle for page-centric sparse decode attention
 * (Vortex, arXiv 2606.06453).
 *
 * TEST INFRASTRUCTURE ONLY: it is loaded by the tests, the smoke check and the benchmark's
 * CPU-baseline leg, never by the product path.  It is deliberately slow and literal: every
 * function follows the paper's definition step by step, in fp64, with no blocking, fusion
 * or reordering.  OpenMP only spreads independent (request, KV head) units over cores; it
 * does not change any arithmetic.
 *
 * Pins (tests/test_oracle_*.py): summaries against numpy mean/max/min; the block-mean
 * score against the token-wise route it equals by linearity; Quest against its upper-bound
 * property and a hand-worked example; selection against brute force over all subsets;
 * attention with every page selected against torch's fp64 scaled-dot-product attention
 * with the GQA head mapping; layout invariance under page permutation and prefix sharing;
 * fp8 caches: every code against torch's OCP E4M3 / E5M2 decoding, the scaled value against
 * torch's fp32 product, the whole step against the bf16 step where the values are exact,
 * summaries and attention against torch on the cache values; the content-channel score
 * against the token-wise route on those channels; per-head logits against torch; NSA scores
 * against torch's softmax, conv1d and sum, and their mass and shift invariants; smoothing
 * against torch's conv1d.
 */
#include "vxo.h"

#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static __thread char g_err[256];

const char *vxo_error(void) { return g_err; }

int vxo_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

void vxo_set_num_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

static int fail(const char *msg, long a, long b) {
  snprintf(g_err, sizeof g_err, "%s (%ld, %ld)", msg, a, b);
  return 1;
}

/* bfloat16 is the upper half of an IEEE binary32; widening is exact. */
static double bf16(uint16_t h) {
  uint32_t bits = (uint32_t)h << 16;
  float f;
  memcpy(&f, &bits, sizeof f);
  return (double)f;
}

/* 8-bit floating-point KV caches (Sec. 5.3: precision support of the attention backends;
 * Appendix E: the fp8_e4m3 and fp8_e5m2 cache dtypes), in the
 * OCP 8-bit floating point formats:
 *   E4M3: sign, 4 exponent bits (bias 7), 3 mantissa bits; no infinities, S.1111.111 is NaN,
 *         largest finite value 448; exponent 0 is subnormal, value m/8 * 2^-6.
 *   E5M2: sign, 5 exponent bits (bias 15), 2 mantissa bits; exponent 31 holds +-inf (m = 0)
 *         and NaN (m != 0); exponent 0 is subnormal, value m/4 * 2^-14.
 * A cache entry's value is the fp32 product scale * code value (one rounding to nearest
 * even): the dequantised key or value that every later step uses. */
static double fp8_code_value(uint8_t c, int fmt) {
  int neg = c >> 7;
  double v;
  if (fmt == VXO_KV_FP8_E4M3) {
    int e = (c >> 3) & 15, m = c & 7;
    if (e == 15 && m == 7) return NAN;
    v = e ? ldexp(1.0 + m / 8.0, e - 7) : ldexp(m / 8.0, -6);
  } else {
    int e = (c >> 2) & 31, m = c & 3;
    if (e == 31) return m ? NAN : (neg ? -INFINITY : INFINITY);
    v = e ? ldexp(1.0 + m / 4.0, e - 15) : ldexp(m / 4.0, -14);
  }
  return neg ? -v : v;
}

static double fp8_dequant(uint8_t c, int fmt, float scale) {
  float x = scale * (float)fp8_code_value(c, fmt);   /* fp32 product, rounded to nearest even */
  return (double)x;
}

int vxo_fp8_dequantize(const uint8_t *codes, int64_t n, int fmt, float scale, float *out) {
  if (fmt != VXO_KV_FP8_E4M3 && fmt != VXO_KV_FP8_E5M2) return fail("bad fp8 format", fmt, 0);
  for (int64_t x = 0; x < n; x++) out[x] = (float)fp8_dequant(codes[x], fmt, scale);
  return 0;
}

/* Element idx of a K or V cache of the given dtype (bf16 bits, or fp8 codes with a scale). */
static double kv_value(const void *base, int64_t idx, int fmt, float scale) {
  if (fmt == VXO_KV_BF16) return bf16(((const uint16_t *)base)[idx]);
  return fp8_dequant(((const uint8_t *)base)[idx], fmt, scale);
}

/* Round an fp32-representable value to bfloat16, to nearest even (the precision at which
 * Max and Min summaries are stored; the identity on bf16 values). */
static double to_bf16_rne(double x) {
  float f = (float)x;
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  if (f != f) return x;
  u = (u + 0x7FFFu + ((u >> 16) & 1u)) & 0xFFFF0000u;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* Number of pages of request i (Sec. 3.1: the sequence is split into blocks of b tokens;
 * the last one may be partial, see the partial-block reading) and the valid tokens of
 * logical page j. */
static int num_pages(const int32_t *seq_lens, int i, int ps) { return (seq_lens[i] + ps - 1) / ps; }

static int valid_tokens(const int32_t *seq_lens, int i, int j, int ps) {
  int n = seq_lens[i] - j * ps;
  return n < ps ? n : ps;
}

static int check_batch(int batch, int ps, const int32_t *page_indptr, const int32_t *seq_lens) {
  if (page_indptr[0] != 0) return fail("page_indptr[0] must be 0", page_indptr[0], 0);
  for (int i = 0; i < batch; i++) {
    if (seq_lens[i] < 1) return fail("seq_lens must be >= 1", i, seq_lens[i]);
    int P = num_pages(seq_lens, i, ps);
    if (page_indptr[i + 1] - page_indptr[i] != P)
      return fail("page list length != ceil(seq_len / page_size)", i, page_indptr[i + 1] - page_indptr[i]);
  }
  return 0;
}

/* ---------------------------------------------------------------------------------------
 * Cache stage (Sec. 3.1, Eq. 1: block mean; Sec. 3.2 Quest: per-channel Max and Min).
 * For every requested logical page j of request i with physical page p and n valid tokens:
 *   Mean[p,h,c] = (1/n) sum_{t<n} K[p,h,t,c],  Max = max_t,  Min = min_t,
 * over the (dequantised) key values; Max and Min are stored in bf16 (exact for a bf16 cache).
 * A physical page shared by two requests (prefix sharing, Appendix A) must have the same
 * number of valid tokens in both. */
int vxo_summarize(const void *k, int kv_fmt, float k_scale, int64_t num_phys_pages, int H, int ps, int D,
                  int batch, const int32_t *page_indptr, const int32_t *page_indices,
                  const int32_t *seq_lens, const int32_t *first_page,
                  double *mean, double *maxv, double *minv) {
  if (check_batch(batch, ps, page_indptr, seq_lens)) return 1;
  if (kv_fmt != VXO_KV_BF16 && kv_fmt != VXO_KV_FP8_E4M3 && kv_fmt != VXO_KV_FP8_E5M2)
    return fail("bad kv format", kv_fmt, 0);
  int *n_of = (int *)malloc(sizeof(int) * (size_t)(num_phys_pages > 0 ? num_phys_pages : 1));
  for (int64_t p = 0; p < num_phys_pages; p++) n_of[p] = -1;
  for (int i = 0; i < batch; i++) {
    int P = num_pages(seq_lens, i, ps);
    for (int j = 0; j < P; j++) {
      int p = page_indices[page_indptr[i] + j];
      if (p < 0 || p >= num_phys_pages) { free(n_of); return fail("page id out of range", i, p); }
      int n = valid_tokens(seq_lens, i, j, ps);
      if (n_of[p] >= 0 && n_of[p] != n) { free(n_of); return fail("shared page with different valid counts", p, n); }
      n_of[p] = n;
    }
  }
  free(n_of);

  for (int i = 0; i < batch; i++) {
    int P = num_pages(seq_lens, i, ps);
    int j0 = first_page ? first_page[i] : 0;
    if (j0 < 0) j0 = 0;
#pragma omp parallel for schedule(dynamic)
    for (int j = j0; j < P; j++) {
      int64_t p = page_indices[page_indptr[i] + j];
      int n = valid_tokens(seq_lens, i, j, ps);
      for (int h = 0; h < H; h++) {
        for (int c = 0; c < D; c++) {
          double s = 0.0, mx = -INFINITY, mn = INFINITY;
          for (int t = 0; t < n; t++) {
            double x = kv_value(k, (((p * H) + h) * ps + t) * D + c, kv_fmt, k_scale);
            s += x;
            if (x > mx) mx = x;
            if (x < mn) mn = x;
          }
          int64_t o = (p * H + h) * D + c;
          if (mean) mean[o] = s / n;
          if (maxv) maxv[o] = to_bf16_rne(mx);
          if (minv) minv[o] = to_bf16_rne(mn);
        }
      }
    }
  }
  return 0;
}

/* ---------------------------------------------------------------------------------------
 * Cache stage at a decode step (Sec. 3.1: summaries are built with the cache and reused;
 * Appendix F: forward_cache runs per block): append the step's key and value rows, then
 * refresh the summaries of the page that received them.  Request i's new token is token
 * L_i - 1 (seq_lens already counts it): logical page j = (L_i - 1) / page_size, slot
 * (L_i - 1) mod page_size of physical page p = page_indices[page_indptr[i] + j]:
 *   K[p][h][slot][:] = k_new[i][h][:],  V[p][h][slot][:] = v_new[i][h][:]   (element copies)
 * then vxo_summarize over logical pages >= j.  v == NULL (V aliased, MLA) writes only K. */
int vxo_kv_append(void *k, void *v, int kv_fmt, int64_t num_phys_pages, int H, int ps, int Dqk, int Dv,
                  int batch, const int32_t *page_indptr, const int32_t *page_indices, const int32_t *seq_lens,
                  const void *k_new, const void *v_new) {
  if (check_batch(batch, ps, page_indptr, seq_lens)) return 1;
  size_t esz = kv_fmt == VXO_KV_BF16 ? 2 : 1;
  if (kv_fmt != VXO_KV_BF16 && kv_fmt != VXO_KV_FP8_E4M3 && kv_fmt != VXO_KV_FP8_E5M2)
    return fail("bad kv format", kv_fmt, 0);
  for (int i = 0; i < batch; i++) {
    int t = seq_lens[i] - 1;
    int j = t / ps, slot = t % ps;
    int64_t p = page_indices[page_indptr[i] + j];
    if (p < 0 || p >= num_phys_pages) return fail("page id out of range", i, p);
    for (int h = 0; h < H; h++) {
      memcpy((char *)k + ((((p * H) + h) * ps + slot) * Dqk) * esz,
             (const char *)k_new + (((int64_t)i * H + h) * Dqk) * esz, (size_t)Dqk * esz);
      if (v)
        memcpy((char *)v + ((((p * H) + h) * ps + slot) * Dv) * esz,
               (const char *)v_new + (((int64_t)i * H + h) * Dv) * esz, (size_t)Dv * esz);
    }
  }
  return 0;
}

/* ---------------------------------------------------------------------------------------
 * Indexer stage, scoring, for KV head h and its query heads G_h = {h*g, ..., h*g+g-1}:
 *   MEAN_DOT / MAX_DOT (Sec. 3.1, Eq. 2): s_j = mean over r in G_h of  q_r . S_j,
 *        with S = the block's Mean (block top-k) or Max summary.
 *   MEAN_DOT_CONTENT: Eq. 2 over the first Dc channels only.  On an MLA latent these are the
 *        compressed content channels; the decoupled rope channels are left out (the
 *        rope-unaware block-sparse flow of Sec. 6.2, analysed in the rope-component study of
 *        Sec. 6.3).  Other kinds score all D channels and ignore Dc.
 *   QUEST (Sec. 3.2, Quest): per head r, sum over channels of max(q_rc*Max_jc, q_rc*Min_jc),
 *        then the maximum over the heads of the group.
 * No 1/sqrt(d) factor: the block score has none. */
int vxo_score(int kind, const uint16_t *q, int Hq, int H, int D, int Dc, int ps,
              int batch, const int32_t *page_indptr, const int32_t *page_indices,
              const int32_t *seq_lens, const double *sa, const double *sb, double *scores) {
  if (check_batch(batch, ps, page_indptr, seq_lens)) return 1;
  if (H <= 0 || Hq % H != 0) return fail("Hq must be a multiple of H", Hq, H);
  int envelope = kind == VXO_QUEST || kind == VXO_QUEST_CONSENSUS || kind == VXO_ENVELOPE_LOWER ||
                 kind == VXO_QUEST_RECTIFIED;
  if (envelope && kind != VXO_QUEST_RECTIFIED && !sb) return fail("envelope score needs Max and Min summaries", kind, 0);
  if (!envelope && kind != VXO_MEAN_DOT && kind != VXO_MAX_DOT && kind != VXO_MEAN_DOT_CONTENT)
    return fail("bad kind", kind, 0);
  if (kind == VXO_MEAN_DOT_CONTENT && (Dc < 1 || Dc > D)) return fail("need 1 <= Dc <= D", Dc, D);
  int nch = kind == VXO_MEAN_DOT_CONTENT ? Dc : D;   /* channels that enter the dot products */
  int g = Hq / H;
  int units = batch * H;
#pragma omp parallel for schedule(dynamic)
  for (int u = 0; u < units; u++) {
    int i = u / H, h = u % H;
    int P = num_pages(seq_lens, i, ps);
    for (int j = 0; j < P; j++) {
      int64_t p = page_indices[page_indptr[i] + j];
      const double *S = sa + (p * H + h) * D;
      double s;
      if (kind == VXO_QUEST) {
        const double *Smin = sb + (p * H + h) * D;
        s = -INFINITY;
        for (int r = h * g; r < h * g + g; r++) {
          const uint16_t *qr = q + ((int64_t)i * Hq + r) * D;
          double acc = 0.0;
          for (int c = 0; c < D; c++) {
            double a = bf16(qr[c]) * S[c];
            double b = bf16(qr[c]) * Smin[c];
            acc += (a > b ? a : b);
          }
          if (acc > s) s = acc;
        }
      } else if (envelope) {
        /* Envelope flows of Appendix G over the per-channel Max / Min summaries, per head r:
         *   head-consensus Quest: sum_c max(q_rc Max_c, q_rc Min_c), then the MINIMUM over heads;
         *   pessimistic envelope: sum_c min(q_rc Max_c, q_rc Min_c), then the maximum over heads;
         *   rectified Quest:      sum_c ReLU(q_rc Max_c),            then the maximum over heads. */
        const double *Smin = kind == VXO_QUEST_RECTIFIED ? NULL : sb + (p * H + h) * D;
        s = kind == VXO_QUEST_CONSENSUS ? INFINITY : -INFINITY;
        for (int r = h * g; r < h * g + g; r++) {
          const uint16_t *qr = q + ((int64_t)i * Hq + r) * D;
          double acc = 0.0;
          for (int c = 0; c < D; c++) {
            double a = bf16(qr[c]) * S[c];
            if (kind == VXO_QUEST_RECTIFIED) {
              acc += a > 0.0 ? a : 0.0;
            } else {
              double b = bf16(qr[c]) * Smin[c];
              acc += kind == VXO_ENVELOPE_LOWER ? (a < b ? a : b) : (a > b ? a : b);
            }
          }
          if (kind == VXO_QUEST_CONSENSUS) {
            if (acc < s) s = acc;
          } else if (acc > s) {
            s = acc;
          }
        }
      } else {
        double total = 0.0;
        for (int r = h * g; r < h * g + g; r++) {
          const uint16_t *qr = q + ((int64_t)i * Hq + r) * D;
          double dot = 0.0;
          for (int c = 0; c < nch; c++) dot += bf16(qr[c]) * S[c];
          total += dot;
        }
        s = total / g;
      }
      scores[((int64_t)page_indptr[i] + j) * H + h] = s;
    }
  }
  return 0;
}

/* ---------------------------------------------------------------------------------------
 * Score flows built from the operator table's Softmax, Conv1d and Sum (NSA's block top-k
 * flow, Sec. 3.2: softmax of each query head's logits, convolution, head sum, top-K; positional
 * smoothing of Appendix G: the block-mean scores filtered over neighbouring pages).
 * Conv1d along the page axis of request i, zero padding, taps w[0..2]:
 *   y_j = w0 x_{j-1} + w1 x_j + w2 x_{j+1},  x_{-1} = x_{P_i} = 0
 * (the cross-correlation form, as in a deep-learning conv1d with padding 1). */
static void conv3_row(const double *x, int P, const double *w, double *y) {
  for (int j = 0; j < P; j++) {
    double left = j > 0 ? x[j - 1] : 0.0;
    double right = j + 1 < P ? x[j + 1] : 0.0;
    y[j] = w[0] * left + w[1] * x[j] + w[2] * right;
  }
}

/* Per-query-head block logits (the first step of the NSA flow): for query head r of KV
 * head h = r / g, z[r][j] = sum_c q_rc Mean_jc, summed in fp64 and rounded once to fp32, the
 * precision the indexer stores its scores in.  logits is ragged [page_indptr[batch]][Hq]. */
int vxo_head_logits(const uint16_t *q, int Hq, int H, int D, int ps, int batch,
                    const int32_t *page_indptr, const int32_t *page_indices, const int32_t *seq_lens,
                    const double *mean, double *logits) {
  if (check_batch(batch, ps, page_indptr, seq_lens)) return 1;
  if (H <= 0 || Hq % H != 0) return fail("Hq must be a multiple of H", Hq, H);
  int g = Hq / H;
#pragma omp parallel for schedule(dynamic)
  for (int i = 0; i < batch; i++) {
    int P = num_pages(seq_lens, i, ps);
    for (int j = 0; j < P; j++) {
      int64_t p = page_indices[page_indptr[i] + j];
      for (int r = 0; r < Hq; r++) {
        const double *S = mean + (p * H + r / g) * D;
        const uint16_t *qr = q + ((int64_t)i * Hq + r) * D;
        double dot = 0.0;
        for (int c = 0; c < D; c++) dot += bf16(qr[c]) * S[c];
        logits[((int64_t)page_indptr[i] + j) * Hq + r] = (double)(float)dot;
      }
    }
  }
  return 0;
}

/* NSA block scores: per request i, KV head h and query head r in G_h, the softmax over the
 * request's pages of z[r][.] (max-subtracted, fp64), then the 3-tap Conv1d above, then the
 * sum over the group's heads:
 *   p_rj = exp(z_rj - m_r) / sum_j' exp(z_rj' - m_r),  s_j = sum_{r in G_h} conv(p_r)_j.
 * scores is ragged [page_indptr[batch]][H]. */
int vxo_nsa_scores(const double *logits, int Hq, int H, int ps, int batch, const int32_t *page_indptr,
                   const int32_t *seq_lens, const double *taps, double *scores) {
  if (check_batch(batch, ps, page_indptr, seq_lens)) return 1;
  if (H <= 0 || Hq % H != 0) return fail("Hq must be a multiple of H", Hq, H);
  int g = Hq / H;
  int units = batch * H;
#pragma omp parallel for schedule(dynamic)
  for (int u = 0; u < units; u++) {
    int i = u / H, h = u % H;
    int P = num_pages(seq_lens, i, ps);
    double *prob = (double *)malloc(sizeof(double) * (size_t)P);
    double *conv = (double *)malloc(sizeof(double) * (size_t)P);
    double *sum = (double *)calloc((size_t)P, sizeof(double));
    for (int r = h * g; r < h * g + g; r++) {
      double m = -INFINITY;
      for (int j = 0; j < P; j++) {
        double z = logits[((int64_t)page_indptr[i] + j) * Hq + r];
        if (z > m) m = z;
      }
      double l = 0.0;
      for (int j = 0; j < P; j++) {
        prob[j] = exp(logits[((int64_t)page_indptr[i] + j) * Hq + r] - m);
        l += prob[j];
      }
      for (int j = 0; j < P; j++) prob[j] /= l;
      conv3_row(prob, P, taps, conv);
      for (int j = 0; j < P; j++) sum[j] += conv[j];
    }
    for (int j = 0; j < P; j++) scores[((int64_t)page_indptr[i] + j) * H + h] = sum[j];
    free(prob);
    free(conv);
    free(sum);
  }
  return 0;
}

/* Positional smoothing (Appendix G): block scores convolved along the page axis of each
 * request with the 3-tap Conv1d above.  in and out are ragged [page_indptr[batch]][H]. */
int vxo_smooth_scores(const double *in, int H, int ps, int batch, const int32_t *page_indptr,
                      const int32_t *seq_lens, const double *taps, double *out) {
  if (check_batch(batch, ps, page_indptr, seq_lens)) return 1;
  int units = batch * H;
#pragma omp parallel for schedule(dynamic)
  for (int u = 0; u < units; u++) {
    int i = u / H, h = u % H;
    int P = num_pages(seq_lens, i, ps);
    double *x = (double *)malloc(sizeof(double) * (size_t)P);
    double *y = (double *)malloc(sizeof(double) * (size_t)P);
    for (int j = 0; j < P; j++) x[j] = in[((int64_t)page_indptr[i] + j) * H + h];
    conv3_row(x, P, taps, y);
    for (int j = 0; j < P; j++) out[((int64_t)page_indptr[i] + j) * H + h] = y[j];
    free(x);
    free(y);
  }
  return 0;
}

/* ---------------------------------------------------------------------------------------
 * Indexer stage, selection (Sec. 3.1, Eq. 3 top-k over block scores; Sec. 6.4 setup:
 * the first block and the most recent blocks are always attended).
 *   F = {0..n_sink-1} U {P-n_local..P-1};  K_total = min(budget, max_sel).
 *   K_total >= P: every page.  Otherwise the K_free = max(0, K_total - |F|) best pages of
 *   the candidates [0,P) \ F, best meaning larger score, ties to the lower page index.
 *   Output F U top in ascending order. */
typedef struct {
  double s;
  int j;
} cand_t;

static int cand_cmp(const void *a, const void *b) {
  const cand_t *x = (const cand_t *)a, *y = (const cand_t *)b;
  if (x->s > y->s) return -1;
  if (x->s < y->s) return 1;
  return (x->j > y->j) - (x->j < y->j);
}

int vxo_select(const double *scores, int H, int ps, int batch,
               const int32_t *page_indptr, const int32_t *seq_lens, const int32_t *pages_budget,
               int n_sink, int n_local, int max_sel, int32_t *sel_pages, int32_t *sel_count,
               double *s_kth, double *s_next) {
  if (check_batch(batch, ps, page_indptr, seq_lens)) return 1;
  if (n_sink < 0 || n_local < 0 || n_sink + n_local > max_sel) return fail("need 0 <= n_sink + n_local <= max_sel", n_sink, n_local);
  int units = batch * H;
  int bad = 0;
#pragma omp parallel for schedule(dynamic)
  for (int u = 0; u < units; u++) {
    int i = u / H, h = u % H;
    int P = num_pages(seq_lens, i, ps);
    int Ktot = pages_budget[i] < max_sel ? pages_budget[i] : max_sel;
    if (Ktot < 0) Ktot = 0;
    int32_t *out = sel_pages + (int64_t)u * max_sel;
    for (int m = 0; m < max_sel; m++) out[m] = -1;
    char *chosen = (char *)calloc((size_t)P, 1);
    double kth = INFINITY, next = -INFINITY;
    if (Ktot >= P) {
      for (int j = 0; j < P; j++) chosen[j] = 1;
    } else {
      int nF = 0;
      for (int j = 0; j < P; j++) {
        if (j < n_sink || j >= P - n_local) { chosen[j] = 1; nF++; }
      }
      int Kfree = Ktot - nF;
      if (Kfree < 0) Kfree = 0;
      cand_t *c = (cand_t *)malloc(sizeof(cand_t) * (size_t)(P > 0 ? P : 1));
      int nc = 0;
      for (int j = 0; j < P; j++) {
        if (!chosen[j]) {
          c[nc].s = scores[((int64_t)page_indptr[i] + j) * H + h];
          c[nc].j = j;
          nc++;
        }
      }
      qsort(c, (size_t)nc, sizeof(cand_t), cand_cmp);
      for (int m = 0; m < Kfree && m < nc; m++) chosen[c[m].j] = 1;
      if (Kfree >= 1 && Kfree <= nc) kth = c[Kfree - 1].s;
      if (Kfree < nc) next = c[Kfree].s;
      free(c);
    }
    int cnt = 0;
    for (int j = 0; j < P; j++) {
      if (chosen[j]) {
        if (cnt < max_sel) out[cnt] = j;
        cnt++;
      }
    }
    free(chosen);
    if (cnt > max_sel) {
#pragma omp atomic write
      bad = 1;
    }
    if (h == 0) sel_count[i] = cnt;
    if (s_kth) s_kth[u] = kth;
    if (s_next) s_next[u] = next;
  }
  if (bad) return fail("selection larger than max_sel", 0, 0);
  return 0;
}

/* ---------------------------------------------------------------------------------------
 * Approximate radix top-k (Sec. 5.2: stochastic early termination; Appendix D: remapping and
 * the tolerate ratio of approxTopK in the operator table).  Selection semantics as in
 * vxo_select (forced pages F, K_free best candidates, output ascending), over fp32 scores
 * stored [H][batch][stride]: the scores of (request i, head h) are row h*batch + i, pages
 * 0 .. num_items[i]-1.
 *
 * The result is defined from the sorted keys, pass boundary by pass boundary (no histogram
 * walk), for one (request, head) with K_free > 0:
 *  1. Key of each candidate.  remap 0: the order-preserving 32-bit key of the fp32 score
 *     (larger score, larger key; -0.0 as +0.0; NaN lowest).  remap 1: the monotone affine map
 *     of the candidates' [min, max] onto 32-bit fixed point, floor((s - min) * scale) with
 *     scale = 4294967295 / (max - min) in fp64 (0 when max == min).
 *  2. T = the K_free-th largest candidate key.  A radix select reads 8-bit digits, most
 *     significant first, starting at the highest bit t0 in which the smallest and largest
 *     candidate keys differ; after its p-th pass every bit at or above b_p is resolved, with
 *     b_1 = max(t0 - 7, 0) and b_{p+1} = max(b_p - 8, 0).
 *  3. After pass p, with M_p the mask of bits >= b_p: candidates whose masked key exceeds
 *     T & M_p are certain members (c_p of them); those whose masked key equals it form the
 *     threshold bin (n_p of them); K_free - c_p members are still needed from the bin.
 *  4. The walk ends at the first pass p where
 *       n_p == K_free - c_p            (the whole bin is needed), or
 *       b_p == 0                       (every bit resolved), or
 *       b_p > 0 and c_p * 65536 >= (65536 - tau_q) * K_free   (early termination),
 *     with tau_q = round(65536 tau) computed in fp32 (the tolerate ratio in 16-bit fixed
 *     point, so the test is exact integer arithmetic).  tau = 0 never terminates early.
 *  5. Members: the certain candidates, plus the first K_free - c_p bin members in an order:
 *     ascending page index when the walk ended without early termination (equal keys go to
 *     the lower page, as in the exact selection); after an early termination a random order,
 *     the bin members sorted by a seeded 8-bit hash, larger first, equal hashes in page order:
 *       h8(j) = lowbias32(z ^ j) >> 24,   z = lowbias32(seed ^ lowbias32(i * H + h)).
 *  If every candidate key is equal (no pass), the members are the K_free lowest pages.
 * lowbias32 is C. Wellons' 32-bit integer hash (hash-prospector): x ^= x >> 16;
 * x *= 0x7feb352d; x ^= x >> 15; x *= 0x846ca68b; x ^= x >> 16.
 * ------------------------------------------------------------------------------------- */
static uint32_t lowbias32(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}

static uint32_t order_key(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if (f != f) return 0;                   /* NaN lowest */
  if (u == 0x80000000u) u = 0;            /* -0.0 as +0.0 */
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

/* (value, page) pairs: sorted by value descending, then page ascending */
typedef struct {
  uint32_t v;
  int j;
} vxo_vj;

static int vj_desc(const void *a, const void *b) {
  const vxo_vj *x = (const vxo_vj *)a, *y = (const vxo_vj *)b;
  if (x->v != y->v) return x->v < y->v ? 1 : -1;
  return x->j < y->j ? -1 : (x->j > y->j);
}

int vxo_topk_select(const float *scores, int stride, int H, int batch, const int32_t *num_items,
                    const int32_t *pages_budget, int n_sink, int n_local, int max_sel, float tau,
                    uint32_t seed, int remap, int32_t *sel_pages, int32_t *sel_count) {
  if (n_sink < 0 || n_local < 0 || n_sink + n_local > max_sel) return fail("need 0 <= n_sink + n_local <= max_sel", n_sink, n_local);
  if (!(tau >= 0.0f && tau <= 1.0f)) return fail("tau must be in [0, 1]", 0, 0);
  const int64_t tau_q = (int64_t)lroundf(tau * 65536.0f);
  if (remap != 0 && remap != 1) return fail("remap must be 0 or 1", remap, 0);
  for (int i = 0; i < batch; i++)
    if (num_items[i] < 0 || num_items[i] > stride) return fail("num_items out of [0, stride]", i, num_items[i]);
  int units = batch * H;
  int bad = 0;
#pragma omp parallel for schedule(dynamic)
  for (int u = 0; u < units; u++) {
    int i = u % batch, h = u / batch;     /* scores row h*batch + i */
    int P = num_items[i];
    const float *s = scores + ((int64_t)h * batch + i) * stride;
    int Ktot = pages_budget[i] < max_sel ? pages_budget[i] : max_sel;
    if (Ktot < 0) Ktot = 0;
    int32_t *out = sel_pages + ((int64_t)i * H + h) * max_sel;
    for (int m = 0; m < max_sel; m++) out[m] = -1;
    size_t n1 = (size_t)(P > 0 ? P : 1);
    char *chosen = (char *)calloc(n1, 1);
    vxo_vj *kl = (vxo_vj *)malloc(sizeof(vxo_vj) * n1);
    vxo_vj *bin = (vxo_vj *)malloc(sizeof(vxo_vj) * n1);
    if (Ktot >= P) {
      for (int j = 0; j < P; j++) chosen[j] = 1;
    } else {
      int nF = 0, nc = 0;
      for (int j = 0; j < P; j++) {
        const int forced = j < n_sink || P - j <= n_local;   /* sink or local page */
        if (forced) { chosen[j] = 1; nF++; }
        else kl[nc++].j = j;
      }
      int Kfree = Ktot - nF;
      if (Kfree < 0) Kfree = 0;
      /* step 1: keys */
      double mn = INFINITY, mx = -INFINITY;
      for (int m = 0; m < nc; m++) {
        float x = s[kl[m].j];
        kl[m].v = order_key(x);
        if (x == x) {
          if ((double)x < mn) mn = (double)x;
          if ((double)x > mx) mx = (double)x;
        }
      }
      if (remap == 1) {
        double scale = mx > mn ? 4294967295.0 / (mx - mn) : 0.0;
        for (int m = 0; m < nc; m++) {
          float x = s[kl[m].j];
          kl[m].v = (x == x) ? (uint32_t)floor(((double)x - mn) * scale) : 0u;
        }
      }
      if (Kfree > 0) {   /* here nc > Kfree: Ktot < P */
        /* step 2: the K_free-th largest key and the first pass boundary */
        qsort(kl, (size_t)nc, sizeof(vxo_vj), vj_desc);
        const uint32_t T = kl[Kfree - 1].v;
        const uint32_t diff = kl[0].v ^ kl[nc - 1].v;
        int t0 = -1;
        for (int bit = 31; bit >= 0; bit--) if ((diff >> bit) & 1u) { t0 = bit; break; }
        /* steps 3-4: the first pass boundary that ends the walk */
        uint32_t M = 0xffffffffu;          /* no pass: every key equal */
        int early = 0;
        if (t0 >= 0) {
          int b = t0 >= 7 ? t0 - 7 : 0;
          for (;;) {
            M = 0xffffffffu << b;
            int c = 0, n = 0;
            for (int m = 0; m < nc; m++) {
              uint32_t mk = kl[m].v & M;
              if (mk > (T & M)) c++;
              else if (mk == (T & M)) n++;
            }
            if (n == Kfree - c || b == 0) break;
            if ((int64_t)c * 65536 >= (65536 - tau_q) * Kfree) { early = 1; break; }
            b = b >= 8 ? b - 8 : 0;
          }
        }
        /* step 5: certain members, then the bin in its order */
        int c = 0, nb = 0;
        const uint32_t z = lowbias32(seed ^ lowbias32((uint32_t)(i * H + h)));
        for (int m = 0; m < nc; m++) {
          uint32_t mk = kl[m].v & M;
          if (mk > (T & M)) {
            chosen[kl[m].j] = 1;
            c++;
          } else if (mk == (T & M)) {
            bin[nb].j = kl[m].j;
            bin[nb].v = early ? lowbias32(z ^ (uint32_t)kl[m].j) >> 24 : 0u;
            nb++;
          }
        }
        qsort(bin, (size_t)nb, sizeof(vxo_vj), vj_desc);
        for (int m = 0; m < Kfree - c && m < nb; m++) chosen[bin[m].j] = 1;
      }
    }
    int cnt = 0;
    for (int j = 0; j < P; j++) {
      if (chosen[j]) {
        if (cnt < max_sel) out[cnt] = j;
        cnt++;
      }
    }
    free(chosen);
    free(kl);
    free(bin);
    if (cnt > max_sel) {
#pragma omp atomic write
      bad = 1;
    }
    if (h == 0) sel_count[i] = cnt;
  }
  if (bad) return fail("selection larger than max_sel", 0, 0);
  return 0;
}

/* ---------------------------------------------------------------------------------------
 * Sparse attention (Sec. 3.1, Eq. 4): for each query head r of KV head h,
 *   z_t = sm_scale * q_r . k_t over the valid tokens t of the selected pages,
 *   o_r = sum_t softmax(z)_t v_t.
 * MLA with absorbed weights (Sec. 6.2): V is the first Dv channels of the shared latent.
 * k_t and v_t are the (dequantised) cache values. */
int vxo_attend(const uint16_t *q, int Hq, const void *k, const void *v, int kv_fmt, float k_scale,
               float v_scale, int H, int ps, int Dqk, int Dv, int batch, const int32_t *page_indptr,
               const int32_t *page_indices, const int32_t *seq_lens, const int32_t *sel_pages,
               const int32_t *sel_count, int max_sel, double sm_scale, double *out) {
  if (check_batch(batch, ps, page_indptr, seq_lens)) return 1;
  if (kv_fmt != VXO_KV_BF16 && kv_fmt != VXO_KV_FP8_E4M3 && kv_fmt != VXO_KV_FP8_E5M2)
    return fail("bad kv format", kv_fmt, 0);
  if (H <= 0 || Hq % H != 0) return fail("Hq must be a multiple of H", Hq, H);
  if (!v && Dv > Dqk) return fail("aliased V needs Dv <= Dqk", Dv, Dqk);
  int g = Hq / H;
  int units = batch * H;
  int bad = 0;
#pragma omp parallel for schedule(dynamic)
  for (int u = 0; u < units; u++) {
    int i = u / H, h = u % H;
    int P = num_pages(seq_lens, i, ps);
    int cnt = sel_count[i];
    const int32_t *sel = sel_pages + (int64_t)u * max_sel;
    /* gather the selected tokens (physical page, slot) */
    int64_t ntok = 0;
    for (int m = 0; m < cnt; m++) {
      int j = sel[m];
      if (j < 0 || j >= P) {
#pragma omp atomic write
        bad = 1;
        continue;
      }
      ntok += valid_tokens(seq_lens, i, j, ps);
    }
    int64_t *row_k = (int64_t *)malloc(sizeof(int64_t) * (size_t)(ntok > 0 ? ntok : 1));
    int64_t *row_v = (int64_t *)malloc(sizeof(int64_t) * (size_t)(ntok > 0 ? ntok : 1));
    int64_t t_all = 0;
    for (int m = 0; m < cnt; m++) {
      int j = sel[m];
      if (j < 0 || j >= P) continue;
      int64_t p = page_indices[page_indptr[i] + j];
      int n = valid_tokens(seq_lens, i, j, ps);
      for (int t = 0; t < n; t++) {
        row_k[t_all] = (((p * H) + h) * ps + t) * Dqk;
        row_v[t_all] = v ? (((p * H) + h) * ps + t) * Dv : row_k[t_all];
        t_all++;
      }
    }
    double *z = (double *)malloc(sizeof(double) * (size_t)(ntok > 0 ? ntok : 1));
    const void *vsrc = v ? v : k;
    const float vs = v ? v_scale : k_scale;
    for (int r = h * g; r < h * g + g; r++) {
      const uint16_t *qr = q + ((int64_t)i * Hq + r) * Dqk;
      double *o = out + ((int64_t)i * Hq + r) * Dv;
      for (int c = 0; c < Dv; c++) o[c] = 0.0;
      if (ntok == 0) continue;
      double zmax = -INFINITY;
      for (int64_t t = 0; t < ntok; t++) {
        double dot = 0.0;
        for (int c = 0; c < Dqk; c++) dot += bf16(qr[c]) * kv_value(k, row_k[t] + c, kv_fmt, k_scale);
        z[t] = sm_scale * dot;
        if (z[t] > zmax) zmax = z[t];
      }
      double wsum = 0.0;
      for (int64_t t = 0; t < ntok; t++) {
        z[t] = exp(z[t] - zmax);
        wsum += z[t];
      }
      for (int64_t t = 0; t < ntok; t++) {
        double w = z[t] / wsum;
        for (int c = 0; c < Dv; c++) o[c] += w * kv_value(vsrc, row_v[t] + c, kv_fmt, vs);
      }
    }
    free(z);
    free(row_k);
    free(row_v);
  }
  if (bad) return fail("selected page id out of range", 0, 0);
  return 0;
}

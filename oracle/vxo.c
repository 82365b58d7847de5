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
 * with the GQA head mapping; layout invariance under page permutation and prefix sharing.
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
 *   Mean[p,h,c] = (1/n) sum_{t<n} K[p,h,t,c],  Max = max_t,  Min = min_t.
 * A physical page shared by two requests (prefix sharing, Appendix A) must have the same
 * number of valid tokens in both. */
int vxo_summarize(const uint16_t *k, int64_t num_phys_pages, int H, int ps, int D,
                  int batch, const int32_t *page_indptr, const int32_t *page_indices,
                  const int32_t *seq_lens, const int32_t *first_page,
                  double *mean, double *maxv, double *minv) {
  if (check_batch(batch, ps, page_indptr, seq_lens)) return 1;
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
            double x = bf16(k[(((p * H) + h) * ps + t) * D + c]);
            s += x;
            if (x > mx) mx = x;
            if (x < mn) mn = x;
          }
          int64_t o = (p * H + h) * D + c;
          if (mean) mean[o] = s / n;
          if (maxv) maxv[o] = mx;
          if (minv) minv[o] = mn;
        }
      }
    }
  }
  return 0;
}

/* ---------------------------------------------------------------------------------------
 * Indexer stage, scoring, for KV head h and its query heads G_h = {h*g, ..., h*g+g-1}:
 *   MEAN_DOT / MAX_DOT (Sec. 3.1, Eq. 2): s_j = mean over r in G_h of  q_r . S_j,
 *        with S = the block's Mean (block top-k) or Max summary.
 *   QUEST (Sec. 3.2, Quest): per head r, sum over channels of max(q_rc*Max_jc, q_rc*Min_jc),
 *        then the maximum over the heads of the group.
 * No 1/sqrt(d) factor: the block score has none. */
int vxo_score(int kind, const uint16_t *q, int Hq, int H, int D, int ps,
              int batch, const int32_t *page_indptr, const int32_t *page_indices,
              const int32_t *seq_lens, const double *sa, const double *sb, double *scores) {
  if (check_batch(batch, ps, page_indptr, seq_lens)) return 1;
  if (H <= 0 || Hq % H != 0) return fail("Hq must be a multiple of H", Hq, H);
  if (kind == VXO_QUEST && !sb) return fail("Quest needs Max and Min summaries", 0, 0);
  if (kind != VXO_MEAN_DOT && kind != VXO_QUEST && kind != VXO_MAX_DOT) return fail("bad kind", kind, 0);
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
      } else {
        double total = 0.0;
        for (int r = h * g; r < h * g + g; r++) {
          const uint16_t *qr = q + ((int64_t)i * Hq + r) * D;
          double dot = 0.0;
          for (int c = 0; c < D; c++) dot += bf16(qr[c]) * S[c];
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
 * Sparse attention (Sec. 3.1, Eq. 4): for each query head r of KV head h,
 *   z_t = sm_scale * q_r . k_t over the valid tokens t of the selected pages,
 *   o_r = sum_t softmax(z)_t v_t.
 * MLA with absorbed weights (Sec. 6.2): V is the first Dv channels of the shared latent. */
int vxo_attend(const uint16_t *q, int Hq, const uint16_t *k, const uint16_t *v, int H,
               int ps, int Dqk, int Dv, int batch, const int32_t *page_indptr,
               const int32_t *page_indices, const int32_t *seq_lens, const int32_t *sel_pages,
               const int32_t *sel_count, int max_sel, double sm_scale, double *out) {
  if (check_batch(batch, ps, page_indptr, seq_lens)) return 1;
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
    const uint16_t *vsrc = v ? v : k;
    for (int r = h * g; r < h * g + g; r++) {
      const uint16_t *qr = q + ((int64_t)i * Hq + r) * Dqk;
      double *o = out + ((int64_t)i * Hq + r) * Dv;
      for (int c = 0; c < Dv; c++) o[c] = 0.0;
      if (ntok == 0) continue;
      double zmax = -INFINITY;
      for (int64_t t = 0; t < ntok; t++) {
        double dot = 0.0;
        for (int c = 0; c < Dqk; c++) dot += bf16(qr[c]) * bf16(k[row_k[t] + c]);
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
        for (int c = 0; c < Dv; c++) o[c] += w * bf16(vsrc[row_v[t] + c]);
      }
    }
    free(z);
    free(row_k);
    free(row_v);
  }
  if (bad) return fail("selected page id out of range", 0, 0);
  return 0;
}

/* vxo.h -- plain CPU fp64 oracle for page-centric sparse decode attention
 * (Vortex, arXiv 2606.06453).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may load this library.  It shares no code, header, table or constant
 * with the HIP path.
 *
 * All pointers are host pointers.  bf16 tensors are passed as their raw 16-bit patterns.
 * Every bf16 value is widened exactly to fp64 and all arithmetic is fp64.
 *
 * Layouts (paged layout, Appendix A):
 *   k           [num_phys_pages][H][page_size][Dqk]   bf16 bits
 *   v           [num_phys_pages][H][page_size][Dv]    bf16 bits, or NULL: V_t = K_t[0:Dv] (MLA)
 *   q           [batch][Hq][Dqk]                      bf16 bits
 *   page_indptr [batch+1], page_indices [page_indptr[batch]] physical page ids
 *   seq_lens    [batch]  tokens incl. the current one; P_i = ceil(seq_lens[i] / page_size)
 *               must equal page_indptr[i+1] - page_indptr[i].
 * Query head r belongs to KV head r / g, g = Hq / H.
 *
 * Return value: 0 on success, nonzero on a violated precondition (message in vxo_error()).
 */
#ifndef VXO_H
#define VXO_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define VXO_MEAN_DOT 0
#define VXO_QUEST 1
#define VXO_MAX_DOT 2

const char *vxo_error(void);
int vxo_num_threads(void);

/* Cache stage: per-page Mean / Max / Min of keys over the page's valid tokens.
 * Summaries are written for logical pages j >= first_page[i] (all pages when first_page is
 * NULL), at [phys][H][Dqk].  Each output may be NULL. */
int vxo_summarize(const uint16_t *k, int64_t num_phys_pages, int H, int page_size, int Dqk,
                  int batch, const int32_t *page_indptr, const int32_t *page_indices,
                  const int32_t *seq_lens, const int32_t *first_page,
                  double *mean, double *maxv, double *minv);

/* Indexer stage, scoring.  scores is ragged: [page_indptr[batch]][H], row page_indptr[i]+j.
 * MEAN_DOT: sa = Mean summaries, MAX_DOT: sa = Max summaries, QUEST: sa = Max, sb = Min. */
int vxo_score(int kind, const uint16_t *q, int Hq, int H, int Dqk, int page_size,
              int batch, const int32_t *page_indptr, const int32_t *page_indices,
              const int32_t *seq_lens, const double *sa, const double *sb, double *scores);

/* Indexer stage, selection: sink + local pages plus the best-scoring remaining pages.
 * sel_pages [batch][H][max_sel] ascending logical page ids, -1 padded; sel_count [batch].
 * s_kth / s_next [batch][H]: the K_free-th and (K_free+1)-th best candidate scores
 * (+inf / -inf when absent), used for the comparison band. */
int vxo_select(const double *scores, int H, int page_size, int batch,
               const int32_t *page_indptr, const int32_t *seq_lens, const int32_t *pages_budget,
               int n_sink, int n_local, int max_sel, int32_t *sel_pages, int32_t *sel_count,
               double *s_kth, double *s_next);

/* Approximate radix top-k (approxTopK): selection from fp32 scores [H][batch][stride] with
 * num_items[i] pages per request; tau in [0, 1] is the tolerate ratio (0: exact selection on
 * the keys), seed drives the random fill, remap 0/1 picks the key (order key / affine fixed
 * point).  Same outputs as vxo_select (without the score band). */
int vxo_topk_select(const float *scores, int stride, int H, int batch, const int32_t *num_items,
                    const int32_t *pages_budget, int n_sink, int n_local, int max_sel, float tau,
                    uint32_t seed, int remap, int32_t *sel_pages, int32_t *sel_count);

/* Exact softmax attention over the tokens of the selected pages.  out [batch][Hq][Dv].
 * A request with no selected page gets a zero output. */
int vxo_attend(const uint16_t *q, int Hq, const uint16_t *k, const uint16_t *v, int H,
               int page_size, int Dqk, int Dv, int batch, const int32_t *page_indptr,
               const int32_t *page_indices, const int32_t *seq_lens, const int32_t *sel_pages,
               const int32_t *sel_count, int max_sel, double sm_scale, double *out);

#ifdef __cplusplus
}
#endif
#endif

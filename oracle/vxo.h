/* vxo.h -- plain CPU fp64 oracle for page-centric sparse decode attention
 * (Vortex, arXiv 2606.06453).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may load this library.  It shares no code, header, table or constant
 * with the HIP path.
 *
 * All pointers are host pointers.  bf16 tensors are passed as their raw 16-bit patterns.
 * Every bf16 value is widened exactly to fp64 and all arithmetic is fp64.  A KV cache is
 * bf16 (kv_fmt VXO_KV_BF16) or 8-bit floating point (VXO_KV_FP8_E4M3 / VXO_KV_FP8_E5M2, OCP
 * formats, one byte per element) with a per-tensor scale: the cache value is the fp32
 * product scale * code value.
 *
 * Layouts (paged layout, Appendix A):
 *   k           [num_phys_pages][H][page_size][Dqk]   bf16 bits or fp8 codes
 *   v           [num_phys_pages][H][page_size][Dv]    same dtype as k, or NULL: V_t = K_t[0:Dv] (MLA)
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
/* Envelope flows of the agent-proposed algorithms (Appendix G). */
#define VXO_QUEST_CONSENSUS 3
#define VXO_ENVELOPE_LOWER 4
#define VXO_QUEST_RECTIFIED 5
/* Eq. 2 over the first Dc channels (rope-unaware MLA block score). */
#define VXO_MEAN_DOT_CONTENT 6

#define VXO_KV_BF16 0
#define VXO_KV_FP8_E4M3 1
#define VXO_KV_FP8_E5M2 2

const char *vxo_error(void);
int vxo_num_threads(void);
/* Threads used by the following calls (OpenMP over independent units; no arithmetic change). */
void vxo_set_num_threads(int n);

/* Dequantised values (fp32) of n fp8 codes of the given format with the given scale. */
int vxo_fp8_dequantize(const uint8_t *codes, int64_t n, int fmt, float scale, float *out);

/* Cache stage: per-page Mean / Max / Min of keys over the page's valid tokens.
 * Summaries are written for logical pages j >= first_page[i] (all pages when first_page is
 * NULL), at [phys][H][Dqk].  Max and Min are bf16 values (rounded to nearest even from the
 * fp32 key values of an fp8 cache).  Each output may be NULL. */
int vxo_summarize(const void *k, int kv_fmt, float k_scale, int64_t num_phys_pages, int H, int page_size, int Dqk,
                  int batch, const int32_t *page_indptr, const int32_t *page_indices,
                  const int32_t *seq_lens, const int32_t *first_page,
                  double *mean, double *maxv, double *minv);

/* Cache stage at a decode step: copy each request's new key and value rows (kv_fmt elements,
 * k_new [batch][H][Dqk], v_new [batch][H][Dv]) into slot (L_i - 1) mod page_size of its page
 * (L_i - 1) / page_size; v == NULL (V aliased) writes only K.  The caller then summarises the
 * pages from that one on (vxo_summarize with first_page). */
int vxo_kv_append(void *k, void *v, int kv_fmt, int64_t num_phys_pages, int H, int page_size, int Dqk, int Dv,
                  int batch, const int32_t *page_indptr, const int32_t *page_indices, const int32_t *seq_lens,
                  const void *k_new, const void *v_new);

/* Indexer stage, scoring.  scores is ragged: [page_indptr[batch]][H], row page_indptr[i]+j.
 * MEAN_DOT and MEAN_DOT_CONTENT: sa = Mean summaries, MAX_DOT: sa = Max summaries, QUEST,
 * QUEST_CONSENSUS and ENVELOPE_LOWER: sa = Max, sb = Min; QUEST_RECTIFIED: sa = Max.
 * MEAN_DOT_CONTENT scores the channels c < Dc only; other kinds ignore Dc. */
int vxo_score(int kind, const uint16_t *q, int Hq, int H, int Dqk, int Dc, int page_size,
              int batch, const int32_t *page_indptr, const int32_t *page_indices,
              const int32_t *seq_lens, const double *sa, const double *sb, double *scores);

/* Score flows over the operator table's Softmax / Conv1d / Sum.  taps[3]: the Conv1d kernel
 * along the page axis, y_j = taps[0] x_{j-1} + taps[1] x_j + taps[2] x_{j+1}, zero padding.
 * vxo_head_logits: per-query-head logits fp32(q_r . Mean_j), ragged [page_indptr[batch]][Hq].
 * vxo_nsa_scores: NSA block scores, sum over G_h of Conv1d(softmax over pages of the logits),
 *   ragged [page_indptr[batch]][H].
 * vxo_smooth_scores: Conv1d of a ragged [..][H] score table (positional smoothing). */
int vxo_head_logits(const uint16_t *q, int Hq, int H, int Dqk, int page_size, int batch,
                    const int32_t *page_indptr, const int32_t *page_indices, const int32_t *seq_lens,
                    const double *mean, double *logits);
int vxo_nsa_scores(const double *logits, int Hq, int H, int page_size, int batch, const int32_t *page_indptr,
                   const int32_t *seq_lens, const double *taps, double *scores);
int vxo_smooth_scores(const double *in, int H, int page_size, int batch, const int32_t *page_indptr,
                      const int32_t *seq_lens, const double *taps, double *out);

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
 * the keys), seed drives the random order of the threshold bin after an early termination
 * (a seeded 8-bit hash of the page index), remap 0/1 picks the key (order key / affine fixed
 * point).  Same outputs as vxo_select (without the score band). */
int vxo_topk_select(const float *scores, int stride, int H, int batch, const int32_t *num_items,
                    const int32_t *pages_budget, int n_sink, int n_local, int max_sel, float tau,
                    uint32_t seed, int remap, int32_t *sel_pages, int32_t *sel_count);

/* Exact softmax attention over the tokens of the selected pages.  out [batch][Hq][Dv].
 * A request with no selected page gets a zero output. */
int vxo_attend(const uint16_t *q, int Hq, const void *k, const void *v, int kv_fmt, float k_scale,
               float v_scale, int H, int page_size, int Dqk, int Dv, int batch, const int32_t *page_indptr,
               const int32_t *page_indices, const int32_t *seq_lens, const int32_t *sel_pages,
               const int32_t *sel_count, int max_sel, double sm_scale, double *out);

#ifdef __cplusplus
}
#endif
#endif

/* vx.h -- page-centric sparse decode attention on MI355X (gfx950).
 *
 * The hot path of one decode step of Vortex-style sparse attention (arXiv 2606.06453):
 *   1. vx_page_summarize       cache stage: per-page key summaries (Sec. 3.1 Eq. 1; Sec. 3.2 Quest)
 *      (at a decode step: vx_kv_append_summarize appends the new K/V rows and refreshes the
 *      receiving page's summaries in one launch)
 *   2. vx_page_score_topk      indexer stage: page scores (Sec. 3.1 Eq. 2; Quest; the NSA,
 *                              rope-unaware and agent-proposed flows) and selection of sink,
 *                              local and top-scoring pages (Eq. 3; Sec. 6.4 setup)
 *      (or, as separate operators: vx_page_score, vx_score_flow for the NSA and smoothing
 *      flows, then vx_topk_select, exact or with the approximate radix top-k of Sec. 5.2)
 *      (at a decode step, vx_append_score_topk does the step's append and summary refresh
 *      inside the selection's top-K launch: steps 1 and 2 in two launches)
 *   3. vx_sparse_paged_decode  attention over the selected pages only (Eq. 4), as split-K
 *                              online softmax plus a merge, over a ragged batch.
 *
 * Conventions shared by every call
 * ---------------------------------
 * - Every pointer argument is a DEVICE pointer unless its comment says "host".  The structs
 *   themselves are host memory and are read during the call only.
 * - The caller owns every buffer.  The library never allocates, frees or synchronises.  Every
 *   call only enqueues kernels on `stream`, so it can be captured in a HIP graph.  Workspace
 *   contents do not survive between calls.
 * - Host-side argument checks run before any launch.  They return VX_ERR_INVALID_ARG for bad
 *   pointers or sizes and VX_ERR_UNSUPPORTED for unsupported geometry.  A failed launch returns
 *   VX_ERR_HIP.  vx_last_error() gives a thread-local message for the last non-OK status.
 * - Device-array contents are the caller's contract.  page_indptr must start at 0 and be
 *   non-decreasing, page ids must be in range, seq_lens >= 1, and the page list of request i
 *   must hold at least P_i = ceil(seq_lens[i] / page_size) entries.  Kernels clamp page ids
 *   and page counts so that broken ids or lengths cannot cause an access out of bounds; they
 *   can only give wrong results.
 * - Calls are reentrant.  There is no global mutable state except the thread-local error
 *   message.  Two calls that share a workspace must not overlap on different streams.
 *
 * Data layout in HBM
 * ------------------
 * - bf16 is IEEE binary16-brain (bfloat16).
 * - KV cache element type (Sec. 5.3 and Appendix E: bf16, fp8_e4m3 and fp8_e5m2 caches):
 *   bf16, or one byte per element in the OCP 8-bit floating point formats E4M3 (no
 *   infinities, max 448) or E5M2, with one fp32 scale for K and one for V.  The value of an
 *   fp8 entry is the fp32 product scale * code value; summaries, scores and attention all use
 *   that value.  For an MLA latent (V aliased to its first head_dim_v channels) the V values
 *   are the latent's, at the K scale; v_scale is then unused.
 * - Paged KV cache (Appendix A), "HND": one (page, head) slice is one contiguous run.
 *       k  [num_phys_pages][num_kv_heads][page_size][head_dim_qk]
 *       v  [num_phys_pages][num_kv_heads][page_size][head_dim_v], or NULL when V is the first
 *          head_dim_v channels of K (absorbed-weight MLA latent, Sec. 6.2).
 *   Elements are bf16 or fp8 codes (kv_dtype); k and v have the same element type.
 * - Batch (Sec. 4.1, C = (b, p, I)): page_indptr [batch+1] with page_indptr[0] = 0, and
 *   page_indices [page_indptr[batch]] physical page ids.  The logical page j of request i is
 *   page_indices[page_indptr[i] + j].  Ids may repeat across requests (prefix sharing); a
 *   shared page must have the same number of valid tokens in every request that uses it.
 *   Logical page j of request i holds n_ij = min(page_size, seq_lens[i] - j*page_size) valid
 *   tokens.
 * - q [batch][num_q_heads][head_dim_qk] bf16.  Query head r reads KV head r / g, where
 *   g = num_q_heads / num_kv_heads.
 * - Summaries are indexed by PHYSICAL page, so pages shared by requests are summarised once.
 *   Like the KV cache they are persistent state owned by the caller (Sec. 4.2: named caches
 *   are paged):
 *       mean  float [num_phys_pages][num_kv_heads][head_dim_qk]
 *       max   bf16  [num_phys_pages][num_kv_heads][head_dim_qk]   (exact for a bf16 cache; the
 *             fp32 max rounded to nearest even for an fp8 cache)
 *       min   bf16  [num_phys_pages][num_kv_heads][head_dim_qk]
 * - Selected pages: sel_pages [batch][num_kv_heads][max_sel] int32 holds logical page ids in
 *   ascending order, padded with -1.  sel_count [batch] int32 is the count, the same for every
 *   KV head of a request.
 *
 * Blocks (block_size below page_size, r = page_size / block_size blocks per page): summaries,
 * scores, selection and attention work on blocks of block_size tokens instead of pages.
 *   - logical block jb of request i is tokens [jb*block_size, (jb+1)*block_size) of logical
 *     page jb / r (block jb % r of physical page p = page_indices[page_indptr[i] + jb / r]);
 *     it holds min(block_size, seq_lens[i] - jb*block_size) valid tokens and request i has
 *     PB_i = ceil(seq_lens[i] / block_size) blocks;
 *   - summaries are indexed by physical block p*r + b: mean [num_phys_pages*r][H][D] etc.;
 *   - first_page (vx_page_summarize), pages_budget, n_sink, n_local, sel_pages, sel_count and
 *     every "page" count of the indexer stage are in blocks; the score rows hold PB_i entries
 *     and max_pages_per_seq stays in pages (the score table holds max_pages_per_seq * r
 *     columns);
 *   - vx_sparse_paged_decode attends the valid tokens of the selected blocks.
 * With block_size 0 or page_size every "block" above is a page.
 *
 * Supported geometry: head_dim_qk in {64, 128} with head_dim_v == head_dim_qk and a separate V
 * (GQA); or head_dim_qk = 576 with head_dim_v = 512, V aliased and num_kv_heads = 1 (MLA).
 * page_size in {16, 32, 64}; 1 <= g <= 16; num_kv_heads a power of two <= 16.
 */
#ifndef VX_H
#define VX_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define VX_VERSION_MAJOR 0
#define VX_VERSION_MINOR 3

typedef enum {
  VX_OK = 0,
  VX_ERR_INVALID_ARG = 1,
  VX_ERR_UNSUPPORTED = 2,
  VX_ERR_WORKSPACE = 3,
  VX_ERR_HIP = 4
} vx_status;

/* How a page is scored against the query heads G_h = {h*g, ..., h*g + g - 1} of KV head h. */
typedef enum {
  /* Sec. 3.1 Eq. 2 (block top-k): s_j = mean over r in G_h of q_r . Mean_j. */
  VX_SCORE_MEAN_DOT = 0,
  /* Sec. 3.2 Quest: s_j = max over r in G_h of sum_c max(q_rc*Max_jc, q_rc*Min_jc). */
  VX_SCORE_QUEST = 1,
  /* Eq. 2 with the per-channel Max summary in place of the mean (Table of operators: Max). */
  VX_SCORE_MAX_DOT = 2,
  /* Envelope flows of the agent-proposed algorithms (Appendix G), GQA geometry only:
   * head-consensus Quest: s_j = MIN over r in G_h of sum_c max(q_rc*Max_jc, q_rc*Min_jc). */
  VX_SCORE_QUEST_CONSENSUS = 3,
  /* pessimistic envelope: s_j = max over r in G_h of sum_c min(q_rc*Max_jc, q_rc*Min_jc). */
  VX_SCORE_ENVELOPE_LOWER = 4,
  /* rectified Quest: s_j = max over r in G_h of sum_c ReLU(q_rc*Max_jc) (reads Max only). */
  VX_SCORE_QUEST_RECTIFIED = 5,
  /* Eq. 2 over the content channels c < head_dim_v only (reads Mean): on an MLA latent the
   * decoupled rope channels are left out, the rope-unaware block-sparse flow of Sec. 6.2 and
   * the rope-component study of Sec. 6.3.  With head_dim_v == head_dim_qk it is MEAN_DOT. */
  VX_SCORE_MEAN_DOT_CONTENT = 6,
  /* Block top-k part of NSA (Sec. 3.2, the NSA listing: softmax, convolution, head sum, top-K),
   * GQA geometry only, reads Mean: per query head r in G_h the logits z_rj = q_r . Mean_j
   * (fp64, rounded to fp32), the softmax over the request's pages of z_r, a 1-D convolution
   * along the pages with taps (1/4, 1/2, 1/4) and zero padding, and the sum over G_h. */
  VX_SCORE_NSA = 7,
  /* Positional smoothing (Appendix G), reads Mean: the MEAN_DOT scores convolved along the
   * pages with taps (1/4, 1/2, 1/4) and zero padding:
   * s_j = m_{j-1}/4 + m_j/2 + m_{j+1}/4 with m_{-1} = m_{P_i} = 0. */
  VX_SCORE_MEAN_DOT_SMOOTH = 8
} vx_score_kind;

/* KV cache element type. */
typedef enum {
  VX_KV_BF16 = 0,
  VX_KV_FP8_E4M3 = 1,   /* OCP E4M3: bias 7, no infinities, S.1111.111 is NaN */
  VX_KV_FP8_E5M2 = 2    /* OCP E5M2: bias 15 */
} vx_kv_dtype;

typedef enum {
  VX_STAGE_SCORE_TOPK = 0,
  VX_STAGE_DECODE = 1
} vx_stage;

/* Paged KV cache geometry (Appendix A, paged layout). */
typedef struct {
  const void* k;             /* kv_dtype elements, layout above */
  const void* v;             /* kv_dtype elements, layout above, or NULL: V = K[..., :head_dim_v] */
  int32_t num_phys_pages;
  int32_t num_kv_heads;
  int32_t page_size;
  int32_t head_dim_qk;
  int32_t head_dim_v;
  int32_t kv_dtype;          /* vx_kv_dtype */
  float k_scale;             /* fp8 only: finite and > 0 (ignored for bf16) */
  float v_scale;             /* fp8 only: finite and > 0 (ignored for bf16) */
  int32_t block_size;        /* summary / selection granularity in tokens (Appendix E template:
                                block_size below page_size): 0 or page_size for one block per
                                page, else 16 or 32 dividing page_size; see "Blocks" above */
} vx_paged_cache;

/* Ragged batch over the paged cache (Sec. 4.1, C = (b, p, I)). */
typedef struct {
  int32_t batch;
  int32_t max_pages_per_seq;   /* host: upper bound on P_i over the batch (sizes the score
                                  workspace; pages beyond it are treated as absent) */
  const int32_t* page_indptr;  /* [batch+1] */
  const int32_t* page_indices; /* [page_indptr[batch]] */
  const int32_t* seq_lens;     /* [batch], tokens incl. the current one */
} vx_batch;

/* (major << 16) | minor. */
uint32_t vx_version(void);

/* Thread-local message describing the last non-OK status of a call on this thread. */
const char* vx_last_error(void);

/* Host-only: workspace bytes needed by vx_page_score_topk (stage VX_STAGE_SCORE_TOPK: max(2 H,
 * num_q_heads + H) fp32 planes of batch x (max_pages_per_seq x blocks per page) rounded up to 4,
 * H = num_kv_heads) or by vx_sparse_paged_decode (VX_STAGE_DECODE: split counters and split-K
 * partials; zero-fill it once, see vx_sparse_paged_decode) for this geometry.  max_sel is the
 * row stride of sel_pages. */
vx_status vx_workspace_size(vx_stage stage, const vx_paged_cache* kv, const vx_batch* b,
                            int32_t num_q_heads, int32_t max_sel, size_t* bytes);

/* Cache stage (Sec. 3.1 Eq. 1; Sec. 3.2 Quest; Table of operators: Mean/Max/Min).
 * For every logical page j >= first_page[i] of request i (every page when first_page is
 * NULL), with p its physical page and n its valid tokens, writes for each KV head h and
 * channel c:
 *   mean_out[p][h][c] = (1/n) sum_{t<n} K[p][h][t][c]   (fp32 accumulation, rounded to fp32)
 *   mean_bf16_out[p][h][c] = bf16(mean_out[p][h][c])     (round to nearest even)
 *   max_out[p][h][c]  = max_{t<n} K[p][h][t][c]          (exact)
 *   min_out[p][h][c]  = min_{t<n} K[p][h][t][c]          (exact)
 * Any of the four outputs may be NULL (not computed).  Tokens t >= n are never read.
 * mean_bf16_out has the layout of max_out; it lets vx_page_score_topk make its first pass
 * over half the bytes (see there).
 * At a decode step the caller passes first_page[i] = P_i - 1 so that only the page that
 * received the new token is updated. */
vx_status vx_page_summarize(const vx_paged_cache* kv, const vx_batch* b,
                            const int32_t* first_page,
                            float* mean_out, void* mean_bf16_out, void* max_out, void* min_out,
                            hipStream_t stream);

/* Cache stage of a decode step in one launch (Sec. 3.1: summaries are built with the cache;
 * the operator table's cache-side operators act within one block): appends each request's
 * new key and value rows and refreshes the summaries of the page that receives them.
 * Request i's new token is token L_i - 1 (seq_lens already counts it), so it goes to slot
 * (L_i - 1) mod page_size of logical page (L_i - 1) / page_size:
 *   K[p][h][slot][:] = k_new[i][h][:]   k_new [batch][num_kv_heads][head_dim_qk]
 *   V[p][h][slot][:] = v_new[i][h][:]   v_new [batch][num_kv_heads][head_dim_v]
 * (kv_dtype elements: bf16, or fp8 codes already quantised with the cache's scales).  With V
 * aliased (kv->v NULL, MLA) v_new must be NULL and only K is written.  Then the summaries of
 * that page are written exactly as vx_page_summarize with first_page[i] = (L_i - 1) / page_size
 * writes them (bit-identical), to whichever of the four outputs are non-NULL.
 * This call WRITES the caches through kv->k and kv->v.  The page receiving a request's token
 * must not be shared with another request.  One launch replaces an append kernel plus
 * vx_page_summarize. */
vx_status vx_kv_append_summarize(const vx_paged_cache* kv, const vx_batch* b, const void* k_new, const void* v_new,
                                 float* mean_out, void* mean_bf16_out, void* max_out, void* min_out,
                                 hipStream_t stream);

/* Key remapping of the radix selection (vx_topk_select, and vx_page_score_topk with options;
 * Appendix D: a monotone map applied before the radix passes to spread the scores over the
 * bins). */
typedef enum {
  VX_REMAP_NONE = 0,     /* order-preserving 32-bit key of the fp32 score */
  VX_REMAP_AFFINE = 1    /* floor((s - min) * (2^32 - 1) / (max - min)) over the candidates, fp64 */
} vx_remap;

/* Host struct: options of the radix selection (vx_topk_select, vx_page_score_topk).  Zero-filled
 * (or a NULL pointer) is the exact selection. */
typedef struct {
  float tolerate_ratio;  /* tau in [0, 1] (the approxTopK tolerate ratio), taken in 16-bit fixed
                            point: tau_q = round(65536 tau) */
  uint32_t seed;         /* drives the random part of the selection */
  int32_t remap;         /* vx_remap */
} vx_topk_options;

/* Indexer stage (Sec. 3.1 Eqs. 2-3; Sec. 3.2 Quest; Sec. 6.4 sink and local blocks).
 * For each request i and KV head h:
 *   - score every page with `kind` (scores accumulate in fp64 and round once to fp32; the NSA
 *     and smoothing flows compute their softmax, convolution and sum in fp64 and round once
 *     to fp32).  The block score has no 1/sqrt(d) factor.  MEAN_DOT, MEAN_DOT_CONTENT, NSA
 *     and MEAN_DOT_SMOOTH read `mean`; MAX_DOT and QUEST_RECTIFIED read `max`; the other
 *     envelope kinds read `max` and `min`.
 *   - F = {0 .. n_sink-1} U {P_i - n_local .. P_i - 1} is always kept.
 *   - K_total = min(pages_budget[i], max_sel).  If K_total >= P_i, every page is kept.
 *     Otherwise the K_free = max(0, K_total - |F|) best remaining pages are kept.  Best means
 *     the larger fp32 score, with ties going to the lower page index (-0.0 == +0.0).
 *   - sel_pages[i][h][:] = F U best, ascending, -1 padded.  sel_count[i] = |F U best|.
 * pages_budget [batch] int32 is the total page budget of each request, forced pages
 * included.  Requires 0 <= n_sink, 0 <= n_local, n_sink + n_local <= max_sel, and
 * num_q_heads * head_dim_qk <= 16384 (the query block is staged in LDS).
 * MEAN_DOT or MEAN_DOT_CONTENT with `mean_bf16` (and max_pages_per_seq <= 4096) selects in two
 * exact passes; the bf16 copy is otherwise ignored.
 *   1. An approximate score s' = qbar . bf16(Mean) is computed from half the bytes, with a
 *      rigorous bound |s - s'| <= b, where b comes from the bf16 rounding of each channel plus
 *      the accumulation and output roundings.
 *   2. Pages whose interval [s'-b, s'+b] proves them in or out of the top K_free are decided
 *      at once.
 *   3. The few undecided pages are re-scored from the fp32 `mean` with the same arithmetic
 *      as the one-pass path.
 * The result is identical to the one-pass selection.
 * The four envelope kinds (QUEST, QUEST_CONSENSUS, ENVELOPE_LOWER, QUEST_RECTIFIED) with at
 * most 4 query heads per KV head, head_dim_qk 64 or 128 and max_pages_per_seq <= 4096 (and
 * no approximate options) always select in two exact passes the same way: the first pass sums
 * the exact products in fp32 and bounds the error by 2^-18 |q_r|_1 max_c(|Max_c|, |Min_c|) per
 * head, and the undecided pages are re-scored with the one-pass fp64 arithmetic.
 * opt (host pointer, may be NULL): with a tolerate ratio above 0 or a remap, the selection is
 * the approximate radix top-k of vx_topk_select (Sec. 5.2 stochastic early termination, in the
 * indexer step itself) over the one-pass fp32 scores of `kind` (the block mean then reads the
 * fp32 `mean`; the two-pass path is exact only).  NULL or zero-filled: the exact selection.
 * workspace: device buffer of at least vx_workspace_size(VX_STAGE_SCORE_TOPK) bytes. */
vx_status vx_page_score_topk(const void* q, int32_t num_q_heads,
                             const vx_paged_cache* kv, const vx_batch* b,
                             vx_score_kind kind,
                             const float* mean, const void* mean_bf16, const void* max, const void* min,
                             const int32_t* pages_budget,
                             int32_t n_sink, int32_t n_local, int32_t max_sel,
                             int32_t* sel_pages, int32_t* sel_count,
                             void* workspace, size_t workspace_bytes,
                             const vx_topk_options* opt, hipStream_t stream);

/* The decode step's cache stage and indexer stage in one call (Sec. 3.1: the cache stage is
 * query-independent, then the indexer stage): the effect of
 *   vx_kv_append_summarize(kv, b, k_new, v_new, mean, mean_bf16, max, min)
 *   vx_page_score_topk(q, num_q_heads, kv, b, kind, mean, mean_bf16, max, min, pages_budget,
 *                      n_sink, n_local, max_sel, sel_pages, sel_count, workspace, ..., opt)
 * with the same arguments and the same outputs (caches, summaries, selection), in two launches
 * instead of three: the append runs inside the top-K launch.  This is exact because the block
 * that receives a request's new token is its last block, which n_local >= 1 always keeps, and
 * every score kind but NSA and MEAN_DOT_SMOOTH scores a block from its own summary alone: the
 * score launch reads that block's summary from before the append, and only that block's
 * (unused) score depends on it.  Blocks of more than 8192 elements per head (block size x
 * head_dim_qk, e.g. 64 x 576), which one workgroup would refresh on the selection's critical
 * path, are refreshed by workgroups of their own inside the top-K launch when the selection is
 * the one-pass kind of at most 512 blocks per request (the MLA latent's block mean without
 * mean_bf16).  With n_local == 0, NSA or MEAN_DOT_SMOOTH (whose flows couple the blocks), an
 * approximate selection (opt), more than 4096 blocks per request or such large blocks on the
 * other selection paths, the call appends first and then selects, in three launches.
 * Arguments and requirements are those of the two calls (mean, mean_bf16, max and min are
 * written by the append and read by the selection; seq_lens counts the new token, so every
 * request has L_i >= 1; a request with L_i = 0, or whose token L_i - 1 lies past its page
 * list, appends nothing). */
vx_status vx_append_score_topk(const vx_paged_cache* kv, const vx_batch* b, const void* k_new, const void* v_new,
                               float* mean, void* mean_bf16, void* max, void* min,
                               const void* q, int32_t num_q_heads, vx_score_kind kind,
                               const int32_t* pages_budget, int32_t n_sink, int32_t n_local, int32_t max_sel,
                               int32_t* sel_pages, int32_t* sel_count, void* workspace, size_t workspace_bytes,
                               const vx_topk_options* opt, hipStream_t stream);

/* Indexer scoring on its own (Sec. 3.1 Eq. 2; Sec. 3.2 Quest; the score operators of the
 * operator table): the one-pass fp32 score of every page, as vx_page_score_topk defines it
 * (fp64 accumulation, one rounding to fp32; MEAN_DOT reads the fp32 `mean`), written to
 *   scores[(h * batch + i) * score_stride + j]   for KV head h, request i, page j < P_i.
 * For the two flow kinds it writes the input of their last steps (vx_score_flow):
 *   NSA: the per-query-head logits fp32(q_r . Mean_j) at scores[(r * batch + i) * score_stride + j]
 *        for every query head r (num_q_heads rows per request);
 *   MEAN_DOT_SMOOTH: the MEAN_DOT scores.
 * Other entries of the buffer are left untouched.  Requires score_stride >=
 * max_pages_per_seq and num_q_heads * head_dim_qk <= 16384.  No workspace. */
vx_status vx_page_score(const void* q, int32_t num_q_heads,
                        const vx_paged_cache* kv, const vx_batch* b,
                        vx_score_kind kind,
                        const float* mean, const void* max, const void* min,
                        float* scores, int32_t score_stride,
                        hipStream_t stream);

/* The last steps of the NSA and positional-smoothing flows (the Softmax, Conv1d and Sum
 * operators of the operator table), from what vx_page_score writes for them:
 *   NSA: scores_in holds num_q_heads rows [r][batch][score_stride] of logits; for KV head h and
 *        each query head r of its group, p_rj = exp(z_rj - m_r) / sum_j' exp(z_rj' - m_r) over
 *        the request's pages (m_r their max), then the convolution, then the sum over the group
 *        in head order;
 *   MEAN_DOT_SMOOTH: scores_in holds [h][batch][score_stride] block-mean scores; the convolution.
 * The convolution runs along the pages with taps (1/4, 1/2, 1/4) and zero padding.  All of it is
 * fp64 with one rounding to fp32 into scores_out [h][batch][score_stride], columns j < num_items[i]
 * (capped at score_stride).  scores_in and scores_out must not overlap.  num_items [batch] device
 * array of page counts; num_q_heads / num_kv_heads <= 16. */
vx_status vx_score_flow(vx_score_kind kind, const float* scores_in, float* scores_out, int32_t score_stride,
                        int32_t num_kv_heads, int32_t num_q_heads, int32_t batch, const int32_t* num_items,
                        hipStream_t stream);


/* Selection from precomputed scores (Sec. 3.1 Eq. 3; Sec. 5.2 approximate radix top-k;
 * the TopK / approxTopK operators).  For request i (num_items[i] pages, capped at
 * score_stride) and KV head h, with the scores laid out as vx_page_score writes them:
 * F = sink and local pages as in vx_page_score_topk; K_total = min(pages_budget[i], max_sel);
 * K_total >= P keeps every page; otherwise K_free = max(0, K_total - |F|) candidates are
 * chosen by a radix select over their keys (8-bit digits, most significant first, from the
 * highest bit in which the candidates' extreme keys differ):
 *   - exact (tolerate_ratio 0): the K_free largest keys, ties to the lower page index;
 *   - approximate: after a pass with key bits left, once the candidates in bins above the
 *     threshold bin number at least (1 - tau) K_free, refinement stops; they are kept, and
 *     the rest is a random sample of the threshold bin: its candidates ordered by the 8-bit
 *     hash h8(j) = lowbias32(z ^ j) >> 24 of the page index j, larger first, equal hashes
 *     by lower page, z = lowbias32(seed ^ lowbias32(i * num_kv_heads + h)).  At least
 *     (1 - tau) K_free of the K_free chosen candidates are then true top members.
 * lowbias32 is C. Wellons' 32-bit integer hash: x ^= x >> 16; x *= 0x7feb352d; x ^= x >> 15;
 * x *= 0x846ca68b; x ^= x >> 16.  Outputs as in vx_page_score_topk (sel_pages ascending,
 * -1 padded; sel_count [batch] written by KV head 0).  NaN scores rank lowest.  Requires
 * n_sink + n_local <= max_sel.  opt: host pointer or NULL. */
vx_status vx_topk_select(const float* scores, int32_t score_stride, int32_t num_kv_heads, int32_t batch,
                         const int32_t* num_items, const int32_t* pages_budget,
                         int32_t n_sink, int32_t n_local, int32_t max_sel,
                         const vx_topk_options* opt,
                         int32_t* sel_pages, int32_t* sel_count,
                         hipStream_t stream);

/* Sparse attention (Sec. 3.1 Eq. 4; Sec. 5.3 paged decode fed a sparse block table).
 * For each request i and query head r (KV head h = r / g):
 *   out[i][r][:] = softmax_t(sm_scale * q_r . k_t) V_t over the valid tokens t of the pages
 *   sel_pages[i][h][0 .. sel_count[i]-1]; an empty selection gives zeros.  out is bf16
 *   [batch][num_q_heads][head_dim_v], rounded to nearest even from fp32 accumulators.
 * The path is a device-side plan (Sec. 5.1: balanced work per program): each (request,
 * KV head) pair is cut, from its selection count, into contiguous runs of at most a fixed
 * number of selected pages, one workgroup each (a short pair is not split); a split-K kernel
 * with online softmax; and an LSE-weighted merge of a split pair's partials (for GQA inside
 * the split kernel, by the pair's last split; for MLA by a merge launch).  Logical ids
 * outside [0, P_i) are skipped.  max_sel above 2^24 returns VX_ERR_UNSUPPORTED.
 * workspace: device buffer of at least vx_workspace_size(VX_STAGE_DECODE) bytes.  It starts
 * with one 32-bit split counter per (request, KV head) pair, which must be zero before the
 * first call: zero-fill the buffer once after allocating it.  Every call leaves the counters
 * zero again; the rest of the buffer is scratch.  Do not use the buffer for anything else. */
vx_status vx_sparse_paged_decode(const void* q, int32_t num_q_heads,
                                 const vx_paged_cache* kv, const vx_batch* b,
                                 const int32_t* sel_pages, const int32_t* sel_count,
                                 int32_t max_sel, float sm_scale,
                                 void* out,
                                 void* workspace, size_t workspace_bytes,
                                 hipStream_t stream);

/* vx_sparse_paged_decode for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same computation and
 * outputs, with no workspace argument.  Its split counters and partials live in a static
 * 12 MiB device buffer of the library, one per GPU, held until the process ends; the call
 * itself allocates nothing.  A batch whose decode workspace (vx_workspace_size with
 * VX_STAGE_DECODE) exceeds 12 MiB returns VX_ERR_WORKSPACE.  Every call on a GPU shares that
 * GPU's buffer: calls that overlap on one GPU (different streams, or other host threads) race
 * and give wrong results; serialise them.  The buffer is zero when the library loads, and every
 * call leaves its split counters zero again. */
vx_status vx_sparse_paged_decode_noalloc(const void* q, int32_t num_q_heads,
                                         const vx_paged_cache* kv, const vx_batch* b,
                                         const int32_t* sel_pages, const int32_t* sel_count,
                                         int32_t max_sel, float sm_scale,
                                         void* out, hipStream_t stream);

/* Measurement utility, not a step of the path: reads `bytes` (a positive multiple of 16) from
 * the 16-byte aligned device buffer `buf` with 16-byte loads carrying the non-temporal hint (the
 * load form of the decode and score kernels), over `workgroups` workgroups of 256 threads in a
 * grid-stride loop.  Timing it gives the device's practical streaming-read rate, reported beside
 * the nameplate HBM peak.  sink: device array of `workgroups` uint32, practically never written
 * (the loads feed a value that is stored only if it equals a fixed constant). */
vx_status vx_stream_read(const void* buf, size_t bytes, uint32_t* sink, int32_t workgroups, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* VX_H */

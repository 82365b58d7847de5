// C ABI of libvx: argument validation, workspace sizing and dispatch to the HIP kernels.
// The declarations and their contracts are in include/vx.h.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "vx.h"
#include "vx_internal.h"

namespace {

thread_local char g_err[512];

vx_status fail(vx_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return s;
}

vx_status hip_status(hipError_t e, const char* where) {
  if (e == hipSuccess) return VX_OK;
  return fail(VX_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

// Options of the radix selection (NULL: exact): tau in 16-bit fixed point.
vx_status check_topk_options(const vx_topk_options* opt, int* remap, int* tau_q, uint32_t* seed) {
  *remap = 0;
  *tau_q = 0;
  *seed = 0;
  if (!opt) return VX_OK;
  if (!(opt->tolerate_ratio >= 0.f && opt->tolerate_ratio <= 1.f))
    return fail(VX_ERR_INVALID_ARG, "tolerate_ratio must be in [0, 1]");
  if (opt->remap != VX_REMAP_NONE && opt->remap != VX_REMAP_AFFINE)
    return fail(VX_ERR_INVALID_ARG, "unknown remap %d", (int)opt->remap);
  *remap = opt->remap;
  *tau_q = (int)lroundf(opt->tolerate_ratio * 65536.0f);
  *seed = opt->seed;
  return VX_OK;
}

bool is_pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }

bool is_mla(const vx_paged_cache* kv) { return kv->head_dim_qk == 576; }

// Geometry checks shared by every call.
vx_status check_cache(const vx_paged_cache* kv, bool need_v) {
  if (!kv) return fail(VX_ERR_INVALID_ARG, "kv is NULL");
  if (!kv->k) return fail(VX_ERR_INVALID_ARG, "kv->k is NULL");
  if (kv->num_phys_pages < 1) return fail(VX_ERR_INVALID_ARG, "num_phys_pages must be >= 1");
  if (kv->page_size != 16 && kv->page_size != 32 && kv->page_size != 64)
    return fail(VX_ERR_UNSUPPORTED, "page_size %d not in {16, 32, 64}", kv->page_size);
  if (!is_pow2(kv->num_kv_heads) || kv->num_kv_heads > 16)
    return fail(VX_ERR_UNSUPPORTED, "num_kv_heads %d must be a power of two <= 16", kv->num_kv_heads);
  if (kv->head_dim_qk == 64 || kv->head_dim_qk == 128) {
    if (kv->head_dim_v != kv->head_dim_qk)
      return fail(VX_ERR_UNSUPPORTED, "GQA needs head_dim_v == head_dim_qk (got %d, %d)", kv->head_dim_v,
                  kv->head_dim_qk);
    if (need_v && !kv->v) return fail(VX_ERR_UNSUPPORTED, "GQA needs a separate V cache");
  } else if (kv->head_dim_qk == 576) {
    if (kv->head_dim_v != 512 || kv->v || kv->num_kv_heads != 1)
      return fail(VX_ERR_UNSUPPORTED, "MLA needs head_dim_v = 512, aliased V (v = NULL) and one KV head");
  } else {
    return fail(VX_ERR_UNSUPPORTED, "head_dim_qk %d not in {64, 128, 576}", kv->head_dim_qk);
  }
  if (kv->block_size != 0 && kv->block_size != kv->page_size &&
      !((kv->block_size == 16 || kv->block_size == 32) && kv->page_size % kv->block_size == 0))
    return fail(VX_ERR_UNSUPPORTED, "block_size %d must be 0, page_size, or 16 or 32 dividing page_size %d",
                kv->block_size, kv->page_size);
  if (kv->kv_dtype != VX_KV_BF16 && kv->kv_dtype != VX_KV_FP8_E4M3 && kv->kv_dtype != VX_KV_FP8_E5M2)
    return fail(VX_ERR_INVALID_ARG, "kv_dtype %d is not a vx_kv_dtype", kv->kv_dtype);
  if (kv->kv_dtype != VX_KV_BF16) {
    if (!(kv->k_scale > 0.f) || !(kv->v_scale > 0.f) || std::isinf(kv->k_scale) || std::isinf(kv->v_scale))
      return fail(VX_ERR_INVALID_ARG, "fp8 caches need finite scales > 0 (got %g, %g)", (double)kv->k_scale,
                  (double)kv->v_scale);
  }
  return VX_OK;
}

vx_status check_batch(const vx_batch* b) {
  if (!b) return fail(VX_ERR_INVALID_ARG, "batch is NULL");
  if (b->batch < 0 || b->batch > 65535) return fail(VX_ERR_INVALID_ARG, "batch %d not in [0, 65535]", b->batch);
  if (b->batch > 0 && (!b->page_indptr || !b->page_indices || !b->seq_lens))
    return fail(VX_ERR_INVALID_ARG, "page_indptr, page_indices and seq_lens must be non-NULL");
  if (b->max_pages_per_seq < 1) return fail(VX_ERR_INVALID_ARG, "max_pages_per_seq must be >= 1");
  return VX_OK;
}

vx_status check_heads(const vx_paged_cache* kv, int32_t num_q_heads) {
  if (num_q_heads < 1 || num_q_heads % kv->num_kv_heads)
    return fail(VX_ERR_INVALID_ARG, "num_q_heads %d is not a multiple of num_kv_heads %d", num_q_heads,
                kv->num_kv_heads);
  const int g = num_q_heads / kv->num_kv_heads;
  if (g > 16) return fail(VX_ERR_UNSUPPORTED, "group size %d > 16", g);
  if (is_mla(kv) && g != 16) return fail(VX_ERR_UNSUPPORTED, "MLA path needs 16 query heads (got %d)", g);
  return VX_OK;
}

// A score kind and the summaries it reads.
vx_status check_kind(const vx_paged_cache* kv, vx_score_kind kind, const float* mean, const void* max,
                     const void* min) {
  switch (kind) {
    case VX_SCORE_MEAN_DOT:
    case VX_SCORE_MEAN_DOT_CONTENT:
    case VX_SCORE_MEAN_DOT_SMOOTH:
      if (!mean) return fail(VX_ERR_INVALID_ARG, "score kind %d needs the Mean summaries", (int)kind);
      return VX_OK;
    case VX_SCORE_NSA:
      if (!mean) return fail(VX_ERR_INVALID_ARG, "score kind %d needs the Mean summaries", (int)kind);
      break;
    case VX_SCORE_MAX_DOT:
    case VX_SCORE_QUEST_RECTIFIED:
      if (!max) return fail(VX_ERR_INVALID_ARG, "score kind %d needs the Max summaries", (int)kind);
      break;
    case VX_SCORE_QUEST:
    case VX_SCORE_QUEST_CONSENSUS:
    case VX_SCORE_ENVELOPE_LOWER:
      if (!max || !min) return fail(VX_ERR_INVALID_ARG, "score kind %d needs the Max and Min summaries", (int)kind);
      break;
    default:
      return fail(VX_ERR_INVALID_ARG, "unknown score kind %d", (int)kind);
  }
  if (is_mla(kv)) return fail(VX_ERR_UNSUPPORTED, "score kind %d is not built for the MLA geometry", (int)kind);
  return VX_OK;
}

// Blocks per request bound: max_pages_per_seq times the blocks per page (checked caches only).
int max_blocks(const vx_paged_cache* kv, const vx_batch* b) {
  const int r = kv->block_size > 0 ? kv->page_size / kv->block_size : 1;
  const int64_t m = (int64_t)b->max_pages_per_seq * r;
  return m > (1 << 30) ? (1 << 30) : (int)m;
}

vx::Geometry geometry(const vx_paged_cache* kv, const vx_batch* b) {
  vx::Geometry g;
  g.k = kv->k;
  g.v = kv->v;
  g.kv_dtype = kv->kv_dtype;
  g.k_scale = kv->kv_dtype == VX_KV_BF16 ? 1.f : kv->k_scale;
  g.v_scale = kv->kv_dtype == VX_KV_BF16 ? 1.f : kv->v_scale;
  g.num_phys_pages = kv->num_phys_pages;
  g.H = kv->num_kv_heads;
  g.ps = kv->page_size;
  g.bs = kv->block_size > 0 ? kv->block_size : kv->page_size;
  g.r = g.ps / g.bs;
  g.Dqk = kv->head_dim_qk;
  g.Dv = kv->head_dim_v;
  g.batch = b->batch;
  g.max_pages = max_blocks(kv, b);         // in blocks
  g.indptr = b->page_indptr;
  g.indices = b->page_indices;
  g.seq_lens = b->seq_lens;
  return g;
}

}  // namespace

extern "C" {

uint32_t vx_version(void) { return (VX_VERSION_MAJOR << 16) | VX_VERSION_MINOR; }

const char* vx_last_error(void) { return g_err; }

vx_status vx_workspace_size(vx_stage stage, const vx_paged_cache* kv, const vx_batch* b, int32_t num_q_heads,
                            int32_t max_sel, size_t* bytes) {
  if (!bytes) return fail(VX_ERR_INVALID_ARG, "bytes is NULL");
  vx_status s;
  if ((s = check_cache(kv, false)) != VX_OK) return s;
  if ((s = check_batch(b)) != VX_OK) return s;
  if ((s = check_heads(kv, num_q_heads)) != VX_OK) return s;
  if (max_sel < 1) return fail(VX_ERR_INVALID_ARG, "max_sel must be >= 1");
  if (stage == VX_STAGE_SCORE_TOPK) {
    *bytes = vx::score_workspace_bytes(b->batch, kv->num_kv_heads, num_q_heads, max_blocks(kv, b));
  } else if (stage == VX_STAGE_DECODE) {
    *bytes = vx::decode_layout(b->batch, kv->num_kv_heads, num_q_heads / kv->num_kv_heads, kv->head_dim_v,
                               max_sel, is_mla(kv))
                 .total;
  } else {
    return fail(VX_ERR_INVALID_ARG, "unknown stage %d", (int)stage);
  }
  return VX_OK;
}

vx_status vx_page_summarize(const vx_paged_cache* kv, const vx_batch* b, const int32_t* first_page,
                            float* mean_out, void* mean_bf16_out, void* max_out, void* min_out,
                            hipStream_t stream) {
  vx_status s;
  if ((s = check_cache(kv, false)) != VX_OK) return s;
  if ((s = check_batch(b)) != VX_OK) return s;
  if (!mean_out && !mean_bf16_out && !max_out && !min_out) return VX_OK;
  return hip_status(vx::launch_summarize(geometry(kv, b), first_page, mean_out,
                                         static_cast<uint16_t*>(mean_bf16_out), static_cast<uint16_t*>(max_out),
                                         static_cast<uint16_t*>(min_out), stream),
                    "vx_page_summarize");
}

vx_status vx_kv_append_summarize(const vx_paged_cache* kv, const vx_batch* b, const void* k_new, const void* v_new,
                                 float* mean_out, void* mean_bf16_out, void* max_out, void* min_out,
                                 hipStream_t stream) {
  vx_status s;
  if ((s = check_cache(kv, false)) != VX_OK) return s;
  if ((s = check_batch(b)) != VX_OK) return s;
  if (b->batch > 0 && !k_new) return fail(VX_ERR_INVALID_ARG, "k_new must be non-NULL");
  if (kv->v && b->batch > 0 && !v_new) return fail(VX_ERR_INVALID_ARG, "a separate V cache needs v_new");
  if (!kv->v && v_new) return fail(VX_ERR_INVALID_ARG, "v_new given but V is aliased to K (kv->v is NULL)");
  return hip_status(vx::launch_kv_append_summarize(geometry(kv, b), k_new, kv->v ? v_new : nullptr, mean_out,
                                                   static_cast<uint16_t*>(mean_bf16_out),
                                                   static_cast<uint16_t*>(max_out), static_cast<uint16_t*>(min_out),
                                                   stream),
                    "vx_kv_append_summarize");
}

namespace {
// vx_page_score_topk, and with `app` (k_new non-null) vx_append_score_topk
vx_status score_topk(const void* q, int32_t num_q_heads, const vx_paged_cache* kv, const vx_batch* b,
                     vx_score_kind kind, const float* mean, const void* mean_bf16, const void* max, const void* min,
                     const int32_t* pages_budget, int32_t n_sink, int32_t n_local, int32_t max_sel,
                     int32_t* sel_pages, int32_t* sel_count, void* workspace, size_t workspace_bytes,
                     const vx_topk_options* opt, hipStream_t stream, const vx::StepAppend& app, const char* name) {
  vx_status s;
  if ((s = check_cache(kv, false)) != VX_OK) return s;
  if ((s = check_batch(b)) != VX_OK) return s;
  if ((s = check_heads(kv, num_q_heads)) != VX_OK) return s;
  if (!q || !pages_budget || !sel_pages || !sel_count)
    return fail(VX_ERR_INVALID_ARG, "q, pages_budget, sel_pages and sel_count must be non-NULL");
  if (max_sel < 1) return fail(VX_ERR_INVALID_ARG, "max_sel must be >= 1");
  if (n_sink < 0 || n_local < 0 || (int64_t)n_sink + n_local > max_sel)
    return fail(VX_ERR_INVALID_ARG, "need 0 <= n_sink, 0 <= n_local, n_sink + n_local <= max_sel");
  int remap = 0, tau_q = 0;
  uint32_t seed = 0;
  if ((s = check_topk_options(opt, &remap, &tau_q, &seed)) != VX_OK) return s;
  if ((s = check_kind(kv, kind, mean, max, min)) != VX_OK) return s;
  if ((int64_t)num_q_heads * kv->head_dim_qk > 16384)
    return fail(VX_ERR_UNSUPPORTED, "scoring keeps q in LDS: num_q_heads * head_dim_qk must be <= 16384");
  const size_t need = vx::score_workspace_bytes(b->batch, kv->num_kv_heads, num_q_heads, max_blocks(kv, b));
  if (!workspace || workspace_bytes < need)
    return fail(VX_ERR_WORKSPACE, "score workspace needs %zu bytes (got %zu)", need, workspace_bytes);
  // the two-pass path needs the fp32 means for re-scoring and keeps a request's bounds in LDS;
  // it is exact, so an approximate selection scores in one pass
  const bool two_pass = (kind == VX_SCORE_MEAN_DOT || kind == VX_SCORE_MEAN_DOT_CONTENT) && mean_bf16 &&
                        max_blocks(kv, b) <= vx::kTwoPassMaxPages && remap == 0 && tau_q == 0;
  return hip_status(vx::launch_score_topk(geometry(kv, b), static_cast<const uint16_t*>(q), num_q_heads, (int)kind,
                                          mean, two_pass ? static_cast<const uint16_t*>(mean_bf16) : nullptr,
                                          static_cast<const uint16_t*>(max), static_cast<const uint16_t*>(min),
                                          pages_budget, n_sink, n_local, max_sel, sel_pages, sel_count, workspace,
                                          remap, tau_q, seed, stream, app),
                    name);
}
}  // namespace

vx_status vx_page_score_topk(const void* q, int32_t num_q_heads, const vx_paged_cache* kv, const vx_batch* b,
                             vx_score_kind kind, const float* mean, const void* mean_bf16, const void* max,
                             const void* min,
                             const int32_t* pages_budget, int32_t n_sink, int32_t n_local, int32_t max_sel,
                             int32_t* sel_pages, int32_t* sel_count, void* workspace, size_t workspace_bytes,
                             const vx_topk_options* opt, hipStream_t stream) {
  return score_topk(q, num_q_heads, kv, b, kind, mean, mean_bf16, max, min, pages_budget, n_sink, n_local, max_sel,
                    sel_pages, sel_count, workspace, workspace_bytes, opt, stream, vx::StepAppend{},
                    "vx_page_score_topk");
}

vx_status vx_append_score_topk(const vx_paged_cache* kv, const vx_batch* b, const void* k_new, const void* v_new,
                               float* mean, void* mean_bf16, void* max, void* min, const void* q,
                               int32_t num_q_heads, vx_score_kind kind, const int32_t* pages_budget, int32_t n_sink,
                               int32_t n_local, int32_t max_sel, int32_t* sel_pages, int32_t* sel_count,
                               void* workspace, size_t workspace_bytes, const vx_topk_options* opt,
                               hipStream_t stream) {
  vx_status s;
  if ((s = check_cache(kv, false)) != VX_OK) return s;
  if ((s = check_batch(b)) != VX_OK) return s;
  if (b->batch > 0 && !k_new) return fail(VX_ERR_INVALID_ARG, "k_new must be non-NULL");
  if (kv->v && b->batch > 0 && !v_new) return fail(VX_ERR_INVALID_ARG, "a separate V cache needs v_new");
  if (!kv->v && v_new) return fail(VX_ERR_INVALID_ARG, "v_new given but V is aliased to K (kv->v is NULL)");
  vx::StepAppend app;
  app.k_new = k_new;
  app.v_new = kv->v ? v_new : nullptr;
  app.mean = mean;
  app.mean_bf = static_cast<uint16_t*>(mean_bf16);
  app.maxo = static_cast<uint16_t*>(max);
  app.mino = static_cast<uint16_t*>(min);
  if (b->batch > 0 && n_local < 1) {
    // the appended block is forced only with a local window: append first, then select
    if ((s = hip_status(vx::launch_kv_append_summarize(geometry(kv, b), app.k_new, app.v_new, app.mean, app.mean_bf,
                                                       app.maxo, app.mino, stream),
                        "vx_append_score_topk")) != VX_OK)
      return s;
    app = vx::StepAppend{};
  }
  return score_topk(q, num_q_heads, kv, b, kind, mean, mean_bf16, max, min, pages_budget, n_sink, n_local, max_sel,
                    sel_pages, sel_count, workspace, workspace_bytes, opt, stream, app, "vx_append_score_topk");
}

vx_status vx_page_score(const void* q, int32_t num_q_heads, const vx_paged_cache* kv, const vx_batch* b,
                        vx_score_kind kind, const float* mean, const void* max, const void* min, float* scores,
                        int32_t score_stride, hipStream_t stream) {
  vx_status s;
  if ((s = check_cache(kv, false)) != VX_OK) return s;
  if ((s = check_batch(b)) != VX_OK) return s;
  if ((s = check_heads(kv, num_q_heads)) != VX_OK) return s;
  if (!q || !scores) return fail(VX_ERR_INVALID_ARG, "q and scores must be non-NULL");
  if (score_stride < max_blocks(kv, b))
    return fail(VX_ERR_INVALID_ARG, "score_stride %d < blocks per request %d", score_stride, max_blocks(kv, b));
  if ((s = check_kind(kv, kind, mean, max, min)) != VX_OK) return s;
  if ((int64_t)num_q_heads * kv->head_dim_qk > 16384)
    return fail(VX_ERR_UNSUPPORTED, "scoring keeps q in LDS: num_q_heads * head_dim_qk must be <= 16384");
  return hip_status(vx::launch_score(geometry(kv, b), static_cast<const uint16_t*>(q), num_q_heads, (int)kind, mean,
                                     static_cast<const uint16_t*>(max), static_cast<const uint16_t*>(min), scores,
                                     score_stride, stream),
                    "vx_page_score");
}

vx_status vx_score_flow(vx_score_kind kind, const float* scores_in, float* scores_out, int32_t score_stride,
                        int32_t num_kv_heads, int32_t num_q_heads, int32_t batch, const int32_t* num_items,
                        hipStream_t stream) {
  if (kind != VX_SCORE_NSA && kind != VX_SCORE_MEAN_DOT_SMOOTH)
    return fail(VX_ERR_INVALID_ARG, "vx_score_flow takes the NSA or MEAN_DOT_SMOOTH kind (got %d)", (int)kind);
  if (batch < 0 || batch > 65535) return fail(VX_ERR_INVALID_ARG, "batch %d not in [0, 65535]", batch);
  if (num_kv_heads < 1 || num_kv_heads > 16) return fail(VX_ERR_INVALID_ARG, "num_kv_heads %d not in [1, 16]", num_kv_heads);
  if (num_q_heads < 1 || num_q_heads % num_kv_heads || num_q_heads / num_kv_heads > 16)
    return fail(VX_ERR_INVALID_ARG, "num_q_heads %d must be a multiple of num_kv_heads %d, at most 16 times it",
                num_q_heads, num_kv_heads);
  if (score_stride < 1) return fail(VX_ERR_INVALID_ARG, "score_stride must be >= 1");
  if (batch > 0 && (!scores_in || !scores_out || !num_items))
    return fail(VX_ERR_INVALID_ARG, "scores_in, scores_out and num_items must be non-NULL");
  if (batch > 0 && scores_in == scores_out) return fail(VX_ERR_INVALID_ARG, "scores_in and scores_out must differ");
  return hip_status(vx::launch_score_flow((int)kind, scores_in, scores_out, score_stride, num_kv_heads, num_q_heads,
                                          batch, num_items, 16, 1, score_stride, nullptr, nullptr, stream),
                    "vx_score_flow");
}

vx_status vx_topk_select(const float* scores, int32_t score_stride, int32_t num_kv_heads, int32_t batch,
                         const int32_t* num_items, const int32_t* pages_budget, int32_t n_sink, int32_t n_local,
                         int32_t max_sel, const vx_topk_options* opt, int32_t* sel_pages, int32_t* sel_count,
                         hipStream_t stream) {
  if (batch < 0 || batch > 65535) return fail(VX_ERR_INVALID_ARG, "batch %d not in [0, 65535]", batch);
  if (num_kv_heads < 1 || num_kv_heads > 16) return fail(VX_ERR_INVALID_ARG, "num_kv_heads %d not in [1, 16]", num_kv_heads);
  if (score_stride < 1) return fail(VX_ERR_INVALID_ARG, "score_stride must be >= 1");
  if (batch > 0 && (!scores || !num_items || !pages_budget || !sel_pages || !sel_count))
    return fail(VX_ERR_INVALID_ARG, "scores, num_items, pages_budget, sel_pages and sel_count must be non-NULL");
  if (max_sel < 1) return fail(VX_ERR_INVALID_ARG, "max_sel must be >= 1");
  if (n_sink < 0 || n_local < 0 || (int64_t)n_sink + n_local > max_sel)
    return fail(VX_ERR_INVALID_ARG, "need 0 <= n_sink, 0 <= n_local, n_sink + n_local <= max_sel");
  int remap = 0, tau_q = 0;
  uint32_t seed = 0;
  vx_status s = check_topk_options(opt, &remap, &tau_q, &seed);
  if (s != VX_OK) return s;
  return hip_status(vx::launch_topk_select(scores, score_stride, num_kv_heads, batch, num_items, pages_budget, n_sink,
                                           n_local, max_sel, remap, tau_q, seed, sel_pages, sel_count, stream),
                    "vx_topk_select");
}

}  // extern "C"

namespace {

// Argument checks of the decode entry points.
vx_status check_decode(const void* q, int32_t num_q_heads, const vx_paged_cache* kv, const vx_batch* b,
                       const int32_t* sel_pages, const int32_t* sel_count, int32_t max_sel, float sm_scale,
                       const void* out) {
  vx_status s;
  if ((s = check_cache(kv, true)) != VX_OK) return s;
  if ((s = check_batch(b)) != VX_OK) return s;
  if ((s = check_heads(kv, num_q_heads)) != VX_OK) return s;
  if (!q || !sel_pages || !sel_count || !out)
    return fail(VX_ERR_INVALID_ARG, "q, sel_pages, sel_count and out must be non-NULL");
  if (max_sel < 1) return fail(VX_ERR_INVALID_ARG, "max_sel must be >= 1");
  // the decode kernels index selection slots (below max_sel + 64 * 4 * splits) in 32 bits
  if (max_sel > (1 << 24)) return fail(VX_ERR_UNSUPPORTED, "max_sel above 2^24 is not supported");
  if (!(sm_scale > 0.f) || sm_scale != sm_scale) return fail(VX_ERR_INVALID_ARG, "sm_scale must be positive");
  return VX_OK;
}

}  // namespace

extern "C" {

vx_status vx_sparse_paged_decode(const void* q, int32_t num_q_heads, const vx_paged_cache* kv, const vx_batch* b,
                                 const int32_t* sel_pages, const int32_t* sel_count, int32_t max_sel,
                                 float sm_scale, void* out, void* workspace, size_t workspace_bytes,
                                 hipStream_t stream) {
  vx_status s = check_decode(q, num_q_heads, kv, b, sel_pages, sel_count, max_sel, sm_scale, out);
  if (s != VX_OK) return s;
  const vx::DecodeLayout lay = vx::decode_layout(b->batch, kv->num_kv_heads, num_q_heads / kv->num_kv_heads,
                                                 kv->head_dim_v, max_sel, is_mla(kv));
  if (!workspace || workspace_bytes < lay.total)
    return fail(VX_ERR_WORKSPACE, "decode workspace needs %zu bytes (got %zu)", lay.total, workspace_bytes);
  return hip_status(vx::launch_decode(geometry(kv, b), static_cast<const uint16_t*>(q), num_q_heads, sel_pages,
                                      sel_count, max_sel, sm_scale, static_cast<uint16_t*>(out), workspace, lay,
                                      stream),
                    "vx_sparse_paged_decode");
}

vx_status vx_sparse_paged_decode_noalloc(const void* q, int32_t num_q_heads, const vx_paged_cache* kv,
                                         const vx_batch* b, const int32_t* sel_pages, const int32_t* sel_count,
                                         int32_t max_sel, float sm_scale, void* out, hipStream_t stream) {
  vx_status s = check_decode(q, num_q_heads, kv, b, sel_pages, sel_count, max_sel, sm_scale, out);
  if (s != VX_OK) return s;
  const vx::DecodeLayout lay = vx::decode_layout(b->batch, kv->num_kv_heads, num_q_heads / kv->num_kv_heads,
                                                 kv->head_dim_v, max_sel, is_mla(kv));
  void* scratch = nullptr;
  size_t scratch_bytes = 0;
  if ((s = hip_status(vx::noalloc_scratch(&scratch, &scratch_bytes), "vx_sparse_paged_decode_noalloc")) != VX_OK)
    return s;
  if (lay.total > scratch_bytes)
    return fail(VX_ERR_WORKSPACE,
                "vx_sparse_paged_decode_noalloc: this batch needs %zu bytes of scratch, more than the %zu-byte "
                "static buffer; use vx_sparse_paged_decode with a workspace",
                lay.total, scratch_bytes);
  return hip_status(vx::launch_decode(geometry(kv, b), static_cast<const uint16_t*>(q), num_q_heads, sel_pages,
                                      sel_count, max_sel, sm_scale, static_cast<uint16_t*>(out), scratch, lay,
                                      stream),
                    "vx_sparse_paged_decode_noalloc");
}

vx_status vx_stream_read(const void* buf, size_t bytes, uint32_t* sink, int32_t workgroups, hipStream_t stream) {
  if (!buf || !sink) return fail(VX_ERR_INVALID_ARG, "buf and sink must be non-NULL");
  if (bytes == 0 || bytes % 16 != 0 || (reinterpret_cast<uintptr_t>(buf) & 15) != 0)
    return fail(VX_ERR_INVALID_ARG, "bytes must be a positive multiple of 16 and buf 16-byte aligned");
  if (workgroups < 1 || workgroups > 65536) return fail(VX_ERR_INVALID_ARG, "workgroups %d not in [1, 65536]", workgroups);
  return hip_status(vx::launch_stream_read(buf, (int64_t)bytes, sink, workgroups, stream), "vx_stream_read");
}

}  // extern "C"

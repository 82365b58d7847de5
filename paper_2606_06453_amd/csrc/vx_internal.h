// Host-side launchers shared between the C-ABI layer and the kernel translation units.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace vx {

// ---- work plan and workspace of the decode stage -----------------------------------
// GQA: `splits` workgroups of `waves` waves per (request, KV head) pair, split-major; split s
// covers the selection slots [s*split_slots, (s+1)*split_slots) cut at the pair's count, and
// splits past the count exit at once.  A pair with one split is written directly; the splits
// of a split pair merge in the split kernel through the pair's counter.
// MLA: `splits` workgroups per request over fixed slot ranges, merged by a merge launch.
// Partials: fp32 output and log2-sum-exp per query head, `splits` rows per pair.
// Workspace: [pairs] uint32 split counters (GQA; zero before the first call, every call leaves
// them zero), then the partials.
struct DecodeLayout {
  int32_t splits;             // workgroups (partial rows) per pair
  int32_t split_slots;        // GQA: selection slots per split
  int32_t waves;              // waves per workgroup
  int64_t n_wg;               // grid
  size_t off_ctr, off_lse, off_o, total;
};

// Compute units of the current device (256 when the query fails).
int device_cus();

DecodeLayout decode_layout(int batch, int num_kv_heads, int group, int head_dim_v, int max_sel,
                           bool mla);

// fp32 planes [H][B][stride] of the score stage: max(2 H, Hq + H) of them.  Plane 0 holds the
// scores (or lower bounds), plane 1 the upper bounds; the NSA and smoothing flows put their
// first step (per-query-head logits, block-mean scores) in the planes from H on.
size_t score_workspace_bytes(int batch, int num_kv_heads, int num_q_heads, int max_pages);

// KV cache element types (the values of vx_kv_dtype).
constexpr int kKvBf16 = 0, kKvFp8E4M3 = 1, kKvFp8E5M2 = 2;

struct Geometry {
  const void* k;          // bf16 or fp8 codes (kv_dtype)
  const void* v;          // nullptr: V aliases the first head_dim_v channels of K
  int kv_dtype;
  float k_scale, v_scale; // fp8 cache values are scale * code (1 for bf16)
  int num_phys_pages, H, ps, Dqk, Dv;
  int bs, r;              // block size (tokens) and blocks per page (1: a block is a page)
  int batch, max_pages;   // max_pages: blocks per request bound (max_pages_per_seq * r)
  const int32_t* indptr;
  const int32_t* indices;
  const int32_t* seq_lens;
};

hipError_t launch_summarize(const Geometry& g, const int32_t* first_page, float* mean, uint16_t* mean_bf,
                            uint16_t* maxo, uint16_t* mino, hipStream_t stream);

// The decode step's cache stage in one launch: k_new / v_new rows written at token L_i - 1
// (v_new nullptr: V aliased), then that page's summaries.
hipError_t launch_kv_append_summarize(const Geometry& g, const void* k_new, const void* v_new, float* mean,
                                      uint16_t* mean_bf, uint16_t* maxo, uint16_t* mino, hipStream_t stream);

// mean_bf != nullptr (MEAN_DOT only, max_pages <= kTwoPassMaxPages) selects the exact
// two-pass path: a bounded first pass over the bf16 means, then fp32 re-scoring of the
// undecided pages.
constexpr int kTwoPassMaxPages = 4096;
// remap / tau_q / seed other than 0: the approximate radix top-k of vx_topk_select on the
// one-pass scores (the two-pass block-mean path and the bucketed selection are exact only).
// The decode step's cache stage carried by the selection launch: k_new / v_new rows appended
// at token seq_lens[i] - 1 and that block's summaries refreshed (the summary buffers' contents
// before the call are what the score launch reads).  k_new == nullptr: none.
struct StepAppend {
  const void* k_new = nullptr;
  const void* v_new = nullptr;
  float* mean = nullptr;
  uint16_t* mean_bf = nullptr;
  uint16_t* maxo = nullptr;
  uint16_t* mino = nullptr;
};
hipError_t launch_score_topk(const Geometry& g, const uint16_t* q, int Hq, int kind, const float* mean,
                             const uint16_t* mean_bf, const uint16_t* maxs, const uint16_t* mins,
                             const int32_t* budget, int n_sink, int n_local, int max_sel, int32_t* sel_pages,
                             int32_t* sel_count, void* ws, int remap, int tau_q, uint32_t seed, hipStream_t stream,
                             const StepAppend& app = StepAppend{});

// One-pass fp32 scores of every page into scores[h][i][j] (row stride `stride`).
hipError_t launch_score(const Geometry& g, const uint16_t* q, int Hq, int kind, const float* mean,
                        const uint16_t* maxs, const uint16_t* mins, float* scores, int stride, hipStream_t stream);

// The last steps of the NSA (kind 7) and smoothing (kind 8) flows: in [rows][batch][stride] ->
// out [H][batch][stride], items[i] pages per request (items == nullptr: from seq_lens).
hipError_t launch_score_flow(int kind, const float* in, float* out, int stride, int H, int Hq, int batch,
                             const int32_t* items, int ps, int r, int max_pages, const int32_t* indptr,
                             const int32_t* seq_lens, hipStream_t stream);

// Radix selection from fp32 scores [H][batch][stride] with items[i] pages per request; remap
// and tau_q (16-bit fixed-point tolerate ratio) as in the approximate top-k.
hipError_t launch_topk_select(const float* scores, int stride, int H, int batch, const int32_t* items,
                              const int32_t* budget, int n_sink, int n_local, int max_sel, int remap, int tau_q,
                              uint32_t seed, int32_t* sel_pages, int32_t* sel_count, hipStream_t stream);

// Plain stream of 16-byte non-temporal loads over `bytes` (a multiple of 16) from buf.
hipError_t launch_stream_read(const void* buf, int64_t bytes, uint32_t* sink, int workgroups, hipStream_t stream);

// The per-device scratch of the allocation-free decode entry point: its device address (from
// hipGetSymbolAddress, resolved once per device) and size.
hipError_t noalloc_scratch(void** ptr, size_t* bytes);

hipError_t launch_decode(const Geometry& g, const uint16_t* q, int Hq, const int32_t* sel_pages,
                         const int32_t* sel_count, int max_sel, float sm_scale, uint16_t* out, void* ws,
                         const DecodeLayout& lay, hipStream_t stream);

}  // namespace vx

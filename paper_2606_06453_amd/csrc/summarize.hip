// Cache stage: per-page Mean / Max / Min key summaries (Sec. 3.1 Eq. 1; Sec. 3.2 Quest).
//
// Work decomposition: a task is 8 consecutive channels (16 bytes of bf16, 8 of fp8) of one
// (page, KV head) slice.  TS adjacent lanes share a task and take every TS-th valid token; quad DPP
// combines them (TS = 1 for a full pass over many pages, TS = 2 or 4 at a decode step where
// only one page per request changes).  Each lane loads up to 8 token rows per round trip.  A token row of a slice is D*2 contiguous bytes, so a load
// instruction reads whole rows of several slices.  HBM-bound: it reads page_size*D*2 bytes
// (page_size*D for an fp8 cache) and writes D*(4 + 2 + 2) bytes per (page, head).
// fp8 caches: each code is converted exactly to fp32 and multiplied by the K scale (one fp32
// rounding), which is the cache value the summaries are taken over.
//
// Append mode (the decode step's cache stage fused into one launch): request i's new key and
// value rows are written at token L_i - 1, and the page holding it is summarised in the same
// pass.  The new key row is taken from the step's input, not read back, and enters the
// running sums last, exactly where a separate summarize pass over the page would add it, so
// the summaries are bit-identical to an append followed by vx_page_summarize.
//
// Blocks below the page size (r = ps / bs blocks per page): the unit is the block.  Logical
// block j of request i is block j % r of physical page indices[j / r], its summary row is
// (p * r + j % r), and every page count above is a block count.  r = 1 is the page case.
#include <type_traits>

#include "summary_task.h"
#include "vx_device.h"
#include "vx_internal.h"

namespace vx {
namespace {

constexpr int kThreads = 256;
using summ::AppendArgs;

template <int TS, int KT, bool APPEND, int KB>
__global__ __launch_bounds__(kThreads) void summarize_kernel(
    const void* __restrict__ kv, float k_scale, int num_phys, int H, int ps, int bs, int r, int D, int max_pages,
    const int32_t* __restrict__ indptr, const int32_t* __restrict__ indices,
    const int32_t* __restrict__ seq_lens, const int32_t* __restrict__ first_page,
    float* __restrict__ mean, uint16_t* __restrict__ mean_bf, uint16_t* __restrict__ maxo,
    uint16_t* __restrict__ mino, int pages_per_block, int split_tasks, const AppendArgs app) {
  const int i = blockIdx.y;
  const int L = seq_lens[i];
  const int base = indptr[i];
  int P = num_pages(L, bs, (indptr[i + 1] - base) * r, max_pages);     // blocks
  int j0 = first_page ? first_page[i] : 0;
  if constexpr (APPEND) {
    j0 = (L - 1) / bs;                   // the block receiving token L - 1, and only that one
    P = min(P, j0 + 1);
  }
  j0 = j0 < 0 ? 0 : j0;
  const int chunks = D / 8;
  const int tasks_per_page = H * chunks;

  static_assert(TS == 1 || TS == 2 || TS == 4, "token slices per task");
  const int slice = (int)threadIdx.x % TS;
  // Decode-step launches (split_tasks): the x workgroups of a request share out the tasks of
  // each page from j0 on.  Full passes: workgroup x takes pages x*pages_per_block.. with stride.
  const int x_pg = split_tasks ? 0 : (int)blockIdx.x, n_pg = split_tasks ? 1 : (int)gridDim.x;
  const int t_first = split_tasks ? (int)blockIdx.x * (kThreads / TS) : 0;
  const int t_step = split_tasks ? (int)gridDim.x * (kThreads / TS) : kThreads / TS;
  for (int jb = j0 + x_pg * pages_per_block; jb < P; jb += n_pg * pages_per_block) {
    const int nj = min(pages_per_block, P - jb);
    const int ntask = nj * tasks_per_page;
    // t0 is uniform over the workgroup: every lane of a quad runs the same task count, so the
    // DPP combine sees full quads
    for (int t0 = t_first; t0 < ntask; t0 += t_step) {
      const int task = t0 + (int)threadIdx.x / TS;
      const bool active = task < ntask;
      const int tk = active ? task : 0;
      const int jj = tk / tasks_per_page;
      const int rem = tk - jj * tasks_per_page;
      const int h = rem / chunks;
      const int c8 = rem - h * chunks;
      const int j = jb + jj;                              // logical block
      summ::task<TS, KT, APPEND, KB>(kv, k_scale, num_phys, H, ps, bs, r, D, indices, base, L, i, j, h, c8, active,
                                     slice, mean, mean_bf, maxo, mino, app);
    }
  }
}

// Workgroups per request at a decode step: one per 64 tasks (8-channel chunks of a page's
// heads), so each of a task's 4 lanes walks at most page_size / 4 token rows.
int step_wgs(const Geometry& g) {
  const int tasks_per_page = g.H * (g.Dqk / 8);
  return (tasks_per_page + kThreads / 4 - 1) / (kThreads / 4);
}

template <int TS, bool APPEND = false, int KB = summ::kBatch>
void dispatch(const Geometry& g, const int32_t* first_page, float* mean, uint16_t* mean_bf, uint16_t* maxo,
              uint16_t* mino, dim3 grid, int ppb, int split, hipStream_t stream, const AppendArgs& app = AppendArgs{}) {
#define VX_SUMMARIZE(KT)                                                                                        \
  hipLaunchKernelGGL((summarize_kernel<TS, KT, APPEND, KB>), grid, dim3(kThreads), 0, stream, g.k, g.k_scale,   \
                     g.num_phys_pages, g.H, g.ps, g.bs, g.r, g.Dqk, g.max_pages, g.indptr, g.indices, g.seq_lens,  \
                     first_page,                                                                                 \
                     mean, mean_bf, maxo, mino, ppb, split, app)
  if (g.kv_dtype == kKvFp8E4M3) VX_SUMMARIZE(kKvFp8E4M3);
  else if (g.kv_dtype == kKvFp8E5M2) VX_SUMMARIZE(kKvFp8E5M2);
  else VX_SUMMARIZE(kKvBf16);
#undef VX_SUMMARIZE
}

}  // namespace

hipError_t launch_summarize(const Geometry& g, const int32_t* first_page, float* mean, uint16_t* mean_bf,
                            uint16_t* maxo, uint16_t* mino, hipStream_t stream) {
  if (g.batch == 0) return hipSuccess;
  const int tasks_per_page = g.H * (g.Dqk / 8);
  if (first_page) {
    // decode step: usually one new page per request, whose tasks are shared out over
    // step_wgs() workgroups of the request, 4 lanes per task splitting its tokens
    if (g.bs > 4 * summ::kBatch)   // blocks of 64 tokens: a lane's 16 rows in one round trip
      dispatch<4, false, 2 * summ::kBatch>(g, first_page, mean, mean_bf, maxo, mino, dim3(step_wgs(g), g.batch), 1,
                                           1, stream);
    else
      dispatch<4>(g, first_page, mean, mean_bf, maxo, mino, dim3(step_wgs(g), g.batch), 1, 1, stream);
  } else {
    const int ppb = tasks_per_page >= 4 * kThreads ? 1 : (4 * kThreads) / tasks_per_page;
    int gx = (g.max_pages + ppb - 1) / ppb;
    if (gx < 1) gx = 1;
    dispatch<1>(g, first_page, mean, mean_bf, maxo, mino, dim3(gx, g.batch), ppb, 0, stream);
  }
  return hipGetLastError();
}

hipError_t launch_kv_append_summarize(const Geometry& g, const void* k_new, const void* v_new, float* mean,
                                      uint16_t* mean_bf, uint16_t* maxo, uint16_t* mino, hipStream_t stream) {
  if (g.batch == 0) return hipSuccess;
  const AppendArgs app{k_new, v_new, const_cast<void*>(g.k), const_cast<void*>(g.v)};
  // the launch shape of the decode step's incremental summary (same token slices, so the
  // summaries come out bit-identical)
  if (g.bs > 4 * summ::kBatch)     // blocks of 64 tokens: a lane's 16 rows in one round trip
    dispatch<4, true, 2 * summ::kBatch>(g, nullptr, mean, mean_bf, maxo, mino, dim3(step_wgs(g), g.batch), 1, 1,
                                        stream, app);
  else
    dispatch<4, true>(g, nullptr, mean, mean_bf, maxo, mino, dim3(step_wgs(g), g.batch), 1, 1, stream, app);
  return hipGetLastError();
}

}  // namespace vx

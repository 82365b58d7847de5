// Cache stage: per-page Mean / Max / Min key summaries (Sec. 3.1 Eq. 1; Sec. 3.2 Quest).
//
// Work decomposition: one thread owns 8 consecutive channels (16 bytes) of one
// (page, KV head) slice and walks that slice's valid tokens.  A token row of a slice is
// D*2 contiguous bytes, so the threads of a wave read whole rows of several slices per
// load instruction.  HBM-bound: it reads page_size*D*2 bytes and writes
// D*(4 + 2 + 2) bytes per (page, head).  No cross-lane reduction is needed.
#include "vx_device.h"
#include "vx_internal.h"

namespace vx {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void summarize_kernel(
    const uint16_t* __restrict__ k, int num_phys, int H, int ps, int D, int max_pages,
    const int32_t* __restrict__ indptr, const int32_t* __restrict__ indices,
    const int32_t* __restrict__ seq_lens, const int32_t* __restrict__ first_page,
    float* __restrict__ mean, uint16_t* __restrict__ maxo, uint16_t* __restrict__ mino,
    int pages_per_block) {
  const int i = blockIdx.y;
  const int L = seq_lens[i];
  const int base = indptr[i];
  const int P = num_pages(L, ps, indptr[i + 1] - base, max_pages);
  int j0 = first_page ? first_page[i] : 0;
  j0 = j0 < 0 ? 0 : j0;
  const int chunks = D / 8;
  const int tasks_per_page = H * chunks;

  for (int jb = j0 + (int)blockIdx.x * pages_per_block; jb < P; jb += (int)gridDim.x * pages_per_block) {
    const int nj = min(pages_per_block, P - jb);
    for (int task = threadIdx.x; task < nj * tasks_per_page; task += kThreads) {
      const int jj = task / tasks_per_page;
      const int rem = task - jj * tasks_per_page;
      const int h = rem / chunks;
      const int c8 = rem - h * chunks;
      const int j = jb + jj;
      const int64_t p = clamp_page(indices[base + j], num_phys);
      const int n = min(ps, L - j * ps);
      const uint16_t* src = k + (p * H + h) * (int64_t)ps * D + c8 * 8;

      float s[8], mx[8], mn[8];
#pragma unroll
      for (int e = 0; e < 8; e++) {
        s[e] = 0.f;
        mx[e] = -INFINITY;
        mn[e] = INFINITY;
      }
#pragma unroll 4
      for (int t = 0; t < n; t++) {
        const uint4 w = *reinterpret_cast<const uint4*>(src + (int64_t)t * D);
        const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int e2 = 0; e2 < 4; e2++) {
          const float a = bf16lo(ws[e2]), b = bf16hi(ws[e2]);
          s[2 * e2] += a;
          s[2 * e2 + 1] += b;
          mx[2 * e2] = fmaxf(mx[2 * e2], a);
          mx[2 * e2 + 1] = fmaxf(mx[2 * e2 + 1], b);
          mn[2 * e2] = fminf(mn[2 * e2], a);
          mn[2 * e2 + 1] = fminf(mn[2 * e2 + 1], b);
        }
      }
      const int64_t o = (p * H + h) * (int64_t)D + c8 * 8;
      if (mean) {
        const float nf = (float)n;   // correctly rounded division below
        float4 a = make_float4(s[0] / nf, s[1] / nf, s[2] / nf, s[3] / nf);
        float4 b = make_float4(s[4] / nf, s[5] / nf, s[6] / nf, s[7] / nf);
        *reinterpret_cast<float4*>(mean + o) = a;
        *reinterpret_cast<float4*>(mean + o + 4) = b;
      }
      // Max and Min of bf16 values are bf16 values: truncating the fp32 bits is exact.
      if (maxo) {
        uint4 w;
        w.x = (__float_as_uint(mx[0]) >> 16) | (__float_as_uint(mx[1]) & 0xffff0000u);
        w.y = (__float_as_uint(mx[2]) >> 16) | (__float_as_uint(mx[3]) & 0xffff0000u);
        w.z = (__float_as_uint(mx[4]) >> 16) | (__float_as_uint(mx[5]) & 0xffff0000u);
        w.w = (__float_as_uint(mx[6]) >> 16) | (__float_as_uint(mx[7]) & 0xffff0000u);
        *reinterpret_cast<uint4*>(maxo + o) = w;
      }
      if (mino) {
        uint4 w;
        w.x = (__float_as_uint(mn[0]) >> 16) | (__float_as_uint(mn[1]) & 0xffff0000u);
        w.y = (__float_as_uint(mn[2]) >> 16) | (__float_as_uint(mn[3]) & 0xffff0000u);
        w.z = (__float_as_uint(mn[4]) >> 16) | (__float_as_uint(mn[5]) & 0xffff0000u);
        w.w = (__float_as_uint(mn[6]) >> 16) | (__float_as_uint(mn[7]) & 0xffff0000u);
        *reinterpret_cast<uint4*>(mino + o) = w;
      }
    }
  }
}

}  // namespace

hipError_t launch_summarize(const Geometry& g, const int32_t* first_page, float* mean, uint16_t* maxo,
                            uint16_t* mino, hipStream_t stream) {
  if (g.batch == 0) return hipSuccess;
  const int tasks_per_page = g.H * (g.Dqk / 8);
  int ppb, gx;
  if (first_page) {
    // decode step: usually one new page per request
    ppb = tasks_per_page >= kThreads ? 1 : kThreads / tasks_per_page;
    gx = 1;
  } else {
    ppb = tasks_per_page >= 4 * kThreads ? 1 : (4 * kThreads) / tasks_per_page;
    gx = (g.max_pages + ppb - 1) / ppb;
    if (gx < 1) gx = 1;
  }
  dim3 grid(gx, g.batch);
  hipLaunchKernelGGL(summarize_kernel, grid, dim3(kThreads), 0, stream, g.k, g.num_phys_pages, g.H, g.ps, g.Dqk, g.max_pages,
                     g.indptr, g.indices, g.seq_lens, first_page, mean, maxo, mino, ppb);
  return hipGetLastError();
}

}  // namespace vx

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

#include "vx_device.h"
#include "vx_internal.h"

namespace vx {
namespace {

constexpr int kThreads = 256;
constexpr int kBatch = 8;        // token rows a lane loads per round trip

template <int CTRL>
__device__ __forceinline__ float quad_dpp(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xf, 0xf, false));
}

// 8 consecutive channels of one token row: raw bits and their fp32 values.
template <int KT>
struct RowChunk {
  using Raw = typename std::conditional<KT == kKvBf16, uint4, uint2>::type;
  static constexpr int kBytes = KT == kKvBf16 ? 16 : 8;
  __device__ static __forceinline__ void values(const Raw& w, float scale, float (&x)[8]) {
    if constexpr (KT == kKvBf16) {
      const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int e2 = 0; e2 < 4; e2++) {
        x[2 * e2] = bf16lo(ws[e2]);
        x[2 * e2 + 1] = bf16hi(ws[e2]);
      }
    } else {
      const int ws[2] = {(int)w.x, (int)w.y};
#pragma unroll
      for (int h = 0; h < 2; h++) {
        float2_t lo, hi;
        if constexpr (KT == kKvFp8E4M3) {
          lo = __builtin_amdgcn_cvt_pk_f32_fp8(ws[h], false);
          hi = __builtin_amdgcn_cvt_pk_f32_fp8(ws[h], true);
        } else {
          lo = __builtin_amdgcn_cvt_pk_f32_bf8(ws[h], false);
          hi = __builtin_amdgcn_cvt_pk_f32_bf8(ws[h], true);
        }
        x[4 * h] = lo[0] * scale;
        x[4 * h + 1] = lo[1] * scale;
        x[4 * h + 2] = hi[0] * scale;
        x[4 * h + 3] = hi[1] * scale;
      }
    }
  }
};

// Append mode: the step's rows, k_new [batch][H][D] and v_new [batch][H][Dv] (v_new null: V
// aliased), and the caches they are written to (the same buffers the kernel reads k from).
struct AppendArgs {
  const void* knew;
  const void* vnew;
  void* kw;
  void* vw;
};

template <int TS, int KT, bool APPEND>
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
      const int64_t p = clamp_page(indices[base + j / r], num_phys);
      const int blk = j - (j / r) * r;                    // block within the page
      const int n = active ? min(bs, L - j * bs) : 0;
      using RC = RowChunk<KT>;
      // element offset of the block's first token row, channel chunk c8
      const int64_t row0 = (p * H + h) * (int64_t)ps * D + (int64_t)blk * bs * D + c8 * 8;
      const char* src = static_cast<const char*>(kv) + row0 * (RC::kBytes / 8);
      const int64_t row_bytes = (int64_t)D * (RC::kBytes / 8);
      // append: the new token is row n - 1 of this page; its chunk comes from the step's input
      const int n_mem = APPEND ? n - 1 : n;
      typename RC::Raw new_row{};
      if constexpr (APPEND) {
        new_row = *reinterpret_cast<const typename RC::Raw*>(static_cast<const char*>(app.knew) +
                                                              (((int64_t)i * H + h) * D + c8 * 8) * (RC::kBytes / 8));
        if (active && slice == 0) {
          *reinterpret_cast<typename RC::Raw*>(static_cast<char*>(app.kw) +
                                               (row0 + (int64_t)(n - 1) * D) * (RC::kBytes / 8)) = new_row;
          if (app.vnew)   // V rows have D channels too (GQA); an aliased V has no rows of its own
            *reinterpret_cast<typename RC::Raw*>(static_cast<char*>(app.vw) +
                                                 (row0 + (int64_t)(n - 1) * D) * (RC::kBytes / 8)) =
                *reinterpret_cast<const typename RC::Raw*>(static_cast<const char*>(app.vnew) +
                                                           (((int64_t)i * H + h) * D + c8 * 8) * (RC::kBytes / 8));
        }
      }

      float s[8], mx[8], mn[8];
#pragma unroll
      for (int e = 0; e < 8; e++) {
        s[e] = 0.f;
        mx[e] = -INFINITY;
        mn[e] = INFINITY;
      }
      // kBatch token rows per round trip: clamped, unconditional loads, then guarded adds
      for (int t0 = slice; t0 < n_mem; t0 += TS * kBatch) {
        typename RC::Raw w[kBatch];
#pragma unroll
        for (int b = 0; b < kBatch; b++)
          w[b] = *reinterpret_cast<const typename RC::Raw*>(src + (int64_t)min(t0 + TS * b, n_mem - 1) * row_bytes);
#pragma unroll
        for (int b = 0; b < kBatch; b++) {
          if (t0 + TS * b >= n_mem) break;
          float x[8];
          RC::values(w[b], k_scale, x);
#pragma unroll
          for (int e = 0; e < 8; e++) {
            s[e] += x[e];
            mx[e] = fmaxf(mx[e], x[e]);
            mn[e] = fminf(mn[e], x[e]);
          }
        }
      }
      if constexpr (APPEND) {
        if (n >= 1 && slice == (n - 1) % TS) {   // the new token, last in its slice's order
          float x[8];
          RC::values(new_row, k_scale, x);
#pragma unroll
          for (int e = 0; e < 8; e++) {
            s[e] += x[e];
            mx[e] = fmaxf(mx[e], x[e]);
            mn[e] = fminf(mn[e], x[e]);
          }
        }
      }
      if (TS >= 2) {
        // combine the token slices of a pair (quad_perm [1,0,3,2]) and of a quad ([2,3,0,1])
#pragma unroll
        for (int e = 0; e < 8; e++) {
          s[e] += quad_dpp<0xB1>(s[e]);
          mx[e] = fmaxf(mx[e], quad_dpp<0xB1>(mx[e]));
          mn[e] = fminf(mn[e], quad_dpp<0xB1>(mn[e]));
          if (TS == 4) {
            s[e] += quad_dpp<0x4E>(s[e]);
            mx[e] = fmaxf(mx[e], quad_dpp<0x4E>(mx[e]));
            mn[e] = fminf(mn[e], quad_dpp<0x4E>(mn[e]));
          }
        }
      }
      if (!active || slice != 0) continue;
      const int64_t o = ((p * r + blk) * H + h) * (int64_t)D + c8 * 8;
      if (mean || mean_bf) {
        const float nf = (float)n;   // correctly rounded division below
        float m8[8];
#pragma unroll
        for (int e = 0; e < 8; e++) m8[e] = s[e] / nf;
        if (mean) {
          *reinterpret_cast<float4*>(mean + o) = make_float4(m8[0], m8[1], m8[2], m8[3]);
          *reinterpret_cast<float4*>(mean + o + 4) = make_float4(m8[4], m8[5], m8[6], m8[7]);
        }
        if (mean_bf) {
          uint4 w;
          w.x = f32_to_bf16_rne(m8[0]) | (f32_to_bf16_rne(m8[1]) << 16);
          w.y = f32_to_bf16_rne(m8[2]) | (f32_to_bf16_rne(m8[3]) << 16);
          w.z = f32_to_bf16_rne(m8[4]) | (f32_to_bf16_rne(m8[5]) << 16);
          w.w = f32_to_bf16_rne(m8[6]) | (f32_to_bf16_rne(m8[7]) << 16);
          *reinterpret_cast<uint4*>(mean_bf + o) = w;
        }
      }
      // Max and Min of bf16 values are bf16 values: truncating the fp32 bits is exact.  Those
      // of fp8 cache values are rounded to nearest even.
      auto pack = [](float a, float b) -> uint32_t {
        if constexpr (KT == kKvBf16) return (__float_as_uint(a) >> 16) | (__float_as_uint(b) & 0xffff0000u);
        else return f32_to_bf16_rne(a) | (f32_to_bf16_rne(b) << 16);
      };
      if (maxo) {
        *reinterpret_cast<uint4*>(maxo + o) = make_uint4(pack(mx[0], mx[1]), pack(mx[2], mx[3]), pack(mx[4], mx[5]),
                                                         pack(mx[6], mx[7]));
      }
      if (mino) {
        *reinterpret_cast<uint4*>(mino + o) = make_uint4(pack(mn[0], mn[1]), pack(mn[2], mn[3]), pack(mn[4], mn[5]),
                                                         pack(mn[6], mn[7]));
      }
    }
  }
}

// Workgroups per request at a decode step: one per 64 tasks (8-channel chunks of a page's
// heads), so each of a task's 4 lanes walks at most page_size / 4 token rows.
int step_wgs(const Geometry& g) {
  const int tasks_per_page = g.H * (g.Dqk / 8);
  return (tasks_per_page + kThreads / 4 - 1) / (kThreads / 4);
}

template <int TS, bool APPEND = false>
void dispatch(const Geometry& g, const int32_t* first_page, float* mean, uint16_t* mean_bf, uint16_t* maxo,
              uint16_t* mino, dim3 grid, int ppb, int split, hipStream_t stream, const AppendArgs& app = AppendArgs{}) {
#define VX_SUMMARIZE(KT)                                                                                        \
  hipLaunchKernelGGL((summarize_kernel<TS, KT, APPEND>), grid, dim3(kThreads), 0, stream, g.k, g.k_scale,       \
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
  dispatch<4, true>(g, nullptr, mean, mean_bf, maxo, mino, dim3(step_wgs(g), g.batch), 1, 1, stream, app);
  return hipGetLastError();
}

}  // namespace vx

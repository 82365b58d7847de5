// Indexer stage: page scores (Sec. 3.1 Eq. 2; Sec. 3.2 Quest) and the selection of sink,
// local and top-scoring pages (Sec. 3.1 Eq. 3; Sec. 6.4 setup).
//
// score_kernel   HBM-bound stream over the summaries.  A row of 16 lanes owns one
//                (page, KV head) item.  Each lane holds D/16 channels of the summary and
//                of the query view.  Products accumulate in fp64 and reduce across the row
//                with DPP, then round once to fp32.  Output goes to a padded scratch table
//                scores[h][i][j].
// topk_kernel    One workgroup per (request, KV head).  It runs an exact radix select
//                (4 passes of 8-bit digits over an order-preserving uint32 key of the fp32
//                score, LDS histogram) to find the K_free-th best candidate.  Ties at the
//                threshold go to the lowest page index: a ballot/popcount prefix count gives
//                each tied page its rank.  A second prefix count compacts forced and chosen
//                pages in ascending order.
#include "vx_device.h"
#include "vx_internal.h"

namespace vx {
namespace {

constexpr int kThreads = 256;
constexpr int kRows = kThreads / 16;     // 16-lane rows per workgroup
constexpr int kUnroll = 4;               // items per row kept in flight

enum { kMeanDot = 0, kQuest = 1, kMaxDot = 2 };

template <int E>
__device__ __forceinline__ void load_f32(const float* p, float (&x)[E]) {
  static_assert(E % 4 == 0, "E multiple of 4");
#pragma unroll
  for (int v = 0; v < E / 4; v++) {
    const float4 w = *reinterpret_cast<const float4*>(p + 4 * v);
    x[4 * v] = w.x;
    x[4 * v + 1] = w.y;
    x[4 * v + 2] = w.z;
    x[4 * v + 3] = w.w;
  }
}

template <int E>
__device__ __forceinline__ void load_bf16(const uint16_t* p, float (&x)[E]) {
  static_assert(E % 4 == 0, "E multiple of 4");
#pragma unroll
  for (int v = 0; v < E / 4; v++) {
    const uint2 w = *reinterpret_cast<const uint2*>(p + 4 * v);
    x[4 * v] = bf16lo(w.x);
    x[4 * v + 1] = bf16hi(w.x);
    x[4 * v + 2] = bf16lo(w.y);
    x[4 * v + 3] = bf16hi(w.y);
  }
}

// ------------------------------------------------------------------------------------
// scores for MEAN_DOT / MAX_DOT: s_j = (mean_r q_r) . S_j  (equal to the mean over the
// group's heads of q_r . S_j by linearity).  The group-mean query is formed in fp64 (the
// sum of bf16 values is exact) and stays in registers: a row always serves the same head.
// ------------------------------------------------------------------------------------
template <int KIND, int D>
__global__ __launch_bounds__(kThreads) void score_dot_kernel(
    const uint16_t* __restrict__ q, int Hq, int H, int ps, int num_phys, int max_pages, int batch,
    const int32_t* __restrict__ indptr, const int32_t* __restrict__ indices,
    const int32_t* __restrict__ seq_lens, const float* __restrict__ mean,
    const uint16_t* __restrict__ maxs, float* __restrict__ scores, int pages_per_block) {
  constexpr int E = D / 16;
  const int i = blockIdx.y;
  const int base = indptr[i];
  const int P = num_pages(seq_lens[i], ps, indptr[i + 1] - base, max_pages);
  const int row = threadIdx.x >> 4, u = threadIdx.x & 15;
  const int h = row % H, slot = row / H, slots = kRows / H;
  const int g = Hq / H;

  double qb[E];
  {
    const uint16_t* qi = q + ((int64_t)i * Hq + (int64_t)h * g) * D + u * E;
#pragma unroll
    for (int e = 0; e < E; e++) qb[e] = 0.0;
    for (int r = 0; r < g; r++) {
      float x[E];
      load_bf16<E>(qi + (int64_t)r * D, x);
#pragma unroll
      for (int e = 0; e < E; e++) qb[e] += (double)x[e];
    }
#pragma unroll
    for (int e = 0; e < E; e++) qb[e] /= (double)g;
  }

  float* out = scores + ((int64_t)h * batch + i) * max_pages;
  for (int jb = (int)blockIdx.x * pages_per_block; jb < P; jb += (int)gridDim.x * pages_per_block) {
    const int nj = min(pages_per_block, P - jb);
    for (int j0 = slot; j0 < nj; j0 += kUnroll * slots) {
      float x[kUnroll][E];
#pragma unroll
      for (int v = 0; v < kUnroll; v++) {
        const int jj = j0 + v * slots;
        if (jj < nj) {
          const int64_t p = clamp_page(indices[base + jb + jj], num_phys);
          const int64_t o = (p * H + h) * D + u * E;
          if (KIND == kMeanDot) load_f32<E>(mean + o, x[v]);
          else load_bf16<E>(maxs + o, x[v]);
        }
      }
#pragma unroll
      for (int v = 0; v < kUnroll; v++) {
        const int jj = j0 + v * slots;
        if (jj < nj) {
          double acc = 0.0;
#pragma unroll
          for (int e = 0; e < E; e++) acc = fma(qb[e], (double)x[v][e], acc);
          acc = row16_sum_f64(acc);
          if (u == 0) out[jb + jj] = (float)acc;
        }
      }
    }
  }
}

// ------------------------------------------------------------------------------------
// Quest: s_j = max_r sum_c max(q_rc Max_jc, q_rc Min_jc).  Each product of two bf16 values
// is exact in fp32; the per-head sums run in fp64.  The group's query heads sit in LDS as
// fp32 [g][D] per KV head.
// ------------------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kThreads) void score_quest_kernel(
    const uint16_t* __restrict__ q, int Hq, int H, int ps, int num_phys, int max_pages, int batch,
    const int32_t* __restrict__ indptr, const int32_t* __restrict__ indices,
    const int32_t* __restrict__ seq_lens, const uint16_t* __restrict__ maxs,
    const uint16_t* __restrict__ mins, float* __restrict__ scores, int pages_per_block) {
  constexpr int E = D / 16;
  extern __shared__ float qs[];        // [Hq][D]
  const int i = blockIdx.y;
  const int base = indptr[i];
  const int P = num_pages(seq_lens[i], ps, indptr[i + 1] - base, max_pages);
  const int row = threadIdx.x >> 4, u = threadIdx.x & 15;
  const int h = row % H, slot = row / H, slots = kRows / H;
  const int g = Hq / H;

  for (int x = threadIdx.x; x < Hq * D; x += kThreads) qs[x] = bf16_to_f32(q[(int64_t)i * Hq * D + x]);
  __syncthreads();

  float* out = scores + ((int64_t)h * batch + i) * max_pages;
  for (int jb = (int)blockIdx.x * pages_per_block; jb < P; jb += (int)gridDim.x * pages_per_block) {
    const int nj = min(pages_per_block, P - jb);
    for (int j0 = slot; j0 < nj; j0 += kUnroll * slots) {
      float mx[kUnroll][E], mn[kUnroll][E];
#pragma unroll
      for (int v = 0; v < kUnroll; v++) {
        const int jj = j0 + v * slots;
        if (jj < nj) {
          const int64_t p = clamp_page(indices[base + jb + jj], num_phys);
          const int64_t o = (p * H + h) * D + u * E;
          load_bf16<E>(maxs + o, mx[v]);
          load_bf16<E>(mins + o, mn[v]);
        }
      }
#pragma unroll
      for (int v = 0; v < kUnroll; v++) {
        const int jj = j0 + v * slots;
        if (jj < nj) {
          double best = -INFINITY;
          for (int r = 0; r < g; r++) {
            const float* qr = qs + (h * g + r) * D + u * E;
            double acc = 0.0;
#pragma unroll
            for (int e = 0; e < E; e++) {
              const float a = qr[e] * mx[v][e];      // exact
              const float b = qr[e] * mn[v][e];      // exact
              acc += (double)fmaxf(a, b);
            }
            acc = row16_sum_f64(acc);
            best = acc > best ? acc : best;
          }
          if (u == 0) out[jb + jj] = (float)best;
        }
      }
    }
  }
}

// ------------------------------------------------------------------------------------
// top-K selection, one workgroup per (request, KV head)
// ------------------------------------------------------------------------------------
__device__ __forceinline__ bool is_forced(int j, int P, int n_sink, int n_local) {
  return j < n_sink || j >= P - n_local;
}

// Block-wide exclusive prefix count of `pred` in thread order; returns the block total.
__device__ __forceinline__ int block_excl_count(bool pred, int* prefix, int* wave_tot) {
  const int w = threadIdx.x >> 6;
  int wt;
  const int lp = wave_excl_count(pred, &wt);
  if (lane_id() == 0) wave_tot[w] = wt;
  __syncthreads();
  int before = 0, total = 0;
#pragma unroll
  for (int x = 0; x < kThreads / kWave; x++) {
    const int t = wave_tot[x];
    before += (x < w) ? t : 0;
    total += t;
  }
  __syncthreads();
  *prefix = before + lp;
  return total;
}

__global__ __launch_bounds__(kThreads) void topk_kernel(
    const float* __restrict__ scores, int H, int ps, int max_pages, int batch,
    const int32_t* __restrict__ indptr, const int32_t* __restrict__ seq_lens,
    const int32_t* __restrict__ budget, int n_sink, int n_local, int max_sel,
    int32_t* __restrict__ sel_pages, int32_t* __restrict__ sel_count) {
  __shared__ int hist[256];
  __shared__ int wave_tot[kThreads / kWave];
  __shared__ int pick[3];              // digit, count above the digit's bin, bin count

  const int i = blockIdx.x / H, h = blockIdx.x % H;
  const int P = num_pages(seq_lens[i], ps, indptr[i + 1] - indptr[i], max_pages);
  int Ktot = budget[i];
  Ktot = Ktot < max_sel ? Ktot : max_sel;
  Ktot = Ktot < 0 ? 0 : Ktot;
  const float* s = scores + ((int64_t)h * batch + i) * max_pages;
  int32_t* out = sel_pages + ((int64_t)i * H + h) * max_sel;

  const bool all = Ktot >= P;
  const int nS = min(n_sink, P), nL = min(n_local, P);
  const int nF = all ? P : nS + nL - max(0, nS - (P - nL));
  const int Kfree = all ? 0 : max(0, Ktot - nF);

  // Threshold prefix: a candidate is chosen when (key & pmask) > prefix, or when it equals
  // the prefix and its rank among equals (by page index) is below `remaining`.
  uint32_t prefix = 0, pmask = 0;
  int remaining = Kfree;
  if (Kfree > 0) {
    for (int pass = 0; pass < 4; pass++) {
      const int shift = 24 - 8 * pass;
      for (int x = threadIdx.x; x < 256; x += kThreads) hist[x] = 0;
      __syncthreads();
      for (int j = threadIdx.x; j < P; j += kThreads) {
        if (is_forced(j, P, nS, nL)) continue;
        const uint32_t key = float_key(s[j]);
        if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255], 1);
      }
      __syncthreads();
      if (threadIdx.x < kWave) {
        // lane l holds bins 255-4l .. 252-4l (descending); find the bin holding the
        // remaining-th largest key
        const int l = threadIdx.x;
        int c[4], tot = 0;
#pragma unroll
        for (int e = 0; e < 4; e++) {
          c[e] = hist[255 - 4 * l - e];
          tot += c[e];
        }
        int incl = tot;
#pragma unroll
        for (int off = 1; off < kWave; off <<= 1) {
          const int y = __shfl_up(incl, off, kWave);
          if (l >= off) incl += y;
        }
        int above = incl - tot;
#pragma unroll
        for (int e = 0; e < 4; e++) {
          if (above < remaining && above + c[e] >= remaining) {
            pick[0] = 255 - 4 * l - e;
            pick[1] = above;
            pick[2] = c[e];
          }
          above += c[e];
        }
      }
      __syncthreads();
      const int digit = pick[0];
      remaining -= pick[1];
      prefix |= (uint32_t)digit << shift;
      pmask |= 255u << shift;
      const bool done = pick[2] == remaining;   // every key with this prefix is chosen
      __syncthreads();
      if (done) break;
    }
  }

  int eq_base = 0, sel_base = 0;
  for (int j0 = 0; j0 < P; j0 += kThreads) {
    const int j = j0 + threadIdx.x;
    bool forced = false, gt = false, eq = false;
    if (j < P) {
      if (all) {
        forced = true;
      } else if (is_forced(j, P, nS, nL)) {
        forced = true;
      } else if (Kfree > 0) {
        const uint32_t mk = float_key(s[j]) & pmask;
        gt = mk > prefix;
        eq = mk == prefix;
      }
    }
    int eq_rank;
    const int eq_tot = block_excl_count(eq, &eq_rank, wave_tot);
    const bool chosen = forced || gt || (eq && eq_base + eq_rank < remaining);
    int pos;
    const int sel_tot = block_excl_count(chosen, &pos, wave_tot);
    if (chosen && sel_base + pos < max_sel) out[sel_base + pos] = j;
    eq_base += eq_tot;
    sel_base += sel_tot;
  }
  for (int m = sel_base + threadIdx.x; m < max_sel; m += kThreads) out[m] = -1;
  if (h == 0 && threadIdx.x == 0) sel_count[i] = min(sel_base, max_sel);
}

template <int KIND, int D>
void launch_dot(const Geometry& g, const uint16_t* q, int Hq, const float* mean, const uint16_t* maxs,
                float* scores, int ppb, int gx, hipStream_t stream) {
  hipLaunchKernelGGL((score_dot_kernel<KIND, D>), dim3(gx, g.batch), dim3(kThreads), 0, stream, q, Hq, g.H,
                     g.ps, g.num_phys_pages, g.max_pages, g.batch, g.indptr, g.indices, g.seq_lens, mean, maxs,
                     scores, ppb);
}

}  // namespace

size_t score_workspace_bytes(int batch, int num_kv_heads, int max_pages) {
  size_t b = (size_t)batch * num_kv_heads * (size_t)max_pages * sizeof(float);
  return (b + 255) & ~(size_t)255;
}

hipError_t launch_score_topk(const Geometry& g, const uint16_t* q, int Hq, int kind, const float* mean,
                             const uint16_t* maxs, const uint16_t* mins, const int32_t* budget, int n_sink,
                             int n_local, int max_sel, int32_t* sel_pages, int32_t* sel_count, void* ws,
                             hipStream_t stream) {
  if (g.batch == 0) return hipSuccess;
  float* scores = reinterpret_cast<float*>(ws);
  const int ppb = 64;
  int gx = (g.max_pages + ppb - 1) / ppb;
  if (gx < 1) gx = 1;
  if (kind == kQuest) {
    const size_t lds = (size_t)Hq * g.Dqk * sizeof(float);
    if (g.Dqk == 64)
      hipLaunchKernelGGL(score_quest_kernel<64>, dim3(gx, g.batch), dim3(kThreads), lds, stream, q, Hq, g.H, g.ps,
                         g.num_phys_pages, g.max_pages, g.batch, g.indptr, g.indices, g.seq_lens, maxs, mins,
                         scores, ppb);
    else
      hipLaunchKernelGGL(score_quest_kernel<128>, dim3(gx, g.batch), dim3(kThreads), lds, stream, q, Hq, g.H,
                         g.ps, g.num_phys_pages, g.max_pages, g.batch, g.indptr, g.indices, g.seq_lens, maxs,
                         mins, scores, ppb);
  } else if (kind == kMeanDot) {
    if (g.Dqk == 64) launch_dot<kMeanDot, 64>(g, q, Hq, mean, maxs, scores, ppb, gx, stream);
    else if (g.Dqk == 128) launch_dot<kMeanDot, 128>(g, q, Hq, mean, maxs, scores, ppb, gx, stream);
    else launch_dot<kMeanDot, 576>(g, q, Hq, mean, maxs, scores, ppb, gx, stream);
  } else {
    if (g.Dqk == 64) launch_dot<kMaxDot, 64>(g, q, Hq, mean, maxs, scores, ppb, gx, stream);
    else if (g.Dqk == 128) launch_dot<kMaxDot, 128>(g, q, Hq, mean, maxs, scores, ppb, gx, stream);
    else launch_dot<kMaxDot, 576>(g, q, Hq, mean, maxs, scores, ppb, gx, stream);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(topk_kernel, dim3(g.batch * g.H), dim3(kThreads), 0, stream, scores, g.H, g.ps,
                     g.max_pages, g.batch, g.indptr, g.seq_lens, budget, n_sink, n_local, max_sel, sel_pages,
                     sel_count);
  return hipGetLastError();
}

}  // namespace vx

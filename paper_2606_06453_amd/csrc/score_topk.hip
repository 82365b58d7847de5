// Indexer stage: page scores (Sec. 3.1 Eq. 2; Sec. 3.2 Quest) and the selection of sink,
// local and top-scoring pages (Sec. 3.1 Eq. 3; Sec. 6.4 setup).
//
// score_kernel   HBM-bound stream over the summaries.  A row of 16 lanes owns one
//                (page, KV head) item.  Each lane holds D/16 channels of the summary and
//                of the query view.  Products accumulate in fp64 and reduce across the row
//                with DPP, then round once to fp32.  Output goes to a padded scratch table
//                scores[h][i][j].
// topk_kernel    One workgroup per (request, KV head).  It runs an exact radix select over
//                an order-preserving uint32 key of the fp32 score: up to 4 passes of 8-bit
//                digits, an LDS histogram with one bin per thread, a block scan over the
//                bins, and keys cached in LDS.  That finds the K_free-th best candidate.
//                Ties at the threshold go to the lowest page index.  Each thread owns a
//                contiguous page range: one block scan ranks the tied pages and a second
//                compacts the forced and chosen pages in ascending order.
#include "vx_device.h"
#include "vx_internal.h"

namespace vx {
namespace {

constexpr int kThreads = 256;
constexpr int kRows = kThreads / 16;     // 16-lane rows per workgroup

enum { kMeanDot = 0, kQuest = 1, kMaxDot = 2 };

// Channel mapping of a 16-lane row: lane u owns the chunks u, u+16, u+32, ... of a summary
// row, so every load instruction of a row reads 16 contiguous chunks.  The query
// view uses the same mapping (a dot product does not care about channel order).
template <int D, bool BF16>
struct RowMap {
  // 16-byte chunks, or 8-byte ones when a bf16 row is only 128 bytes (D = 64)
  static constexpr int kElemsPerChunk = BF16 ? (D / 16 < 8 ? D / 16 : 8) : 4;
  static constexpr int kChunks = D / kElemsPerChunk / 16;     // 16-byte chunks per lane
  static constexpr int E = kChunks * kElemsPerChunk;          // channels per lane
  __device__ static int channel(int u, int c, int e) { return (u + 16 * c) * kElemsPerChunk + e; }
};

template <int D>
__device__ __forceinline__ void load_row_f32(const float* p, int u, float (&x)[D / 16]) {
  using M = RowMap<D, false>;
#pragma unroll
  for (int c = 0; c < M::kChunks; c++) {
    const float4 w = *reinterpret_cast<const float4*>(p + M::channel(u, c, 0));
    x[4 * c] = w.x;
    x[4 * c + 1] = w.y;
    x[4 * c + 2] = w.z;
    x[4 * c + 3] = w.w;
  }
}

template <int D>
__device__ __forceinline__ void load_row_bf16(const uint16_t* p, int u, float (&x)[D / 16]) {
  using M = RowMap<D, true>;
  constexpr int W = M::kElemsPerChunk / 2;      // dwords per chunk
#pragma unroll
  for (int c = 0; c < M::kChunks; c++) {
    uint32_t ws[4];
    if constexpr (W == 4) {
      const uint4 w = *reinterpret_cast<const uint4*>(p + M::channel(u, c, 0));
      ws[0] = w.x; ws[1] = w.y; ws[2] = w.z; ws[3] = w.w;
    } else {
      const uint2 w = *reinterpret_cast<const uint2*>(p + M::channel(u, c, 0));
      ws[0] = w.x; ws[1] = w.y;
    }
#pragma unroll
    for (int e = 0; e < W; e++) {
      x[M::kElemsPerChunk * c + 2 * e] = bf16lo(ws[e]);
      x[M::kElemsPerChunk * c + 2 * e + 1] = bf16hi(ws[e]);
    }
  }
}

constexpr int kPagesPerBlock = 32;

// Items (page, KV head) per row kept in flight: about 256 bytes of loads per lane.
template <int D, int KIND>
constexpr int items_in_flight() {
  constexpr int bytes_per_item = (KIND == kMeanDot ? 4 : (KIND == kQuest ? 4 : 2)) * D / 16;
  constexpr int u = 256 / bytes_per_item;
  return u < 1 ? 1 : (u > 8 ? 8 : u);
}

// Block prologue shared by the score kernels: the pages [jb, jb + nj) of request i get their
// physical ids staged in LDS, so that the summary loads do not wait on dependent id loads.
__device__ __forceinline__ int stage_pages(const int32_t* __restrict__ indptr, const int32_t* __restrict__ indices,
                                           const int32_t* __restrict__ seq_lens, int i, int ps, int max_pages,
                                           int num_phys, int* pid, int* jb_out) {
  const int base = indptr[i];
  const int P = num_pages(seq_lens[i], ps, indptr[i + 1] - base, max_pages);
  const int jb = (int)blockIdx.x * kPagesPerBlock;
  const int nj = min(kPagesPerBlock, P - jb);
  if ((int)threadIdx.x < nj) pid[threadIdx.x] = (int)clamp_page(indices[base + jb + threadIdx.x], num_phys);
  *jb_out = jb;
  return nj;
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
    const uint16_t* __restrict__ maxs, float* __restrict__ scores) {
  constexpr int E = D / 16;
  constexpr bool kBf16 = KIND != kMeanDot;
  using M = RowMap<D, kBf16>;
  constexpr int U = items_in_flight<D, KIND>();
  __shared__ int pid[kPagesPerBlock];
  const int i = blockIdx.y;
  int jb;
  const int nj = stage_pages(indptr, indices, seq_lens, i, ps, max_pages, num_phys, pid, &jb);
  if (nj <= 0) return;                                  // uniform over the block
  const int row = threadIdx.x >> 4, u = threadIdx.x & 15;
  const int h = row % H, slot = row / H, slots = kRows / H;
  const int g = Hq / H;

  // group-mean query view in this row's channel mapping: vector loads of the group's bf16
  // query heads, fp64 sums (exact), one division
  double qb[E];
  {
    const uint16_t* qi = q + ((int64_t)i * Hq + (int64_t)h * g) * D;
#pragma unroll
    for (int e = 0; e < E; e++) qb[e] = 0.0;
    for (int r = 0; r < g; r++) {
#pragma unroll
      for (int c = 0; c < M::kChunks; c++) {
        const uint16_t* src = qi + (int64_t)r * D + M::channel(u, c, 0);
        uint32_t wq[4];
        if constexpr (M::kElemsPerChunk == 8) {
          const uint4 v = *reinterpret_cast<const uint4*>(src);
          wq[0] = v.x; wq[1] = v.y; wq[2] = v.z; wq[3] = v.w;
        } else {
          const uint2 v = *reinterpret_cast<const uint2*>(src);
          wq[0] = v.x; wq[1] = v.y;
        }
#pragma unroll
        for (int e = 0; e < M::kElemsPerChunk / 2; e++) {
          qb[c * M::kElemsPerChunk + 2 * e] += (double)bf16lo(wq[e]);
          qb[c * M::kElemsPerChunk + 2 * e + 1] += (double)bf16hi(wq[e]);
        }
      }
    }
    const double inv_g = 1.0 / (double)g;   // g is a power of two in practice; exact then
#pragma unroll
    for (int e = 0; e < E; e++) qb[e] = (g & (g - 1)) == 0 ? qb[e] * inv_g : qb[e] / (double)g;
  }
  __syncthreads();

  float* out = scores + ((int64_t)h * batch + i) * max_pages + jb;
  for (int j0 = slot; j0 < nj; j0 += U * slots) {
    float x[U][E];
#pragma unroll
    for (int v = 0; v < U; v++) {
      const int jj = j0 + v * slots;
      if (jj < nj) {
        const int64_t o = ((int64_t)pid[jj] * H + h) * D;
        if (KIND == kMeanDot) load_row_f32<D>(mean + o, u, x[v]);
        else load_row_bf16<D>(maxs + o, u, x[v]);
      }
    }
#pragma unroll
    for (int v = 0; v < U; v++) {
      const int jj = j0 + v * slots;
      if (jj < nj) {
        double acc = 0.0;
#pragma unroll
        for (int e = 0; e < E; e++) acc = fma(qb[e], (double)x[v][e], acc);
        acc = row16_sum_f64(acc);
        if (u == 0) out[jj] = (float)acc;
      }
    }
  }
}

// ------------------------------------------------------------------------------------
// Quest: s_j = max_r sum_c max(q_rc Max_jc, q_rc Min_jc).  Each product of two bf16 values
// is exact in fp32; the per-head sums run in fp64.  The group's query heads sit in LDS as
// fp32 [Hq][D], in the row channel mapping.
// ------------------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kThreads) void score_quest_kernel(
    const uint16_t* __restrict__ q, int Hq, int H, int ps, int num_phys, int max_pages, int batch,
    const int32_t* __restrict__ indptr, const int32_t* __restrict__ indices,
    const int32_t* __restrict__ seq_lens, const uint16_t* __restrict__ maxs,
    const uint16_t* __restrict__ mins, float* __restrict__ scores) {
  constexpr int E = D / 16;
  using M = RowMap<D, true>;
  constexpr int U = items_in_flight<D, kQuest>();
  extern __shared__ float qs[];        // [Hq][16 lanes][E]
  __shared__ int pid[kPagesPerBlock];
  const int i = blockIdx.y;
  int jb;
  const int nj = stage_pages(indptr, indices, seq_lens, i, ps, max_pages, num_phys, pid, &jb);
  if (nj <= 0) return;
  const int row = threadIdx.x >> 4, u = threadIdx.x & 15;
  const int h = row % H, slot = row / H, slots = kRows / H;
  const int g = Hq / H;

  for (int x = threadIdx.x; x < Hq * D; x += kThreads) {       // coalesced over channels
    const int r = x / D, c = x - r * D;
    const int chunk = c / M::kElemsPerChunk, e_in = c - chunk * M::kElemsPerChunk;
    const int uu = chunk % 16, cc = chunk / 16;                // inverse of RowMap::channel
    qs[(r * 16 + uu) * E + cc * M::kElemsPerChunk + e_in] = bf16_to_f32(q[(int64_t)i * Hq * D + x]);
  }
  __syncthreads();

  float* out = scores + ((int64_t)h * batch + i) * max_pages + jb;
  for (int j0 = slot; j0 < nj; j0 += U * slots) {
    float mx[U][E], mn[U][E];
#pragma unroll
    for (int v = 0; v < U; v++) {
      const int jj = j0 + v * slots;
      if (jj < nj) {
        const int64_t o = ((int64_t)pid[jj] * H + h) * D;
        load_row_bf16<D>(maxs + o, u, mx[v]);
        load_row_bf16<D>(mins + o, u, mn[v]);
      }
    }
#pragma unroll
    for (int v = 0; v < U; v++) {
      const int jj = j0 + v * slots;
      if (jj < nj) {
        double best = -INFINITY;
        for (int r = 0; r < g; r++) {
          const float* qr = qs + ((h * g + r) * 16 + u) * E;
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
        if (u == 0) out[jj] = (float)best;
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

constexpr int kMaxLdsKeys = 8192;      // candidates kept in LDS; longer requests re-read scores

// Inclusive scan of one int per thread over the kThreads threads of the block, in thread order.
__device__ __forceinline__ int block_incl_scan(int x, int* wave_tot, int* total) {
  const int lane = lane_id(), w = threadIdx.x >> 6;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int y = __shfl_up(x, off, kWave);
    if (lane >= off) x += y;
  }
  if (lane == kWave - 1) wave_tot[w] = x;
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int k = 0; k < kThreads / kWave; k++) {
    const int t = wave_tot[k];
    before += (k < w) ? t : 0;
    tot += t;
  }
  __syncthreads();
  *total = tot;
  return x + before;
}

__global__ __launch_bounds__(kThreads) void topk_kernel(
    const float* __restrict__ scores, int H, int ps, int max_pages, int batch,
    const int32_t* __restrict__ indptr, const int32_t* __restrict__ seq_lens,
    const int32_t* __restrict__ budget, int n_sink, int n_local, int max_sel,
    int32_t* __restrict__ sel_pages, int32_t* __restrict__ sel_count) {
  static_assert(kThreads == 256, "one histogram bin per thread");
  __shared__ uint32_t keys[kMaxLdsKeys];
  __shared__ int hist[256];
  __shared__ int wave_tot[kThreads / kWave];
  __shared__ int pick[3];              // digit, count above the digit's bin, bin count

  const int tid = threadIdx.x;
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
  const bool in_lds = P <= kMaxLdsKeys;
  auto key_at = [&](int j) -> uint32_t { return in_lds ? keys[j] : float_key(s[j]); };

  if (Kfree > 0 && in_lds) {
    for (int j = tid; j < P; j += kThreads) keys[j] = float_key(s[j]);
  }

  // Radix select, 8-bit digits from the most significant.  Threshold prefix: a candidate
  // is chosen when (key & pmask) > prefix, or when it equals the prefix and its rank among
  // equals (by page index) is below `remaining`.
  uint32_t prefix = 0, pmask = 0;
  int remaining = Kfree;
  if (Kfree > 0) {
    for (int pass = 0; pass < 4; pass++) {
      const int shift = 24 - 8 * pass;
      hist[tid] = 0;
      __syncthreads();
      for (int j = tid; j < P; j += kThreads) {
        if (is_forced(j, P, nS, nL)) continue;
        const uint32_t key = key_at(j);
        if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255], 1);
      }
      __syncthreads();
      // thread t owns bin 255 - t: the scan runs over bins in descending order
      const int c = hist[255 - tid];
      int tot;
      const int incl = block_incl_scan(c, wave_tot, &tot);
      const int above = incl - c;
      if (above < remaining && incl >= remaining) {
        pick[0] = 255 - tid;
        pick[1] = above;
        pick[2] = c;
      }
      __syncthreads();
      const int digit = pick[0];
      remaining -= pick[1];
      prefix |= (uint32_t)digit << shift;
      pmask |= 255u << shift;
      const bool done = pick[2] == remaining;   // every key with this prefix is chosen
      if (done) break;
    }
  }

  // Compaction: thread t owns the contiguous pages [t*R, (t+1)*R), so one scan gives each
  // tied candidate its rank by page index and a second gives each chosen page its slot.
  const int R = (P + kThreads - 1) / kThreads;
  const int j_lo = min(P, tid * R), j_hi = min(P, j_lo + R);
  int n_eq = 0;
  if (Kfree > 0) {
    for (int j = j_lo; j < j_hi; j++) {
      if (!is_forced(j, P, nS, nL) && (key_at(j) & pmask) == prefix) n_eq++;
    }
  }
  int tot_eq;
  int eq_rank = block_incl_scan(n_eq, wave_tot, &tot_eq) - n_eq;
  int n_chosen = 0;
  for (int j = j_lo, r = eq_rank; j < j_hi; j++) {
    bool chosen = all || is_forced(j, P, nS, nL);
    if (!chosen && Kfree > 0) {
      const uint32_t mk = key_at(j) & pmask;
      chosen = mk > prefix || (mk == prefix && r++ < remaining);
    }
    n_chosen += chosen;
  }
  int tot_sel;
  int pos = block_incl_scan(n_chosen, wave_tot, &tot_sel) - n_chosen;
  for (int j = j_lo, r = eq_rank; j < j_hi; j++) {
    bool chosen = all || is_forced(j, P, nS, nL);
    if (!chosen && Kfree > 0) {
      const uint32_t mk = key_at(j) & pmask;
      chosen = mk > prefix || (mk == prefix && r++ < remaining);
    }
    if (chosen) {
      if (pos < max_sel) out[pos] = j;
      pos++;
    }
  }
  for (int m = tot_sel + tid; m < max_sel; m += kThreads) out[m] = -1;
  if (h == 0 && tid == 0) sel_count[i] = min(tot_sel, max_sel);
}

template <int KIND, int D>
void launch_dot(const Geometry& g, const uint16_t* q, int Hq, const float* mean, const uint16_t* maxs,
                float* scores, int gx, hipStream_t stream) {
  hipLaunchKernelGGL((score_dot_kernel<KIND, D>), dim3(gx, g.batch), dim3(kThreads), 0, stream, q, Hq, g.H,
                     g.ps, g.num_phys_pages, g.max_pages, g.batch, g.indptr, g.indices, g.seq_lens, mean, maxs,
                     scores);
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
  int gx = (g.max_pages + kPagesPerBlock - 1) / kPagesPerBlock;
  if (gx < 1) gx = 1;
  if (kind == kQuest) {
    const size_t lds = (size_t)Hq * g.Dqk * sizeof(float);
    if (g.Dqk == 64)
      hipLaunchKernelGGL(score_quest_kernel<64>, dim3(gx, g.batch), dim3(kThreads), lds, stream, q, Hq, g.H, g.ps,
                         g.num_phys_pages, g.max_pages, g.batch, g.indptr, g.indices, g.seq_lens, maxs, mins,
                         scores);
    else
      hipLaunchKernelGGL(score_quest_kernel<128>, dim3(gx, g.batch), dim3(kThreads), lds, stream, q, Hq, g.H,
                         g.ps, g.num_phys_pages, g.max_pages, g.batch, g.indptr, g.indices, g.seq_lens, maxs,
                         mins, scores);
  } else if (kind == kMeanDot) {
    if (g.Dqk == 64) launch_dot<kMeanDot, 64>(g, q, Hq, mean, maxs, scores, gx, stream);
    else if (g.Dqk == 128) launch_dot<kMeanDot, 128>(g, q, Hq, mean, maxs, scores, gx, stream);
    else launch_dot<kMeanDot, 576>(g, q, Hq, mean, maxs, scores, gx, stream);
  } else {
    if (g.Dqk == 64) launch_dot<kMaxDot, 64>(g, q, Hq, mean, maxs, scores, gx, stream);
    else launch_dot<kMaxDot, 128>(g, q, Hq, mean, maxs, scores, gx, stream);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(topk_kernel, dim3(g.batch * g.H), dim3(kThreads), 0, stream, scores, g.H, g.ps,
                     g.max_pages, g.batch, g.indptr, g.seq_lens, budget, n_sink, n_local, max_sel, sel_pages,
                     sel_count);
  return hipGetLastError();
}

}  // namespace vx

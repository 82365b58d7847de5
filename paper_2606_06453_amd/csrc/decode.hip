// Sparse paged attention over the selected pages (Sec. 3.1 Eq. 4; Sec. 5.3), as three
// kernels on one stream:
//
// plan_kernel    Device-side workload plan (Sec. 5.1, sequence-local template).  From the
//                per-request selection counts it picks a page chunk so that about
//                `target_units` units cover the batch.  It writes one unit
//                (pair = (request, KV head), page range) per chunk, plus each pair's first
//                unit and unit count, and writes the zero output of pairs with no selected
//                page.  No host sync is needed.
// decode kernel  Each wave is one "program" and walks a balanced contiguous range of units
//                (per = n / programs, the first n % programs take one more).  A unit is
//                16-token tiles of its pages:
//                  S^T = K Q^T    MFMA 16x16x32 bf16: 16 tokens x 16 (padded) query heads,
//                                 contraction over D
//                  online softmax in the log2 domain, one running max per query head
//                  O^T += V^T P^T MFMA 16x16x16 bf16: V^T comes from a register
//                                 transpose of 4 token rows per lane.  P is split into
//                                 bf16 hi + lo parts, so the probabilities keep about 16
//                                 bits.
//                K and V tiles are double-buffered in registers: tile t+1 loads while tile
//                t computes.  A pair covered by a single unit writes bf16 output directly.
//                Otherwise the unit writes a normalised fp32 partial and its log2-sum-exp.
// merge_kernel   LSE-weighted combination of the partials of pairs split over several
//                units.  A separate launch: on MI355X each XCD has its own L2, so a
//                device-scope release/acquire inside the split kernel would write back and
//                invalidate L2 per unit, which costs far more than one extra launch.
#include <climits>

#include "vx_device.h"
#include "vx_internal.h"

namespace vx {
namespace {

constexpr int kDecodeThreads = 256;       // 4 independent programs (waves) per workgroup
constexpr int kPlanThreads = 1024;
constexpr int kMergeThreads = 256;

struct DecodeArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* indptr;
  const int32_t* indices;
  const int32_t* seq_lens;
  const int32_t* sel_pages;
  uint16_t* out;
  const PlanHeader* plan;
  const int4* units;
  float* part_o;
  float* part_lse;
  int max_sel, H, g, Hq, ps, num_phys;
  float scale_log2;   // sm_scale * log2(e)
};

// ------------------------------------------------------------------------------------
// plan
// ------------------------------------------------------------------------------------
// Inclusive block scan of one int per thread (kPlanThreads threads).
__device__ int block_incl_scan(int x, int* wave_sums, int* total) {
  const int lane = lane_id(), w = threadIdx.x >> 6;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int y = __shfl_up(x, off, kWave);
    if (lane >= off) x += y;
  }
  if (lane == kWave - 1) wave_sums[w] = x;
  __syncthreads();
  int before = 0, tot = 0;
  for (int k = 0; k < kPlanThreads / kWave; k++) {
    const int s = wave_sums[k];
    before += (k < w) ? s : 0;
    tot += s;
  }
  __syncthreads();
  *total = tot;
  return x + before;
}

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(const int32_t* __restrict__ sel_count, int batch,
                                                            int H, int max_sel, int target_units,
                                                            PlanHeader* __restrict__ hdr,
                                                            int4* __restrict__ units,
                                                            int2* __restrict__ pairs,
                                                            uint16_t* __restrict__ out, int out_per_pair) {
  __shared__ long long red[kPlanThreads / kWave];
  __shared__ int wave_sums[kPlanThreads / kWave];
  long long local = 0;
  for (int i = threadIdx.x; i < batch; i += kPlanThreads) local += min(max(sel_count[i], 0), max_sel);
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) local += __shfl_xor(local, off, kWave);
  if (lane_id() == 0) red[threadIdx.x >> 6] = local;
  __syncthreads();
  long long total = 0;
  for (int k = 0; k < kPlanThreads / kWave; k++) total += red[k];
  total *= H;
  const int chunk = (int)max(1LL, (total + target_units - 1) / target_units);

  int running = 0;
  for (int b0 = 0; b0 < batch; b0 += kPlanThreads) {
    const int i = b0 + threadIdx.x;
    const int cnt = (i < batch) ? min(max(sel_count[i], 0), max_sel) : 0;
    const int Ui = (cnt + chunk - 1) / chunk;
    int tot;
    const int incl = block_incl_scan(H * Ui, wave_sums, &tot);
    const int off = running + incl - H * Ui;
    if (i < batch) {
      for (int h = 0; h < H; h++) {
        pairs[i * H + h] = make_int2(off + h * Ui, Ui);
        if (Ui == 0) {
          uint16_t* o = out + (int64_t)(i * H + h) * out_per_pair;
          for (int x = 0; x < out_per_pair; x++) o[x] = 0;
        }
        for (int s = 0; s < Ui; s++) {
          units[off + h * Ui + s] = make_int4(i * H + h, s * chunk, min(cnt, (s + 1) * chunk), Ui);
        }
      }
    }
    running += tot;
  }
  if (threadIdx.x == 0) {
    hdr->n_units = running;
    hdr->chunk = chunk;
  }
}

// ------------------------------------------------------------------------------------
// split kernel, GQA (D = head_dim_qk = head_dim_v)
// ------------------------------------------------------------------------------------
template <int D>
struct Tile {
  bf16x8_t k[D / 32];                  // A operand of S^T = K Q^T: row = lane & 15
  uint32_t v[4][D / 32];               // rows 4*grp + r, channels (lane & 15) * D/16 ..
};

template <int D>
__device__ __forceinline__ void load_tile(const uint16_t* __restrict__ kt, const uint16_t* __restrict__ vt,
                                          int col, int grp, Tile<D>& t) {
  constexpr int KS = D / 32, DPL = D / 16;
#pragma unroll
  for (int kk = 0; kk < KS; kk++)
    t.k[kk] = *reinterpret_cast<const bf16x8_t*>(kt + col * D + 32 * kk + 8 * grp);
#pragma unroll
  for (int r = 0; r < 4; r++) {
    const uint16_t* src = vt + (4 * grp + r) * D + col * DPL;
    if constexpr (DPL == 8) {
      const uint4 w = *reinterpret_cast<const uint4*>(src);
      t.v[r][0] = w.x;
      t.v[r][1] = w.y;
      t.v[r][2] = w.z;
      t.v[r][3] = w.w;
    } else {
      const uint2 w = *reinterpret_cast<const uint2*>(src);
      t.v[r][0] = w.x;
      t.v[r][1] = w.y;
    }
  }
}

template <int D>
__device__ __forceinline__ void compute_tile(Tile<D>& t, const bf16x8_t (&qv)[D / 32], int valid, int grp,
                                             float scale_log2, float& m, float& lsum, f32x4_t (&acc)[D / 16]) {
  constexpr int KS = D / 32, DPL = D / 16;
  f32x4_t st = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kk = 0; kk < KS; kk++) st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(t.k[kk], qv[kk], st, 0, 0, 0);

  // lane (grp, col) holds S^T[token 4*grp + i][query head col]
  float sv[4];
#pragma unroll
  for (int i = 0; i < 4; i++) sv[i] = (4 * grp + i < valid) ? st[i] * scale_log2 : -INFINITY;
  float mt = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
  mt = fmaxf(mt, xor_shfl(mt, 16));
  mt = fmaxf(mt, xor_shfl(mt, 32));
  const float m_new = fmaxf(m, mt);                  // finite: the tile has a valid token
  const float alpha = exp2f(m - m_new);
  float p[4];
#pragma unroll
  for (int i = 0; i < 4; i++) p[i] = exp2f(sv[i] - m_new);
  lsum = lsum * alpha + ((p[0] + p[1]) + (p[2] + p[3]));
  m = m_new;
#pragma unroll
  for (int j = 0; j < DPL; j++) {
    acc[j][0] *= alpha;
    acc[j][1] *= alpha;
    acc[j][2] *= alpha;
    acc[j][3] *= alpha;
  }
  // P^T operand (k = token 4*grp + i, n = head col), split into bf16 hi + lo
  s16x4_t ph, pl;
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const uint32_t hb = f32_to_bf16_rne(p[i]);
    const uint32_t lb = f32_to_bf16_rne(p[i] - __uint_as_float(hb << 16));
    ph[i] = (short)hb;
    pl[i] = (short)lb;
  }
  // rows beyond the valid tokens must not inject NaN/Inf through 0 * junk
#pragma unroll
  for (int r = 0; r < 4; r++) {
    if (4 * grp + r >= valid) {
#pragma unroll
      for (int w = 0; w < DPL / 2; w++) t.v[r][w] = 0u;
    }
  }
#pragma unroll
  for (int j = 0; j < DPL; j++) {
    // V^T operand for output channels c*DPL + j: token rows 4*grp + 0..3 of channel j
    const int w = j >> 1;
    s16x4_t a;
    if ((j & 1) == 0) {
      a[0] = (short)(t.v[0][w] & 0xffffu);
      a[1] = (short)(t.v[1][w] & 0xffffu);
      a[2] = (short)(t.v[2][w] & 0xffffu);
      a[3] = (short)(t.v[3][w] & 0xffffu);
    } else {
      a[0] = (short)(t.v[0][w] >> 16);
      a[1] = (short)(t.v[1][w] >> 16);
      a[2] = (short)(t.v[2][w] >> 16);
      a[3] = (short)(t.v[3][w] >> 16);
    }
    acc[j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, ph, acc[j], 0, 0, 0);
    acc[j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, pl, acc[j], 0, 0, 0);
  }
}

template <int D>
__global__ __launch_bounds__(kDecodeThreads) void decode_gqa_kernel(const DecodeArgs a) {
  constexpr int KS = D / 32, DPL = D / 16;
  const int lane = lane_id();
  const int col = lane & 15, grp = lane >> 4;
  const int prog = (int)blockIdx.x * (kDecodeThreads / kWave) + (int)(threadIdx.x >> 6);
  const int nprog = (int)gridDim.x * (kDecodeThreads / kWave);
  const int n_units = a.plan->n_units;
  const int per = n_units / nprog, rem = n_units % nprog;
  const int w_begin = prog * per + min(prog, rem);
  const int w_end = w_begin + per + (prog < rem ? 1 : 0);

  for (int w = w_begin; w < w_end; w++) {
    const int4 un = a.units[w];
    const int pair = un.x, i = pair / a.H, h = pair - (pair / a.H) * a.H;
    const int L = a.seq_lens[i];
    const int base = a.indptr[i];
    const int P = num_pages(L, a.ps, a.indptr[i + 1] - base, INT_MAX);
    const int32_t* sel = a.sel_pages + (int64_t)pair * a.max_sel;

    bf16x8_t qv[KS];
    const bool hv = col < a.g;
    {
      const uint16_t* qp = a.q + ((int64_t)i * a.Hq + h * a.g + (hv ? col : 0)) * D + 8 * grp;
#pragma unroll
      for (int kk = 0; kk < KS; kk++) {
        qv[kk] = *reinterpret_cast<const bf16x8_t*>(qp + 32 * kk);
        if (!hv) qv[kk] = bf16x8_t{};
      }
    }
    f32x4_t acc[DPL];
#pragma unroll
    for (int j = 0; j < DPL; j++) acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float m = -INFINITY, lsum = 0.f;

    const int64_t head_off = (int64_t)h * a.ps * D;
    const int64_t page_stride = (int64_t)a.H * a.ps * D;

    for (int sb = un.y; sb < un.z; sb += kWave) {
      // page metadata of up to 64 selected pages, one per lane
      int my_p = 0, my_n = 0;
      if (sb + lane < un.z) {
        const int j = sel[sb + lane];
        if (j >= 0 && j < P) {
          my_p = (int)clamp_page(a.indices[base + j], a.num_phys);
          my_n = min(a.ps, L - j * a.ps);
        }
      }
      const int nb = min(kWave, un.z - sb);
      // Tile cursor over (page slot s, tile tt) of pages with n > 0.  Two statically named
      // register tiles alternate: the next tile loads while the current one computes.
      int s = 0, tt = 0;
      while (s < nb && __builtin_amdgcn_readlane(my_n, s) <= 0) s++;
      if (s >= nb) continue;
      int cur_n = __builtin_amdgcn_readlane(my_n, s);
      int cur_p = __builtin_amdgcn_readlane(my_p, s);
      int nxt_n = 0, nxt_p = 0, ns = 0, ntt = 0;
      auto advance = [&]() -> bool {
        ns = s;
        ntt = tt + 1;
        nxt_n = cur_n;
        nxt_p = cur_p;
        if (ntt * 16 >= cur_n) {
          ntt = 0;
          ns = s + 1;
          while (ns < nb && __builtin_amdgcn_readlane(my_n, ns) <= 0) ns++;
          if (ns >= nb) return false;
          nxt_n = __builtin_amdgcn_readlane(my_n, ns);
          nxt_p = __builtin_amdgcn_readlane(my_p, ns);
        }
        return true;
      };
      auto tile_ptr_k = [&](int p, int t16) { return a.k + p * page_stride + head_off + (int64_t)t16 * 16 * D; };
      auto tile_ptr_v = [&](int p, int t16) { return a.v + p * page_stride + head_off + (int64_t)t16 * 16 * D; };
      Tile<D> ta, tb;
      load_tile<D>(tile_ptr_k(cur_p, 0), tile_ptr_v(cur_p, 0), col, grp, ta);
      while (true) {
        bool more = advance();
        if (more) load_tile<D>(tile_ptr_k(nxt_p, ntt), tile_ptr_v(nxt_p, ntt), col, grp, tb);
        compute_tile<D>(ta, qv, min(16, cur_n - 16 * tt), grp, a.scale_log2, m, lsum, acc);
        if (!more) break;
        s = ns; tt = ntt; cur_n = nxt_n; cur_p = nxt_p;
        more = advance();
        if (more) load_tile<D>(tile_ptr_k(nxt_p, ntt), tile_ptr_v(nxt_p, ntt), col, grp, ta);
        compute_tile<D>(tb, qv, min(16, cur_n - 16 * tt), grp, a.scale_log2, m, lsum, acc);
        if (!more) break;
        s = ns; tt = ntt; cur_n = nxt_n; cur_p = nxt_p;
      }
    }

    float lt = lsum + xor_shfl(lsum, 16);
    lt += xor_shfl(lt, 32);
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
    if (un.w == 1) {
      if (hv) {
        // channels (4*grp + i)*DPL + j: 4*DPL contiguous values starting at 4*grp*DPL
        uint16_t* dst = a.out + ((int64_t)i * a.Hq + h * a.g + col) * D + 4 * grp * DPL;
#pragma unroll
        for (int i4 = 0; i4 < 4; i4++) {
          uint32_t wv[DPL / 2];
#pragma unroll
          for (int j = 0; j < DPL; j += 2)
            wv[j / 2] = f32_to_bf16_rne(acc[j][i4] * inv) | (f32_to_bf16_rne(acc[j + 1][i4] * inv) << 16);
          if constexpr (DPL == 8) {
            *reinterpret_cast<uint4*>(dst + i4 * DPL) = make_uint4(wv[0], wv[1], wv[2], wv[3]);
          } else {
            *reinterpret_cast<uint2*>(dst + i4 * DPL) = make_uint2(wv[0], wv[1]);
          }
        }
      }
    } else if (hv) {
      float* dst = a.part_o + ((int64_t)w * a.g + col) * D + 4 * grp * DPL;
#pragma unroll
      for (int i4 = 0; i4 < 4; i4++) {
#pragma unroll
        for (int j = 0; j < DPL; j += 4)
          *reinterpret_cast<float4*>(dst + i4 * DPL + j) =
              make_float4(acc[j][i4] * inv, acc[j + 1][i4] * inv, acc[j + 2][i4] * inv, acc[j + 3][i4] * inv);
      }
      if (grp == 0) a.part_lse[(int64_t)w * a.g + col] = lt > 0.f ? m + __log2f(lt) : -INFINITY;
    }
  }
}

// ------------------------------------------------------------------------------------
// merge: one workgroup per pair split over several units; 4 output channels per thread
// ------------------------------------------------------------------------------------
__global__ __launch_bounds__(kMergeThreads) void merge_kernel(const int2* __restrict__ pairs, int H, int g,
                                                              int Hq, int Dv,
                                                              const float* __restrict__ part_o,
                                                              const float* __restrict__ part_lse,
                                                              uint16_t* __restrict__ out) {
  const int pair = blockIdx.x;
  const int2 pu = pairs[pair];                   // first unit, unit count
  const int first = pu.x, Ui = pu.y;
  if (Ui <= 1) return;                           // written by the split kernel or the plan
  const int i = pair / H, h = pair - i * H;
  uint16_t* dst = out + ((int64_t)i * Hq + (int64_t)h * g) * Dv;
  const int n4 = g * Dv / 4;
  for (int x = threadIdx.x; x < n4; x += kMergeThreads) {
    const int c = (4 * x) / Dv, d = 4 * x - c * Dv;
    float mx = -INFINITY;
    for (int s = 0; s < Ui; s++) mx = fmaxf(mx, part_lse[(int64_t)(first + s) * g + c]);
    float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
    if (mx > -INFINITY) {
      float wsum = 0.f;
      for (int s = 0; s < Ui; s++) {
        const float wgt = exp2f(part_lse[(int64_t)(first + s) * g + c] - mx);
        const float4 p = *reinterpret_cast<const float4*>(part_o + ((int64_t)(first + s) * g + c) * Dv + d);
        wsum += wgt;
        o.x += wgt * p.x;
        o.y += wgt * p.y;
        o.z += wgt * p.z;
        o.w += wgt * p.w;
      }
      const float inv = 1.f / wsum;
      o.x *= inv;
      o.y *= inv;
      o.z *= inv;
      o.w *= inv;
    }
    *reinterpret_cast<uint2*>(dst + c * Dv + d) = make_uint2(f32_to_bf16_rne(o.x) | (f32_to_bf16_rne(o.y) << 16),
                                                             f32_to_bf16_rne(o.z) | (f32_to_bf16_rne(o.w) << 16));
  }
}

}  // namespace

DecodeLayout decode_layout(int batch, int num_kv_heads, int group, int head_dim_v, int max_sel, bool mla) {
  DecodeLayout L;
  L.target_units = mla ? 512 : 2048;
  const long long pairs = (long long)batch * num_kv_heads;
  long long mu = L.target_units + pairs;
  const long long cap = pairs * (long long)(max_sel > 0 ? max_sel : 1);   // chunk >= 1
  if (mu > cap) mu = cap;
  if (mu < 1) mu = 1;
  L.max_units = (int)mu;
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  size_t off = sizeof(PlanHeader);
  L.off_units = off;
  off = al(off + sizeof(int4) * (size_t)L.max_units);
  L.off_pairs = off;     // per pair: first unit, unit count
  off = al(off + sizeof(int2) * (size_t)pairs);
  L.off_lse = off;
  off = al(off + sizeof(float) * (size_t)L.max_units * group);
  L.off_o = off;
  off = al(off + sizeof(float) * (size_t)L.max_units * group * head_dim_v);
  L.total = off;
  return L;
}

hipError_t launch_decode(const Geometry& g, const uint16_t* q, int Hq, const int32_t* sel_pages,
                         const int32_t* sel_count, int max_sel, float sm_scale, uint16_t* out, void* ws,
                         const DecodeLayout& lay, hipStream_t stream) {
  if (g.batch == 0) return hipSuccess;
  char* base = reinterpret_cast<char*>(ws);
  PlanHeader* hdr = reinterpret_cast<PlanHeader*>(base);
  int4* units = reinterpret_cast<int4*>(base + lay.off_units);
  float* part_lse = reinterpret_cast<float*>(base + lay.off_lse);
  float* part_o = reinterpret_cast<float*>(base + lay.off_o);

  int2* pairs = reinterpret_cast<int2*>(base + lay.off_pairs);
  const int group = Hq / g.H;
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kPlanThreads), 0, stream, sel_count, g.batch, g.H, max_sel,
                     lay.target_units, hdr, units, pairs, out, group * g.Dv);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;

  DecodeArgs a;
  a.q = q;
  a.k = g.k;
  a.v = g.v;
  a.indptr = g.indptr;
  a.indices = g.indices;
  a.seq_lens = g.seq_lens;
  a.sel_pages = sel_pages;
  a.out = out;
  a.plan = hdr;
  a.units = units;
  a.part_o = part_o;
  a.part_lse = part_lse;
  a.max_sel = max_sel;
  a.H = g.H;
  a.g = group;
  a.Hq = Hq;
  a.ps = g.ps;
  a.num_phys = g.num_phys_pages;
  a.scale_log2 = sm_scale * 1.4426950408889634f;

  const int waves_per_block = kDecodeThreads / kWave;
  const int blocks = (lay.max_units + waves_per_block - 1) / waves_per_block;
  if (g.Dqk == 128)
    hipLaunchKernelGGL(decode_gqa_kernel<128>, dim3(blocks), dim3(kDecodeThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(decode_gqa_kernel<64>, dim3(blocks), dim3(kDecodeThreads), 0, stream, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(merge_kernel, dim3(g.batch * g.H), dim3(kMergeThreads), 0, stream, pairs, g.H, group, Hq,
                     g.Dv, part_o, part_lse, out);
  return hipGetLastError();
}

}  // namespace vx

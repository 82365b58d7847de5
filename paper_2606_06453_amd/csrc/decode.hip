// Sparse paged attention over the selected pages (Sec. 3.1 Eq. 4; Sec. 5.3).
//
// Work plan (Sec. 5.1: balanced contiguous workload ranges per program).  The host fixes
// a page chunk from the shape it knows (batch, KV heads, max_sel) so that about
// `target_units` units cover the batch: chunk = ceil(B*H*max_sel / target), and
// U = ceil(max_sel / chunk) units per (request, KV head) pair.  Unit w is pair w / U,
// split w % U.  It derives its page range [s*chunk, min(cnt, (s+1)*chunk)) from the
// device-side selection count.  Nothing is materialised and no plan kernel runs; units
// past a pair's count exit at once.  A program walks a balanced contiguous range of units
// (per = n / programs, the first n % programs take one more).
//
// decode_gqa_kernel  one wave per program; a unit is 16-token tiles of its pages:
//                  S^T = K Q^T    MFMA 16x16x32 bf16: 16 tokens x 16 (padded) query heads,
//                                 contraction over D
//                  online softmax in the log2 domain, one running max per query head
//                  O^T += V^T P^T MFMA 16x16x16 bf16: V^T comes from a register
//                                 transpose of 4 token rows per lane.  P is split into
//                                 bf16 hi + lo parts, so the probabilities keep about 16
//                                 bits.
//                K and V tiles are double-buffered in registers: tile t+1 loads while tile
//                t computes.  A pair covered by a single unit writes bf16 output directly
//                (and a pair with no selected page writes zeros).  Otherwise the unit
//                writes a normalised fp32 partial and its log2-sum-exp.
// decode_mla_kernel  the same for the absorbed-weight MLA geometry, one workgroup per
//                program (see its comment below).
// merge_kernel   LSE-weighted combination of the partials of pairs split over several
//                units.  It is launched only when U > 1.  It is a separate launch because
//                on MI355X each XCD has its own L2: a device-scope release/acquire inside
//                the split kernel would write back and invalidate L2 per unit, which costs
//                far more than one extra launch.
#include <climits>

#include "vx_device.h"
#include "vx_internal.h"

namespace vx {
namespace {

constexpr int kDecodeThreads = 256;       // 4 independent programs (waves) per workgroup
constexpr int kGqaTargetUnits = 2048;     // work units the plan aims for (GQA: one wave each)
constexpr int kMlaTargetUnits = 512;      // (MLA: one workgroup each)
constexpr int kMergeThreads = 256;
constexpr int kMergeBatch = 8;            // split partials a merge thread loads per round trip

struct DecodeArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* indptr;
  const int32_t* indices;
  const int32_t* seq_lens;
  const int32_t* sel_pages;
  const int32_t* sel_count;
  uint16_t* out;
  float* part_o;
  float* part_lse;
  int max_sel, H, g, Hq, ps, num_phys;
  int chunk, U, n_units;      // work plan: pages per unit, units per pair, B*H*U
  float scale_log2;           // sm_scale * log2(e)
};

struct Unit {
  int pair, i, h, pb, pe, Ui;
};

// Unit w of the implicit plan: its pair, page range and the pair's unit count.
__device__ __forceinline__ Unit unit_of(const DecodeArgs& a, int w) {
  Unit u;
  u.pair = w / a.U;
  const int s = w - u.pair * a.U;
  u.i = u.pair / a.H;
  u.h = u.pair - u.i * a.H;
  const int cnt = min(max(a.sel_count[u.i], 0), a.max_sel);
  u.pb = s * a.chunk;
  u.pe = min(cnt, u.pb + a.chunk);
  u.Ui = (cnt + a.chunk - 1) / a.chunk;
  return u;
}

// Balanced contiguous range of units for program `prog` of `nprog` (Appendix C template).
__device__ __forceinline__ void program_range(int n, int prog, int nprog, int* b, int* e) {
  const int per = n / nprog, rem = n % nprog;
  *b = prog * per + min(prog, rem);
  *e = *b + per + (prog < rem ? 1 : 0);
}

// ------------------------------------------------------------------------------------
// split kernel, GQA (D = head_dim_qk = head_dim_v)
// ------------------------------------------------------------------------------------
template <int D>
struct Tile {
  bf16x8_t k[D / 32];                  // A operand of S^T = K Q^T: row = lane & 15
  uint32_t v[4][D / 32];               // rows 4*grp + r, channels (lane & 15) * D/16 ..
};

// One 16-token K and V tile into registers.  Every selected token is read once per step, so
// the loads carry the streaming (non-temporal) hint.
template <int D>
__device__ __forceinline__ void load_tile(const uint16_t* __restrict__ kt, const uint16_t* __restrict__ vt,
                                          int col, int grp, Tile<D>& t) {
  constexpr int KS = D / 32, DPL = D / 16;
#pragma unroll
  for (int kk = 0; kk < KS; kk++)
    t.k[kk] = __builtin_bit_cast(bf16x8_t, load_stream_u4(kt + col * D + 32 * kk + 8 * grp));
#pragma unroll
  for (int r = 0; r < 4; r++) {
    const uint16_t* src = vt + (4 * grp + r) * D + col * DPL;
    if constexpr (DPL == 8) {
      const uint4 w = load_stream_u4(src);
      t.v[r][0] = w.x;
      t.v[r][1] = w.y;
      t.v[r][2] = w.z;
      t.v[r][3] = w.w;
    } else {
      const uint2 w = load_stream_u2(src);
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
  int w_begin, w_end;
  program_range(a.n_units, prog, nprog, &w_begin, &w_end);

  for (int w = w_begin; w < w_end; w++) {
    const Unit un = unit_of(a, w);
    const int pair = un.pair, i = un.i, h = un.h;
    if (un.pb >= un.pe) {
      if (un.pb == 0) {                               // no selected page: zero output
        uint16_t* dst = a.out + ((int64_t)i * a.Hq + (int64_t)h * a.g) * D;
        for (int x = lane; x < a.g * D; x += kWave) dst[x] = 0;
      }
      continue;
    }
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

    for (int sb = un.pb; sb < un.pe; sb += kWave) {
      // page metadata of up to 64 selected pages, one per lane
      int my_p = 0, my_n = 0;
      if (sb + lane < un.pe) {
        const int j = sel[sb + lane];
        if (j >= 0 && j < P) {
          my_p = (int)clamp_page(a.indices[base + j], a.num_phys);
          my_n = min(a.ps, L - j * a.ps);
        }
      }
      const int nb = min(kWave, un.pe - sb);
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
    if (un.Ui == 1) {
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
// split kernel, MLA with absorbed weights: 16 query heads share one latent of 576 channels
// (512 content + 64 rope) per token, and V is the first 512 channels of that latent.
// One workgroup (4 waves) is one program.  Each 16-token tile (18 KiB) is copied from
// HBM once into LDS (double-buffered, rows padded to avoid bank conflicts).
//   S^T = K Q^T     the 18 k-steps of 32 channels are split 5/5/4/4 over the waves; the
//                   partial S^T tiles meet in LDS and every wave sums them in the same order
//   O^T += V^T P^T  wave w owns output channels [128w, 128w + 128): 8 MFMA tiles whose
//                   V^T operands come from a register transpose of 4 LDS rows per lane
// ------------------------------------------------------------------------------------
namespace mla {
constexpr int kD = 576, kDv = 512, kTok = 16;
constexpr int kRowBytes = kD * 2 + 16;                  // padded LDS row
constexpr int kTileBytes = kTok * kRowBytes;
constexpr int kChunks = kTok * kD * 2 / 16;             // 16-byte chunks per tile (1152)
constexpr int kChunksPerRow = kD * 2 / 16;              // 72
__device__ __forceinline__ int ks_begin(int w) { return w < 2 ? 5 * w : 10 + 4 * (w - 2); }
__device__ __forceinline__ int ks_count(int w) { return w < 2 ? 5 : 4; }

// HBM -> registers: the tile is one contiguous 18 KiB run of 1152 16-byte chunks; thread t
// takes chunks t, t+256, t+512, t+768 and (t < 128) t+1024.
static_assert(kChunks == 4 * kDecodeThreads + kDecodeThreads / 2, "tile split");

__device__ __forceinline__ void put_chunk(unsigned char* dst, int c, const uint4 v) {
  const int r = c / kChunksPerRow, cc = c - r * kChunksPerRow;
  *reinterpret_cast<uint4*>(dst + r * kRowBytes + cc * 16) = v;
}

// Advance a tile cursor (page slot s of the batch, 16-token tile tt, the page's valid tokens n
// and physical page p) to the next tile of a page with tokens; false when there is none.
// my_n / my_p hold one page per lane, and s is uniform, so every wave walks the same tiles.
__device__ __forceinline__ bool next_tile(int my_n, int my_p, int nb, int& s, int& tt, int& n, int& p) {
  tt++;
  if (tt * kTok < n) return true;
  tt = 0;
  s++;
  while (s < nb && __builtin_amdgcn_readlane(my_n, s) <= 0) s++;
  if (s >= nb) return false;
  n = __builtin_amdgcn_readlane(my_n, s);
  p = __builtin_amdgcn_readlane(my_p, s);
  return true;
}

// One 16-token tile T (in LDS) for the 16 query heads: partial S^T over this wave's k-steps,
// summed over the four waves through sx; online softmax in the log2 domain; O^T += V^T P^T
// for this wave's 128 output channels with P split into bf16 hi + lo.
__device__ __forceinline__ void mla_tile(const unsigned char* T, f32x4_t (*sx)[kWave], int w, int lane, int col,
                                         int grp, int kb, int kn, const bf16x8_t (&qv)[5], int valid,
                                         float scale_log2, float& m, float& lsum, f32x4_t (&acc)[8]) {
  f32x4_t st = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int x = 0; x < 5; x++) {
    if (x < kn) {
      const bf16x8_t kv = *reinterpret_cast<const bf16x8_t*>(T + col * kRowBytes + (32 * (kb + x) + 8 * grp) * 2);
      st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kv, qv[x], st, 0, 0, 0);
    }
  }
  sx[w][lane] = st;
  __syncthreads();
  f32x4_t sf = sx[0][lane];
#pragma unroll
  for (int ww = 1; ww < 4; ww++) {
    const f32x4_t o = sx[ww][lane];
    sf[0] += o[0];
    sf[1] += o[1];
    sf[2] += o[2];
    sf[3] += o[3];
  }
  float sv[4];
#pragma unroll
  for (int r = 0; r < 4; r++) sv[r] = (4 * grp + r < valid) ? sf[r] * scale_log2 : -INFINITY;
  float mt = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
  mt = fmaxf(mt, xor_shfl(mt, 16));
  mt = fmaxf(mt, xor_shfl(mt, 32));
  const float m_new = fmaxf(m, mt);
  const float alpha = exp2f(m - m_new);
  float pr[4];
#pragma unroll
  for (int r = 0; r < 4; r++) pr[r] = exp2f(sv[r] - m_new);
  lsum = lsum * alpha + ((pr[0] + pr[1]) + (pr[2] + pr[3]));
  m = m_new;
#pragma unroll
  for (int j = 0; j < 8; j++) {
    acc[j][0] *= alpha;
    acc[j][1] *= alpha;
    acc[j][2] *= alpha;
    acc[j][3] *= alpha;
  }
  s16x4_t ph, pl;
#pragma unroll
  for (int r = 0; r < 4; r++) {
    const uint32_t hb = f32_to_bf16_rne(pr[r]);
    ph[r] = (short)hb;
    pl[r] = (short)f32_to_bf16_rne(pr[r] - __uint_as_float(hb << 16));
  }
  // V rows 4*grp + r, channels 128*w + 8*col .. +8 (V is the latent's first 512)
  uint32_t vr[4][4];
#pragma unroll
  for (int r = 0; r < 4; r++) {
    const uint4 x = *reinterpret_cast<const uint4*>(T + (4 * grp + r) * kRowBytes + (128 * w + 8 * col) * 2);
    const bool ok = 4 * grp + r < valid;
    vr[r][0] = ok ? x.x : 0u;
    vr[r][1] = ok ? x.y : 0u;
    vr[r][2] = ok ? x.z : 0u;
    vr[r][3] = ok ? x.w : 0u;
  }
#pragma unroll
  for (int j = 0; j < 8; j++) {
    const int q2 = j >> 1;
    s16x4_t av;
    if ((j & 1) == 0) {
      av[0] = (short)(vr[0][q2] & 0xffffu);
      av[1] = (short)(vr[1][q2] & 0xffffu);
      av[2] = (short)(vr[2][q2] & 0xffffu);
      av[3] = (short)(vr[3][q2] & 0xffffu);
    } else {
      av[0] = (short)(vr[0][q2] >> 16);
      av[1] = (short)(vr[1][q2] >> 16);
      av[2] = (short)(vr[2][q2] >> 16);
      av[3] = (short)(vr[3][q2] >> 16);
    }
    acc[j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(av, ph, acc[j], 0, 0, 0);
    acc[j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(av, pl, acc[j], 0, 0, 0);
  }
}
}  // namespace mla

__global__ __launch_bounds__(kDecodeThreads) void decode_mla_kernel(const DecodeArgs a) {
  using namespace mla;
  __shared__ __attribute__((aligned(16))) unsigned char tiles[2][kTileBytes];
  __shared__ f32x4_t sx[2][4][kWave];
  const int tid = threadIdx.x, lane = lane_id(), w = tid >> 6;
  const int col = lane & 15, grp = lane >> 4;
  int w_begin, w_end;
  program_range(a.n_units, (int)blockIdx.x, (int)gridDim.x, &w_begin, &w_end);
  const int kb = ks_begin(w), kn = ks_count(w);

  for (int wu = w_begin; wu < w_end; wu++) {
    const Unit un = unit_of(a, wu);
    const int i = un.i;                                   // one KV head: pair == request
    if (un.pb >= un.pe) {
      if (un.pb == 0) {
        uint16_t* dst = a.out + (int64_t)i * a.Hq * kDv;
        for (int x = tid; x < a.Hq * kDv; x += kDecodeThreads) dst[x] = 0;
      }
      continue;                                           // uniform over the workgroup
    }
    const int L = a.seq_lens[i];
    const int base = a.indptr[i];
    const int P = num_pages(L, a.ps, a.indptr[i + 1] - base, INT_MAX);
    const int32_t* sel = a.sel_pages + (int64_t)i * a.max_sel;

    // Q^T operand for this wave's k-steps: head col, channels 32*kk + 8*grp .. +8
    bf16x8_t qv[5];
    {
      const uint16_t* qp = a.q + ((int64_t)i * a.Hq + col) * kD + 8 * grp;
#pragma unroll
      for (int x = 0; x < 5; x++) qv[x] = *reinterpret_cast<const bf16x8_t*>(qp + 32 * min(kb + x, 17));
    }
    f32x4_t acc[8];
#pragma unroll
    for (int j = 0; j < 8; j++) acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float m = -INFINITY, lsum = 0.f;
    const int64_t page_elems = (int64_t)a.ps * kD;

    for (int sb = un.pb; sb < un.pe; sb += kWave) {
      int my_p = 0, my_n = 0;
      if (sb + lane < un.pe) {
        const int j = sel[sb + lane];
        if (j >= 0 && j < P) {
          my_p = (int)clamp_page(a.indices[base + j], a.num_phys);
          my_n = min(a.ps, L - j * a.ps);
        }
      }
      const int nb = min(kWave, un.pe - sb);
      int s = 0, tt = 0;
      while (s < nb && __builtin_amdgcn_readlane(my_n, s) <= 0) s++;
      if (s >= nb) continue;
      int cur_n = __builtin_amdgcn_readlane(my_n, s);
      int cur_p = __builtin_amdgcn_readlane(my_p, s);

      // The next tile loads into five named registers (plain values, never an array: an
      // array would land in scratch) while the current one computes from LDS.
      uint4 r0, r1, r2, r3, r4;
      const int c4 = tid < kDecodeThreads / 2 ? tid + 4 * kDecodeThreads : tid;   // in bounds either way
#define VX_MLA_GLOAD(ptr)                                          \
  do {                                                             \
    const uint4* src_ = reinterpret_cast<const uint4*>(ptr);       \
    r0 = src_[tid];                                                \
    r1 = src_[tid + kDecodeThreads];                               \
    r2 = src_[tid + 2 * kDecodeThreads];                           \
    r3 = src_[tid + 3 * kDecodeThreads];                           \
    r4 = src_[c4];                                                 \
  } while (0)
#define VX_MLA_LSTORE(dst)                                                         \
  do {                                                                             \
    put_chunk(dst, tid, r0);                                                       \
    put_chunk(dst, tid + kDecodeThreads, r1);                                      \
    put_chunk(dst, tid + 2 * kDecodeThreads, r2);                                  \
    put_chunk(dst, tid + 3 * kDecodeThreads, r3);                                  \
    if (tid < kDecodeThreads / 2) put_chunk(dst, tid + 4 * kDecodeThreads, r4);   \
  } while (0)
#define VX_MLA_TILE(p_, tt_) (a.k + (int64_t)(p_) * page_elems + (int64_t)(tt_) * kTok * kD)
      VX_MLA_GLOAD(VX_MLA_TILE(cur_p, 0));
      VX_MLA_LSTORE(tiles[0]);
      __syncthreads();
      int cur = 0;
      while (true) {
        // the next tile's cursor is the same in every wave; its loads overlap this tile
        int ns = s, ntt = tt, nn = cur_n, np = cur_p;
        const bool more = next_tile(my_n, my_p, nb, ns, ntt, nn, np);
        if (more) VX_MLA_GLOAD(VX_MLA_TILE(np, ntt));
        mla_tile(tiles[cur], sx[cur], w, lane, col, grp, kb, kn, qv, min(kTok, cur_n - kTok * tt), a.scale_log2,
                 m, lsum, acc);
        if (more) VX_MLA_LSTORE(tiles[cur ^ 1]);
        __syncthreads();
        if (!more) break;
        s = ns;
        tt = ntt;
        cur_n = nn;
        cur_p = np;
        cur ^= 1;
      }
#undef VX_MLA_TILE
    }

#undef VX_MLA_GLOAD
#undef VX_MLA_LSTORE
    float lt = lsum + xor_shfl(lsum, 16);
    lt += xor_shfl(lt, 32);
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
    // lane (grp, col) holds channels 128*w + 8*(4*grp + r) + j: 32 contiguous from 128*w + 32*grp
    if (un.Ui == 1) {
      uint16_t* dst = a.out + ((int64_t)i * a.Hq + col) * kDv + 128 * w + 32 * grp;
#pragma unroll
      for (int r = 0; r < 4; r++) {
        uint32_t wv[4];
#pragma unroll
        for (int j = 0; j < 8; j += 2)
          wv[j / 2] = f32_to_bf16_rne(acc[j][r] * inv) | (f32_to_bf16_rne(acc[j + 1][r] * inv) << 16);
        *reinterpret_cast<uint4*>(dst + 8 * r) = make_uint4(wv[0], wv[1], wv[2], wv[3]);
      }
    } else {
      float* dst = a.part_o + ((int64_t)wu * a.g + col) * kDv + 128 * w + 32 * grp;
#pragma unroll
      for (int r = 0; r < 4; r++) {
        *reinterpret_cast<float4*>(dst + 8 * r) =
            make_float4(acc[0][r] * inv, acc[1][r] * inv, acc[2][r] * inv, acc[3][r] * inv);
        *reinterpret_cast<float4*>(dst + 8 * r + 4) =
            make_float4(acc[4][r] * inv, acc[5][r] * inv, acc[6][r] * inv, acc[7][r] * inv);
      }
      if (w == 0 && grp == 0) a.part_lse[(int64_t)wu * a.g + col] = lt > 0.f ? m + __log2f(lt) : -INFINITY;
    }
    __syncthreads();          // the next unit reuses the LDS tiles
  }
}

// ------------------------------------------------------------------------------------
// merge: grid (pair, slice of the pair's g*Dv outputs); one thread per 4 output channels
// ------------------------------------------------------------------------------------
__global__ __launch_bounds__(kMergeThreads) void merge_kernel(const int32_t* __restrict__ sel_count, int max_sel,
                                                              int chunk, int U, int H, int g, int Hq, int Dv,
                                                              const float* __restrict__ part_o,
                                                              const float* __restrict__ part_lse,
                                                              uint16_t* __restrict__ out) {
  const int pair = blockIdx.x;
  const int cnt = min(max(sel_count[pair / H], 0), max_sel);
  const int Ui = (cnt + chunk - 1) / chunk;
  if (Ui <= 1) return;                           // written by the split kernel
  const int first = pair * U;
  const int x = (int)blockIdx.y * kMergeThreads + (int)threadIdx.x;
  if (x >= g * Dv / 4) return;
  const int i = pair / H, h = pair - i * H;
  const int c = (4 * x) / Dv, d = 4 * x - c * Dv;
  // online LSE combine over batches of kMergeBatch splits; every load of a batch is issued
  // before any is used (splits past Ui re-read the last one and weigh zero)
  float mx = -INFINITY, wsum = 0.f;
  float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s0 = 0; s0 < Ui; s0 += kMergeBatch) {
    float l[kMergeBatch];
    float4 p[kMergeBatch];
#pragma unroll
    for (int b = 0; b < kMergeBatch; b++) {
      const int64_t u = first + min(s0 + b, Ui - 1);
      l[b] = part_lse[u * g + c];
      p[b] = *reinterpret_cast<const float4*>(part_o + (u * g + c) * Dv + d);
    }
    float bm = -INFINITY;
#pragma unroll
    for (int b = 0; b < kMergeBatch; b++) {
      if (s0 + b >= Ui) l[b] = -INFINITY;
      bm = fmaxf(bm, l[b]);
    }
    const float m_new = fmaxf(mx, bm);
    if (m_new == -INFINITY) continue;                       // no tokens so far
    const float scale = exp2f(mx - m_new);                  // 0 while mx is -inf
    wsum *= scale;
    o.x *= scale;
    o.y *= scale;
    o.z *= scale;
    o.w *= scale;
#pragma unroll
    for (int b = 0; b < kMergeBatch; b++) {
      const float wgt = exp2f(l[b] - m_new);
      wsum += wgt;
      o.x += wgt * p[b].x;
      o.y += wgt * p[b].y;
      o.z += wgt * p[b].z;
      o.w += wgt * p[b].w;
    }
    mx = m_new;
  }
  if (wsum > 0.f) {
    const float inv = 1.f / wsum;
    o.x *= inv;
    o.y *= inv;
    o.z *= inv;
    o.w *= inv;
  }
  uint16_t* dst = out + ((int64_t)i * Hq + (int64_t)h * g) * Dv;
  *reinterpret_cast<uint2*>(dst + c * Dv + d) = make_uint2(f32_to_bf16_rne(o.x) | (f32_to_bf16_rne(o.y) << 16),
                                                           f32_to_bf16_rne(o.z) | (f32_to_bf16_rne(o.w) << 16));
}

}  // namespace

DecodeLayout decode_layout(int batch, int num_kv_heads, int group, int head_dim_v, int max_sel, bool mla) {
  DecodeLayout L;
  L.target_units = mla ? kMlaTargetUnits : kGqaTargetUnits;
  const long long pairs = (long long)batch * num_kv_heads;
  const long long ms = max_sel > 0 ? max_sel : 1;
  long long chunk = (pairs * ms + L.target_units - 1) / L.target_units;
  chunk = chunk < 1 ? 1 : chunk;
  L.chunk = (int)chunk;
  L.units_per_pair = (int)((ms + chunk - 1) / chunk);
  L.n_units = pairs * L.units_per_pair;
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  size_t off = 0;
  L.off_lse = off;
  off = al(off + sizeof(float) * (size_t)L.n_units * group);
  L.off_o = off;
  off = al(off + sizeof(float) * (size_t)L.n_units * group * head_dim_v);
  L.total = L.units_per_pair > 1 ? off : 256;      // no partials when every pair is one unit
  return L;
}

hipError_t launch_decode(const Geometry& g, const uint16_t* q, int Hq, const int32_t* sel_pages,
                         const int32_t* sel_count, int max_sel, float sm_scale, uint16_t* out, void* ws,
                         const DecodeLayout& lay, hipStream_t stream) {
  if (g.batch == 0) return hipSuccess;
  char* base = reinterpret_cast<char*>(ws);
  float* part_lse = reinterpret_cast<float*>(base + lay.off_lse);
  float* part_o = reinterpret_cast<float*>(base + lay.off_o);
  const int group = Hq / g.H;

  DecodeArgs a;
  a.q = q;
  a.k = g.k;
  a.v = g.v;
  a.indptr = g.indptr;
  a.indices = g.indices;
  a.seq_lens = g.seq_lens;
  a.sel_pages = sel_pages;
  a.sel_count = sel_count;
  a.out = out;
  a.part_o = part_o;
  a.part_lse = part_lse;
  a.max_sel = max_sel;
  a.H = g.H;
  a.g = group;
  a.Hq = Hq;
  a.ps = g.ps;
  a.num_phys = g.num_phys_pages;
  a.chunk = lay.chunk;
  a.U = lay.units_per_pair;
  a.n_units = (int)lay.n_units;
  a.scale_log2 = sm_scale * 1.4426950408889634f;

  const int waves_per_block = kDecodeThreads / kWave;
  if (g.Dqk == 576) {
    hipLaunchKernelGGL(decode_mla_kernel, dim3(a.n_units), dim3(kDecodeThreads), 0, stream, a);
  } else {
    const int blocks = (a.n_units + waves_per_block - 1) / waves_per_block;
    if (g.Dqk == 128)
      hipLaunchKernelGGL(decode_gqa_kernel<128>, dim3(blocks), dim3(kDecodeThreads), 0, stream, a);
    else
      hipLaunchKernelGGL(decode_gqa_kernel<64>, dim3(blocks), dim3(kDecodeThreads), 0, stream, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.U == 1) return e;
  const int slices = (group * g.Dv / 4 + kMergeThreads - 1) / kMergeThreads;
  hipLaunchKernelGGL(merge_kernel, dim3(g.batch * g.H, slices), dim3(kMergeThreads), 0, stream, sel_count, max_sel,
                     a.chunk, a.U, g.H, group, Hq, g.Dv, part_o, part_lse, out);
  return hipGetLastError();
}

}  // namespace vx

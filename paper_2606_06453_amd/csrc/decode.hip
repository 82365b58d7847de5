// Sparse paged attention over the selected pages (Sec. 3.1 Eq. 4; Sec. 5.3).
//
// Work plan (Sec. 5.1 and Appendix C: balanced contiguous workload ranges per program), made on
// the device without a plan launch.  The host fixes a split size T (selection slots) and the
// grid, S workgroups per (request, KV head) pair with S * T >= max_sel, in split-major order.
// From the pair's selection count cnt, loaded in the workgroup's first round trip, the pair has
// ceil(cnt / T) splits: split s covers the contiguous slot range [s T, min((s + 1) T, cnt)), so no
// unit holds more than T pages and a short pair is not split at all; workgroups past the last
// split exit at once (they sit at the end of the grid).  The slot range is known before cnt is,
// so the selection row, the count, the request's length and page-list bounds and the query all
// load in one round trip.  A plan made on the device from every count (one more dependent round
// trip, and a split size that fills one resident round) measured slower on every workload.
//   GQA: the NW waves of a split take its slots round robin, so their shares differ by at most
//        one page.  A split pair is merged in the same kernel: every split stores its partial
//        (o, lse) with agent-coherent stores that write through the L2 of its XCD, waits for
//        them, and bumps the pair's counter; the split that brings the counter to the pair's
//        split count merges the partials, in split order, with agent-coherent loads.  The
//        counter wraps back to zero there, so the counters are zero again after every call.
//        Neither an L2 writeback nor a wait on another workgroup is involved.
//   MLA: split s takes the fixed slot range [s*max_sel/S, (s+1)*max_sel/S), cut at cnt; its
//        partials (16 heads x 512 channels) are too large for one workgroup to merge at a CU's
//        streaming rate, so merge_kernel spreads that merge over the chip.
//
// decode_gqa_kernel  four (or three) waves per workgroup; each wave walks its pages in 16-token
//                tiles:
//                  S^T = K Q^T    MFMA 16x16x32 bf16: 16 tokens x 16 (padded) query heads,
//                                 contraction over D
//                  online softmax in the log2 domain, one running max per query head
//                  O^T += V^T P^T MFMA 16x16x16 bf16: V^T comes from a register
//                                 transpose of 4 token rows per lane.  P is split into
//                                 bf16 hi + lo parts, so the probabilities keep about 16
//                                 bits.
//                K and V tiles are double-buffered in registers: tile t+1 loads while tile
//                t computes.  The waves' (max, sum, accumulator) states meet in LDS and
//                are combined there, so with S = 1 the workgroup writes the bf16 output and
//                no partial result leaves the chip.
// decode_mla_kernel  the same for the absorbed-weight MLA geometry, where the four waves
//                of a workgroup share every latent tile (see its comment below).
// merge_kernel   LSE-weighted combination of the S partials of each MLA request, launched
//                only when S > 1.
#include <algorithm>
#include <climits>
#include <mutex>
#include <type_traits>

#include "vx_device.h"
#include "vx_internal.h"

namespace vx {
namespace {

constexpr int kDecodeWaves = 4;           // waves per GQA workgroup (3 for some batch shapes)
constexpr int kGqaTargetWgs = 512;        // two 4-wave workgroups per CU
constexpr int kGqaWavesPerCu = 12;        // resident GQA split waves per CU (168 VGPRs each)
constexpr int kMlaTargetWgs = 256;        // one workgroup per CU
constexpr int kMergeThreads = 256;
constexpr int kMergeBatch = 8;            // split partials a merge thread loads per round trip

struct DecodeArgs {
  const uint16_t* q;
  const void* k;              // bf16, or fp8 codes
  const void* v;
  const int32_t* indptr;
  const int32_t* indices;
  const int32_t* seq_lens;
  const int32_t* sel_pages;
  const int32_t* sel_count;
  uint16_t* out;
  float* part_o;
  float* part_lse;
  int max_sel, H, g, Hq, ps, num_phys;
  int bs, r;                  // selection unit: blocks of bs tokens, r per page (r = 1: pages)
  int S;                      // workgroups per pair (GQA: most splits of a pair)
  int T;                      // GQA: selection slots per split
  uint32_t* ctr;              // [pairs] split counters, zero between calls (GQA)
  float scale_log2;           // sm_scale * log2(e), times the K scale of an fp8 cache
  float v_scale;              // V scale of an fp8 cache (1 for bf16)
  int order_block;            // GQA, one workgroup per pair: > 0 orders the requests by selection
                              // count (balanced_request) with blocks of this many; 0 keeps them
};

// Every argument into SGPRs at once: one scalar round trip at the kernel's start, where the
// compiler would otherwise load the arguments in batches at their first uses, each behind a
// wait for the one before.
__device__ __forceinline__ void load_args(const DecodeArgs& a) {
  asm volatile("" ::"s"(a.q), "s"(a.k), "s"(a.v), "s"(a.indptr), "s"(a.indices), "s"(a.seq_lens), "s"(a.sel_pages),
               "s"(a.sel_count), "s"(a.out), "s"(a.part_o), "s"(a.part_lse), "s"(a.ctr));
  asm volatile("" ::"s"(a.max_sel), "s"(a.H), "s"(a.g), "s"(a.Hq), "s"(a.ps), "s"(a.num_phys), "s"(a.bs), "s"(a.r),
               "s"(a.S), "s"(a.T), "s"(a.scale_log2), "s"(a.v_scale), "s"(a.order_block));
}

// ------------------------------------------------------------------------------------
// request order by selection count (one workgroup per pair)
// ------------------------------------------------------------------------------------
// The dispatcher places a grid's workgroups one per CU in turn, so with H pairs per request the
// requests whose workgroups share a CU sit C = CUs / H positions apart in the grid.  With skewed
// selection counts (lognormal contexts) a CU that draws several long requests ends last.  The
// workgroup at request position ui serves instead the request of rank snake(ui) when the requests
// are ranked by count (descending; equal counts keep their own order, so equal counts change
// nothing): snake reverses every other block of C positions, so each CU pairs long requests with
// short ones.
constexpr int kBalanceMaxBatch = 1024;

__device__ __forceinline__ int snake_pos(int i, int C, int B) {
  const int m = i / C, j = i - m * C, n = min(C, B - m * C);
  return m * C + ((m & 1) ? n - 1 - j : j);
}

// B <= kBalanceMaxBatch requests.  Ranks by the key (count << 16) | (0xffff - snake_pos(i)): keys
// are distinct, so the ranks are a permutation, and with equal counts rank(i) = snake_pos(i) and
// every workgroup keeps its request.  Uniform over the workgroup (two barriers).
__device__ __forceinline__ int balanced_request(const DecodeArgs& a, int ui, int B) {
  __shared__ uint32_t key[kBalanceMaxBatch];
  __shared__ int target;
  const int C = a.order_block, nt = (int)blockDim.x;
  for (int i = (int)threadIdx.x; i < B; i += nt) {
    const uint32_t c = (uint32_t)min(max(a.sel_count[i], 0), 0xffff);
    key[i] = (c << 16) | (uint32_t)(0xffff - snake_pos(i, C, B));
  }
  __syncthreads();
  const int want = snake_pos(ui, C, B);
  for (int i = (int)threadIdx.x; i < B; i += nt) {
    const uint32_t k = key[i];
    int r = 0;
    for (int x = 0; x < B; x++) r += key[x] > k;
    if (r == want) target = i;
  }
  __syncthreads();
  return target;
}

// ------------------------------------------------------------------------------------
// merge of a split pair (LSE-weighted combination of its S partials)
// ------------------------------------------------------------------------------------
// Output channels 4x .. 4x+3 of pair `pair` from its first S partials (rows pair*Smax + s):
// online LSE combine over batches of kMergeBatch splits, every load of a batch issued before
// any is used (slots past S re-read the last split and weigh zero).  A split that saw no token
// has lse = -inf and an unwritten partial, which is never read into the sum.  lse_at(u) and
// o_at(u) load the log2-sum-exp and the 4 channels of partial row u (offset (u*g + c)*Dv + d).
template <class LseAt, class OAt>
__device__ __forceinline__ void merge_one(int S, int Smax, int H, int g, int Hq, int Dv, uint16_t* out, int pair,
                                          int x, LseAt lse_at, OAt o_at) {
  const int i = pair / H, h = pair - i * H;
  const int c = (4 * x) / Dv, d = 4 * x - c * Dv;
  const int64_t first = (int64_t)pair * Smax;
  float mx = -INFINITY, wsum = 0.f;
  float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s0 = 0; s0 < S; s0 += kMergeBatch) {
    float l[kMergeBatch];
    float4 p[kMergeBatch];
#pragma unroll
    for (int b = 0; b < kMergeBatch; b++) {
      const int64_t u = first + min(s0 + b, S - 1);
      l[b] = lse_at(u * g + c);
      p[b] = o_at((u * g + c) * Dv + d);
    }
    float bm = -INFINITY;
#pragma unroll
    for (int b = 0; b < kMergeBatch; b++) {
      if (s0 + b >= S) l[b] = -INFINITY;
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
      if (l[b] == -INFINITY) continue;
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

// ---- agent-coherent partials -------------------------------------------------------------
// Buffer loads and stores with the sc1 cache policy are coherent across the XCDs' L2 caches
// (the form the compiler gives agent-scope atomic loads and stores): a store writes through
// to memory, a load does not return a line another XCD may have changed.  Raw buffer accesses
// are also bounds-checked against the resource's byte count.
constexpr int kAgentCoherent = 16;                 // cache policy bits: sc1
typedef unsigned int u32x4v_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ __amdgpu_buffer_rsrc_t coherent_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ void coherent_store4(__amdgpu_buffer_rsrc_t r, uint32_t byte_off, float4 v) {
  const u32x4v_t w = {__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z), __float_as_uint(v.w)};
  __builtin_amdgcn_raw_buffer_store_b128(w, r, (int)byte_off, 0, kAgentCoherent);
}
__device__ __forceinline__ void coherent_store1(__amdgpu_buffer_rsrc_t r, uint32_t byte_off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, (int)byte_off, 0, kAgentCoherent);
}
__device__ __forceinline__ float4 coherent_load4(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  const u32x4v_t w = __builtin_amdgcn_raw_buffer_load_b128(r, (int)byte_off, 0, kAgentCoherent);
  return make_float4(__uint_as_float(w.x), __uint_as_float(w.y), __uint_as_float(w.z), __uint_as_float(w.w));
}
__device__ __forceinline__ float coherent_load1(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)byte_off, 0, kAgentCoherent));
}
// Wait until this wave's vector-memory operations (the partial stores) have completed.
__device__ __forceinline__ void wait_vm_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// ------------------------------------------------------------------------------------
// the GQA work plan
// ------------------------------------------------------------------------------------
// A pair with selection count cnt has ceil(cnt / T) splits of at most T slots (one split when
// cnt = 0, which writes zeros).  T is fixed on the host, so a split's slot range is known before
// the count is.
__device__ __forceinline__ int splits_of(int cnt, int T) { return cnt > 0 ? (cnt + T - 1) / T : 1; }

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

// The same tile from an fp8 cache: raw codes, converted to the bf16 Tile just before use
// (every E4M3 / E5M2 value is a bf16 value, so the conversion is exact; the scales are
// applied to the scores and to the output).  A lane's K codes are its KS*8 consecutive
// channels (k-step kk takes the kk-th 8 of them, and the query operand is loaded in the same
// channel order), so they arrive in 16-byte loads: the kernel's time goes with the number of
// load instructions as much as with bytes, and 8-byte loads (channels 32*kk + 8*grp, the bf16
// order) made the E4M3 decode call 23% slower.
template <int D>
struct Tile8 {
  static constexpr int KS = D / 32, DPL = D / 16;
  uint2 k[KS];                         // 8 codes of token col: channels KS*8*grp + 8*kk .. +8
  uint32_t v[4][DPL / 4];              // DPL codes of token rows 4*grp + r, channels col*DPL ..
};

template <int D>
__device__ __forceinline__ void load_tile8(const uint8_t* __restrict__ kt, const uint8_t* __restrict__ vt, int col,
                                           int grp, Tile8<D>& t) {
  constexpr int KS = D / 32, DPL = D / 16;
#pragma unroll
  for (int c = 0; c < KS / 2; c++) {
    const uint4 w = load_stream_u4(kt + col * D + KS * 8 * grp + 16 * c);
    t.k[2 * c] = make_uint2(w.x, w.y);
    t.k[2 * c + 1] = make_uint2(w.z, w.w);
  }
#pragma unroll
  for (int r = 0; r < 4; r++) {
    const uint8_t* src = vt + (4 * grp + r) * D + col * DPL;
    if constexpr (DPL == 8) {
      const uint2 w = load_stream_u2(src);
      t.v[r][0] = w.x;
      t.v[r][1] = w.y;
    } else {
      t.v[r][0] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(src));
    }
  }
}

// Two codes (bytes 2*HI and 2*HI + 1 of w) as a packed bf16 pair.
template <int KT, bool HI>
__device__ __forceinline__ uint32_t fp8x2_bf16x2(uint32_t w) {
  typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
  bf16x2v r;
  if constexpr (KT == kKvFp8E4M3) r = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w, 1.0f, HI);
  else r = __builtin_amdgcn_cvt_scalef32_pk_bf16_bf8((int)w, 1.0f, HI);
  return __builtin_bit_cast(uint32_t, r);
}

template <int D, int KT>
__device__ __forceinline__ void widen_tile(const Tile8<D>& s, Tile<D>& t) {
  constexpr int KS = D / 32, DPL = D / 16;
#pragma unroll
  for (int kk = 0; kk < KS; kk++) {
    const u32x4_t w = {fp8x2_bf16x2<KT, false>(s.k[kk].x), fp8x2_bf16x2<KT, true>(s.k[kk].x),
                       fp8x2_bf16x2<KT, false>(s.k[kk].y), fp8x2_bf16x2<KT, true>(s.k[kk].y)};
    t.k[kk] = __builtin_bit_cast(bf16x8_t, w);
  }
#pragma unroll
  for (int r = 0; r < 4; r++) {
#pragma unroll
    for (int x = 0; x < DPL / 4; x++) {
      t.v[r][2 * x] = fp8x2_bf16x2<KT, false>(s.v[r][x]);
      t.v[r][2 * x + 1] = fp8x2_bf16x2<KT, true>(s.v[r][x]);
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

// Tile loads and compute for either cache element type.
template <int D, int KT>
struct TileOps {
  using Elem = typename std::conditional<KT == kKvBf16, uint16_t, uint8_t>::type;
  using T = typename std::conditional<KT == kKvBf16, Tile<D>, Tile8<D>>::type;
  __device__ static __forceinline__ void load(const Elem* kt, const Elem* vt, int col, int grp, T& t) {
    if constexpr (KT == kKvBf16) load_tile<D>(kt, vt, col, grp, t);
    else load_tile8<D>(kt, vt, col, grp, t);
  }
  __device__ static __forceinline__ void compute(T& t, const bf16x8_t (&qv)[D / 32], int valid, int grp,
                                                 float scale_log2, float& m, float& lsum, f32x4_t (&acc)[D / 16]) {
    if constexpr (KT == kKvBf16) {
      compute_tile<D>(t, qv, valid, grp, scale_log2, m, lsum, acc);
    } else {
      Tile<D> w;
      widen_tile<D, KT>(t, w);
      compute_tile<D>(w, qv, valid, grp, scale_log2, m, lsum, acc);
    }
  }
};

// One wave's share of a split: the online-softmax state (running max m in the log2 domain,
// per-lane partial sum lsum, O^T accumulators) over the selection slots lo + w, lo + w + U,
// lo + w + 2U, ... below min(hi_fixed, cnt) of request i, KV head h.  cnt_all returns the
// request's count, clamped to [0, max_sel].
template <int D, int KT>
__device__ __forceinline__ void gqa_wave_slots(const DecodeArgs& a, int i, int h, int lo, int hi_fixed, int w,
                                               int U, int lane, float& m, float& lsum, f32x4_t (&acc)[D / 16],
                                               int& cnt_all) {
  using Ops = TileOps<D, KT>;
  using Elem = typename Ops::Elem;
  const Elem* kbase = static_cast<const Elem*>(a.k);
  const Elem* vbase = static_cast<const Elem*>(a.v);
  constexpr int KS = D / 32, DPL = D / 16;
  const int col = lane & 15, grp = lane >> 4;
#pragma unroll
  for (int j = 0; j < DPL; j++) acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  m = -INFINITY;
  lsum = 0.f;
  const int32_t* sel = a.sel_pages + ((int64_t)i * a.H + h) * a.max_sel;

  // one round trip: none of these loads depends on another
  const int cnt_raw = a.sel_count[i];
  const int L = a.seq_lens[i];
  const int base = a.indptr[i];
  const int list_len = a.indptr[i + 1] - base;
  // slots stay below max_sel + 64U: int is enough (max_sel and U are bounded on the host)
  const int slot0 = lo + w + U * lane;
  const int j_first = slot0 < hi_fixed ? sel[slot0] : -1;
  bf16x8_t qv[KS];
  {
    const bool hv = col < a.g;
    // fp8 caches: a lane's k-steps take its KS*8 consecutive channels (two 16-byte K loads)
    const uint16_t* qp = a.q + ((int64_t)i * a.Hq + h * a.g + (hv ? col : 0)) * D + (KT == kKvBf16 ? 8 : KS * 8) * grp;
#pragma unroll
    for (int kk = 0; kk < KS; kk++) {
      qv[kk] = *reinterpret_cast<const bf16x8_t*>(qp + (KT == kKvBf16 ? 32 : 8) * kk);
      if (!hv) qv[kk] = bf16x8_t{};
    }
  }
  cnt_all = min(max(cnt_raw, 0), a.max_sel);
  const int cnt = min(cnt_all, hi_fixed);                       // end of this split's slots
  const int P = num_pages(L, a.bs, list_len * a.r, INT_MAX);     // blocks of the request
  const int64_t head_off = (int64_t)h * a.ps * D;
  const int64_t page_stride = (int64_t)a.H * a.ps * D;

  // windows of 64 of the wave's slots (one per lane); the first was loaded above
  for (int w0 = 0; lo + w + U * w0 < cnt; w0 += kWave) {
    const int slot = slot0 + U * w0;
    const int j = w0 == 0 ? j_first : (slot < hi_fixed ? sel[slot] : -1);
    // lane: physical page of its slot's block, and (tile offset of the block in the page) << 16
    // | valid tokens (>= 1 for a real block, 0 for none)
    int my_p = 0, my_n = 0;
    if (slot < cnt && j >= 0 && j < P) {
      const int jp = j / a.r, blk = j - jp * a.r;
      my_p = (int)clamp_page(a.indices[base + jp], a.num_phys);
      my_n = min(a.bs, L - j * a.bs) | ((blk * (a.bs >> 4)) << 16);
    }
    const int nb = min(kWave, (cnt - lo - w - U * w0 + U - 1) / U);
    // Load cursor over (page slot ls, tile ltt) of the pages with n > 0.  fetch() loads the
    // cursor's tile into a register buffer, advances the cursor and returns the tile's valid
    // tokens (0, loading nothing, past the last tile).  Statically named buffers rotate: bf16
    // keeps one tile in flight while one computes, fp8 (tiles of half the registers) two.
    int ls = 0, ltt = 0;
    while (ls < nb && __builtin_amdgcn_readlane(my_n, ls) <= 0) ls++;
    if (ls >= nb) continue;
    auto tile_ptr_k = [&](int p, int t16) { return kbase + p * page_stride + head_off + (int64_t)t16 * 16 * D; };
    auto tile_ptr_v = [&](int p, int t16) { return vbase + p * page_stride + head_off + (int64_t)t16 * 16 * D; };
    auto fetch = [&](typename Ops::T& buf) -> int {
      if (ls >= nb) return 0;
      int n = __builtin_amdgcn_readlane(my_n, ls);
      const int t0 = n >> 16;
      n &= 0xffff;
      const int p = __builtin_amdgcn_readlane(my_p, ls);
      Ops::load(tile_ptr_k(p, t0 + ltt), tile_ptr_v(p, t0 + ltt), col, grp, buf);
      const int valid = min(16, n - 16 * ltt);
      if (++ltt * 16 >= n) {
        ltt = 0;
        ls++;
        while (ls < nb && __builtin_amdgcn_readlane(my_n, ls) <= 0) ls++;
      }
      return valid;
    };
    auto compute = [&](typename Ops::T& buf, int valid) {
      Ops::compute(buf, qv, valid, grp, a.scale_log2, m, lsum, acc);
    };
    if constexpr (KT == kKvBf16) {
      typename Ops::T ta, tb;
      int na = fetch(ta);
      while (true) {
        const int nbt = fetch(tb);
        compute(ta, na);
        if (!nbt) break;
        na = fetch(ta);
        compute(tb, nbt);
        if (!na) break;
      }
    } else {
      typename Ops::T ta, tb, tc;
      int na = fetch(ta), nbt = fetch(tb);
      while (true) {
        const int nct = fetch(tc);
        compute(ta, na);
        if (!nbt) break;
        na = fetch(ta);
        compute(tb, nbt);
        if (!nct) break;
        nbt = fetch(tb);
        compute(tc, nct);
        if (!na) break;
      }
    }
  }
}

// Dynamic LDS of decode_gqa_kernel: per wave, the unnormalised O (g x D fp32), the running
// maxima and the sums of its g query heads.
__host__ __device__ constexpr size_t gqa_merge_lds_bytes(int g, int D, int waves) {
  return sizeof(float) * (size_t)waves * g * (D + 2);
}

// Three waves per SIMD (at most 168 VGPRs): with short selections the per-wave start-up
// round trips weigh as much as the stream, and more resident waves overlap them.
// NW waves per workgroup (4, or 3 when that makes every workgroup of the grid resident at once);
// KT is the cache element type; BAL: the workgroups serve the requests in the count-balanced
// order (balanced_request), else each its own.
template <int D, int NW, int KT, bool BAL>
__global__ __launch_bounds__(NW * kWave) __attribute__((amdgpu_waves_per_eu(3))) void decode_gqa_kernel(
    const DecodeArgs a) {
  constexpr int DPL = D / 16;
  extern __shared__ __attribute__((aligned(16))) float gqa_lds[];
  load_args(a);
  const int lane = lane_id(), wv = (int)threadIdx.x >> 6;
  const int col = lane & 15, grp = lane >> 4;
  __shared__ int last;
  {
    // split-major grid: the first splits of every pair come first, so that later splits (and
    // the splits past a pair's count, which exit at once) queue behind them
    const int pairs = (int)gridDim.x / a.S;
    const int split = (int)blockIdx.x / pairs;
    int ui = ((int)blockIdx.x - split * pairs) / a.H;
    const int uh = (int)blockIdx.x - split * pairs - ui * a.H;
    if constexpr (BAL) ui = balanced_request(a, ui, pairs / a.H);
    const int T = a.T;
    const int pair = ui * a.H + uh;
    const int lo = split * T;                              // < max_sel

    f32x4_t acc[DPL];
    float m, lsum;
    int cnt;
    gqa_wave_slots<D, KT>(a, ui, uh, lo, min(lo + T, a.max_sel), wv, NW, lane, m, lsum, acc, cnt);
    const int Sp = splits_of(cnt, T);                      // uniform: every wave loaded the count
    if (split >= Sp) return;
    float lt = lsum + xor_shfl(lsum, 16);
    lt += xor_shfl(lt, 32);

    // the waves' states meet in LDS
    const int g = a.g;
    float* obuf = gqa_lds;                                 // [wave][g][D]
    float* mbuf = obuf + NW * g * D;                       // [wave][g]
    float* lbuf = mbuf + NW * g;                           // [wave][g]
    if (col < g) {
      // lane (grp, col) holds channels (4*grp + i4)*DPL + j of query head col
      float* dst = obuf + (wv * g + col) * D + 4 * grp * DPL;
#pragma unroll
      for (int i4 = 0; i4 < 4; i4++) {
#pragma unroll
        for (int j = 0; j < DPL; j += 4)
          *reinterpret_cast<float4*>(dst + i4 * DPL + j) =
              make_float4(acc[j][i4], acc[j + 1][i4], acc[j + 2][i4], acc[j + 3][i4]);
      }
      if (grp == 0) {
        mbuf[wv * g + col] = m;
        lbuf[wv * g + col] = lt;
      }
    }
    __syncthreads();
    // partial rows of this pair: (split * g + head) in a region of a.S * g rows that starts at
    // the pair
    const uint32_t pair_rows = (uint32_t)(a.S * g);
    const __amdgpu_buffer_rsrc_t o_rs = coherent_rsrc(a.part_o + (int64_t)pair * pair_rows * D, pair_rows * D * 4u);
    const __amdgpu_buffer_rsrc_t l_rs = coherent_rsrc(a.part_lse + (int64_t)pair * pair_rows, pair_rows * 4u);
    // combine: one thread per 4 consecutive channels of one query head
    for (int x = (int)threadIdx.x; x < g * D / 4; x += NW * kWave) {
      const int c = (4 * x) / D, d = 4 * x - c * D;
      float M = -INFINITY;
#pragma unroll
      for (int k = 0; k < NW; k++) M = fmaxf(M, mbuf[k * g + c]);
      float Ls = 0.f;
      float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
      if (M != -INFINITY) {
#pragma unroll
        for (int k = 0; k < NW; k++) {
          const float mk = mbuf[k * g + c];
          if (mk == -INFINITY) continue;                 // that wave saw no token
          const float w = exp2f(mk - M);
          const float4 v = *reinterpret_cast<const float4*>(obuf + (k * g + c) * D + d);
          Ls += w * lbuf[k * g + c];
          o.x += w * v.x;
          o.y += w * v.y;
          o.z += w * v.z;
          o.w += w * v.w;
        }
      }
      const float inv = Ls > 0.f ? a.v_scale / Ls : 0.f;
      if (Sp == 1) {
        uint16_t* dst = a.out + ((int64_t)ui * a.Hq + uh * g + c) * D + d;
        *reinterpret_cast<uint2*>(dst) = make_uint2(f32_to_bf16_rne(o.x * inv) | (f32_to_bf16_rne(o.y * inv) << 16),
                                                    f32_to_bf16_rne(o.z * inv) | (f32_to_bf16_rne(o.w * inv) << 16));
      } else {
        const uint32_t row = (uint32_t)(split * g + c);
        coherent_store4(o_rs, (row * D + d) * 4u, make_float4(o.x * inv, o.y * inv, o.z * inv, o.w * inv));
        if (d == 0) coherent_store1(l_rs, row * 4u, Ls > 0.f ? M + __log2f(Ls) : -INFINITY);
      }
    }
    if (Sp > 1) {
      // split pair: the last split to arrive merges (the partials are complete before the
      // counter moves: every thread waits for its stores before the barrier that precedes the
      // increment)
      wait_vm_all();
      __syncthreads();
      if (threadIdx.x == 0)
        last = __builtin_amdgcn_atomic_inc32(a.ctr + pair, (uint32_t)(Sp - 1), __ATOMIC_RELAXED, "agent") ==
               (uint32_t)(Sp - 1);
      __syncthreads();
      if (last) {
        for (int x = (int)threadIdx.x; x < g * D / 4; x += NW * kWave)
          merge_one(Sp, 0, a.H, g, a.Hq, D, a.out, pair, x,
                    [&](int64_t e) { return coherent_load1(l_rs, (uint32_t)e * 4u); },
                    [&](int64_t e) { return coherent_load4(o_rs, (uint32_t)e * 4u); });
      }
    }
  }
}


// ------------------------------------------------------------------------------------
// split kernel, MLA with absorbed weights: 16 query heads share one latent of 576 channels
// (512 content + 64 rope) per token, and V is the first 512 channels of that latent.
// One workgroup (8 waves) covers one split.  Its 16-token latent tiles (18 KiB each) stream
// from HBM straight into a ring of LDS slots with direct-to-LDS loads
// (global_load_lds_dwordx4), two pairs of tiles ahead of the pair being computed, with no
// register staging.  The eight waves form two groups of four that take alternate tiles (two
// waves per SIMD hide each other's latency).  Per tile, the waves of its group compute
//   S^T = K Q^T     MFMA 16x16x32 bf16, the 18 k-steps of 32 channels split 5/5/4/4 over the
//                   waves; the partial S^T tiles meet in LDS and every wave adds them in the
//                   same order
//   online softmax in the log2 domain, one running max per query head (the same values in
//                   every wave of the group)
//   O^T += V^T P^T  each wave for its own 128 output channels: 8 MFMA tiles whose V^T operands
//                   come from a register transpose of 4 LDS rows per lane; P split into bf16
//                   hi + lo
// Two barriers per pair of tiles: one for the ring, one for the partial scores.  The two
// groups' (max, sum, accumulator) states are combined in LDS at the end.
// The direct-to-LDS loads are issued from inline assembly.  If the compiler saw them it would
// wait for all of them before every LDS read, which serialises the ring; it schedules the
// LDS reads itself, and the loop waits for the loads with explicit vmcnt counts (vector
// memory operations complete in issue order).
// A slot holds its tile as 16-byte chunks, C per token row (72 for bf16, 36 for an fp8 latent):
// row r, chunk c (channels 8c .. 8c+7 of bf16, 16c .. 16c+15 of fp8) sits at position
// C r + (c ^ (r & 15)) (in the last C mod 16 chunks of a row, where a 4-bit XOR would leave the
// row, r & 7 or r & 3).  This spreads both read patterns (16 rows of one chunk column, 16
// chunks of one row) over the LDS banks.  fp8 tiles (Sec. 5.3, Appendix E cache dtypes) are
// half the bytes; each wave widens its 8-byte operands to bf16 after the LDS read (exact), the
// latent scale goes into the softmax scale and the output.
// ------------------------------------------------------------------------------------
namespace mla {
constexpr int kD = 576, kDv = 512, kTok = 16;
constexpr int kKSteps = kD / 32;                        // 18
constexpr int kThreads = 512;                           // 8 waves: two groups of four
constexpr int kWaves = kThreads / kWave;
constexpr int kRingPairs = 3;                           // LDS slots for 3 pairs of tiles
constexpr int kMergeRow = kDv + 4;                      // padded row of the group merge buffer
static_assert(kKSteps == 18, "tile split");

// Tile geometry of a bf16 (KT = kKvBf16) or fp8 latent.
template <int KT>
struct Tiles {
  static constexpr int kEB = KT == kKvBf16 ? 2 : 1;                 // bytes per element
  static constexpr int kChunksPerRow = kD * kEB / 16;               // 72 or 36
  static constexpr int kFull = kChunksPerRow / 16 * 16;             // chunks under the 4-bit XOR
  static constexpr int kTileBytes = kTok * kD * kEB;                // 18432 or 9216
  static constexpr int kLoadsPerTile = kTileBytes / (kWave * 16);   // 18 or 9 wave-wide loads
  static constexpr int kPairLoads = 2 * kLoadsPerTile;              // 36 or 18 per pair of tiles
  static constexpr int kMaxLoads = (kPairLoads + kWaves - 1) / kWaves;   // 5 or 3 per wave
  // wave w issues loads w, w+8, w+16, ... of each pair of tiles
  static __device__ __forceinline__ int loads_of_wave(int w) {
    return w < kPairLoads - (kMaxLoads - 1) * kWaves ? kMaxLoads : kMaxLoads - 1;
  }
  static __device__ __forceinline__ int slot_pos(int r, int c) {
    return r * kChunksPerRow + (c ^ (r & (c < kFull ? 15 : kChunksPerRow - kFull - 1)));
  }
};

// Workgroup barrier that also completes this wave's LDS accesses first (the compiler does not
// know that the barrier publishes them).
__device__ __forceinline__ void barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// One direct-to-LDS load: lane l's 16 bytes at gptr go to LDS address lds + 16 l.  M0 holds
// the LDS address; the compiler reserves M0, so its value is saved and restored here.
__device__ __forceinline__ void dma16(const void* gptr, uint32_t lds) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds), "v"(gptr)
      : "memory");
}

template <int N>
__device__ __forceinline__ void vm_wait_n() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }
// wait until at most n vector-memory operations of this wave are outstanding (n <= 20)
__device__ __forceinline__ void vm_wait(int n) {
  switch (n) {
#define VX_VMW(k) case k: vm_wait_n<k>(); break;
    VX_VMW(1) VX_VMW(2) VX_VMW(3) VX_VMW(4) VX_VMW(5) VX_VMW(6) VX_VMW(7) VX_VMW(8) VX_VMW(9) VX_VMW(10)
    VX_VMW(11) VX_VMW(12) VX_VMW(13) VX_VMW(14) VX_VMW(15) VX_VMW(16) VX_VMW(17) VX_VMW(18) VX_VMW(19)
    VX_VMW(20)
#undef VX_VMW
    default: vm_wait_n<0>(); break;
  }
}

// Per-lane view of the split's selected pages, 64 slots at a time, and a cursor over their
// 16-token tiles.  Cursor values are wave-uniform.
struct Pages {
  const int32_t* sel;     // the request's selection row
  const int32_t* indices; // the request's page list
  const int32_t* count;   // the request's selection count
  int lo, hi_fixed, P, L, ps, bs, r, num_phys;   // P in blocks of bs tokens, r per page
};
struct Cursor {
  int base, nb;           // first slot of the loaded batch and its size
  int my_p, my_n;         // lane l: physical page, and (tile offset of the block) << 16 | valid
                          // tokens, of slot base + l
  int s, tt, n, p, t0;    // current slot (in batch), tile in block, the block's tokens, page id and
                          // first tile in the page
};
// Slots [sb, sb + 64) of the split: lane l takes slot sb + l.  The selection row is read over
// the split's fixed slot range [lo, hi_fixed) and masked by the selection count afterwards, so
// the row load does not wait for the count.
__device__ __forceinline__ void cursor_load(const Pages& g, int sb, Cursor& c) {
  c.base = sb;
  c.nb = min(kWave, g.hi_fixed - sb);
  int p = 0, n = 0;
  const int lane = lane_id();
  if (lane < c.nb) {
    const int j = g.sel[sb + lane];
    if (sb + lane < *g.count && j >= 0 && j < g.P) {
      const int jp = j / g.r, blk = j - jp * g.r;
      p = (int)clamp_page(g.indices[jp], g.num_phys);
      n = min(g.bs, g.L - j * g.bs) | ((blk * (g.bs / kTok)) << 16);
    }
  }
  c.my_p = p;
  c.my_n = n;
}
// Move to the first slot at or after s (in the loaded batch, then later batches) whose page
// has tokens; false when the split has none left.
__device__ __forceinline__ bool cursor_seek(const Pages& g, Cursor& c, int s) {
  while (true) {
    while (s < c.nb && __builtin_amdgcn_readlane(c.my_n, s) <= 0) s++;
    if (s < c.nb) {
      c.s = s;
      c.tt = 0;
      c.n = __builtin_amdgcn_readlane(c.my_n, s);
      c.t0 = c.n >> 16;
      c.n &= 0xffff;
      c.p = __builtin_amdgcn_readlane(c.my_p, s);
      return true;
    }
    if (c.base + kWave >= g.hi_fixed) return false;
    cursor_load(g, c.base + kWave, c);
    s = 0;
  }
}
__device__ __forceinline__ bool cursor_next(const Pages& g, Cursor& c) {
  if ((c.tt + 1) * kTok < c.n) {
    c.tt++;
    return true;
  }
  return cursor_seek(g, c, c.s + 1);
}

// This wave's direct-to-LDS loads of a pair of tiles (at byte offsets ta and tb of the cache)
// into the two slots at LDS address `slots`: load j = w + 8x (< kPairLoads) belongs to tile
// j / kLoadsPerTile and fills positions 64 (j % kLoadsPerTile) .. + 63 of its slot; goff[x] is
// the byte offset (inside a tile) of the chunk this lane fetches for it.
template <int KT>
__device__ __forceinline__ void issue_pair(const unsigned char* __restrict__ k, int64_t ta, int64_t tb, uint32_t slots,
                                           int w, const int (&goff)[Tiles<KT>::kMaxLoads]) {
  using TL = Tiles<KT>;
#pragma unroll
  for (int x = 0; x < TL::kMaxLoads; x++) {
    const int j = w + kWaves * x;
    if (j < TL::kPairLoads) {
      const int tile = j >= TL::kLoadsPerTile ? 1 : 0;
      const int jj = j - tile * TL::kLoadsPerTile;
      dma16(k + (tile ? tb : ta) + goff[x], slots + (uint32_t)(tile * TL::kTileBytes + jj * kWave * 16));
    }
  }
}
template <int KT>
__device__ __forceinline__ int64_t tile_byte(const Cursor& c, int ps) {
  return ((int64_t)c.p * ps + (int64_t)(c.t0 + c.tt) * kTok) * kD * Tiles<KT>::kEB;
}

// LDS byte offsets (inside a slot) of a lane's operands, the same for every tile:
//   K operand of the wave's k-step ks_begin(w) + x: kofs[x]   (token row col, channels
//     32 kk + 8 grp .. +8: bf16 chunk 4kk + grp, or half grp & 1 of fp8 chunk 2kk + grp / 2)
//   V rows 4*grp + r of the wave's channels 8 (16w + col) .. +8: vofs[r]
// The 18 k-steps of S^T are split 5, 5, 4, 4 over the four waves of a group.
__device__ __forceinline__ int ks_begin(int w) { return w < 2 ? 5 * w : 10 + 4 * (w - 2); }
__device__ __forceinline__ int ks_count(int w) { return w < 2 ? 5 : 4; }
struct TileOffsets {
  uint32_t kofs[5], vofs[4];
};
template <int KT>
__device__ __forceinline__ TileOffsets tile_offsets(int w, int col, int grp) {
  using TL = Tiles<KT>;
  TileOffsets o;
#pragma unroll
  for (int x = 0; x < 5; x++) {
    const int kk = min(ks_begin(w) + x, kKSteps - 1);
    if constexpr (KT == kKvBf16) o.kofs[x] = 16u * (uint32_t)TL::slot_pos(col, 4 * kk + grp);
    else o.kofs[x] = 16u * (uint32_t)TL::slot_pos(col, 2 * kk + (grp >> 1)) + 8u * (uint32_t)(grp & 1);
  }
#pragma unroll
  for (int r = 0; r < 4; r++) {
    if constexpr (KT == kKvBf16) o.vofs[r] = 16u * (uint32_t)TL::slot_pos(4 * grp + r, 16 * w + col);
    else o.vofs[r] = 16u * (uint32_t)TL::slot_pos(4 * grp + r, 8 * w + (col >> 1)) + 8u * (uint32_t)(col & 1);
  }
  return o;
}

// Eight channels of a slot as a bf16 operand: 16 bytes of bf16, or 8 fp8 codes widened exactly.
template <int KT>
__device__ __forceinline__ uint4 operand8(const unsigned char* p) {
  if constexpr (KT == kKvBf16) {
    return *reinterpret_cast<const uint4*>(p);
  } else {
    const uint2 c = *reinterpret_cast<const uint2*>(p);
    return make_uint4(fp8x2_bf16x2<KT, false>(c.x), fp8x2_bf16x2<KT, true>(c.x), fp8x2_bf16x2<KT, false>(c.y),
                      fp8x2_bf16x2<KT, true>(c.y));
  }
}

// Two fp32 values to packed bf16 (round to nearest even), one instruction on gfx950.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{lo, hi}), bf16x2_t));
}

// The running max of a head only moves when a tile's max exceeds it by more than 2^8 (log2
// domain): probabilities then stay below 256, which the fp32 accumulators and the bf16
// hi + lo split of P carry exactly as well as values below 1, and most tiles skip the
// rescale of the accumulators.
constexpr float kRescaleLog2 = 8.f;

// Partial S^T of a 16-token tile in LDS slot T over this wave's k-steps (5, 5, 4, 4 of 18).
template <int KT>
__device__ __forceinline__ f32x4_t mla_partial_s(const unsigned char* T, const TileOffsets& of, int kn,
                                                 const bf16x8_t (&qv)[5]) {
  bf16x8_t kop[5];
#pragma unroll
  for (int x = 0; x < 5; x++) kop[x] = __builtin_bit_cast(bf16x8_t, operand8<KT>(T + of.kofs[x]));
  f32x4_t s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
  s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop[0], qv[0], s0, 0, 0, 0);
  s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop[1], qv[1], s1, 0, 0, 0);
  s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop[2], qv[2], s0, 0, 0, 0);
  s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop[3], qv[3], s1, 0, 0, 0);
  if (kn > 4) s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop[4], qv[4], s0, 0, 0, 0);
  return f32x4_t{s0[0] + s1[0], s0[1] + s1[1], s0[2] + s1[2], s0[3] + s1[3]};
}

// Softmax and O^T for the wave's 128 output channels of a tile in LDS slot T, given the tile's
// full S^T (the group's four partials added in wave order, so every wave holds the same
// values).
template <int KT>
__device__ __forceinline__ void mla_finish(const unsigned char* T, const TileOffsets& of, int grp, const f32x4_t st,
                                           int valid, float scale_log2, float& m, float& lsum, f32x4_t (&acc)[8]) {
  // V rows of this wave's channels
  uint4 x4[4];
#pragma unroll
  for (int r = 0; r < 4; r++) x4[r] = operand8<KT>(T + of.vofs[r]);

  // lane (grp, col) holds S^T[token 4*grp + r][query head col]
  float sv[4];
#pragma unroll
  for (int r = 0; r < 4; r++)
    sv[r] = (4 * grp + r < valid) ? st[r] * scale_log2 : -INFINITY;
  float mt = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
  mt = fmaxf(mt, xor_shfl(mt, 16));
  mt = fmaxf(mt, xor_shfl(mt, 32));
  // the tile has a valid token, so mt is finite; m is -inf before the first tile
  if (__builtin_amdgcn_ballot_w64(mt > m + kRescaleLog2) != 0) {   // wave-uniform
    const float m_new = fmaxf(m, mt);
    const float alpha = __builtin_amdgcn_exp2f(m - m_new);
    lsum *= alpha;
    m = m_new;
#pragma unroll
    for (int j = 0; j < 8; j++) {
      acc[j][0] *= alpha;
      acc[j][1] *= alpha;
      acc[j][2] *= alpha;
      acc[j][3] *= alpha;
    }
  }
  float pr[4];
#pragma unroll
  for (int r = 0; r < 4; r++) pr[r] = __builtin_amdgcn_exp2f(sv[r] - m);   // <= 2^8; 0 for masked rows
  lsum += (pr[0] + pr[1]) + (pr[2] + pr[3]);
  // P^T operand split into bf16 hi + lo: lo = bf16(p - hi) keeps about 16 bits of p
  const uint32_t h01 = pack_bf16x2(pr[0], pr[1]), h23 = pack_bf16x2(pr[2], pr[3]);
  const uint32_t l01 = pack_bf16x2(pr[0] - __uint_as_float(h01 << 16), pr[1] - __uint_as_float(h01 & 0xffff0000u));
  const uint32_t l23 = pack_bf16x2(pr[2] - __uint_as_float(h23 << 16), pr[3] - __uint_as_float(h23 & 0xffff0000u));
  const s16x4_t ph = __builtin_bit_cast(s16x4_t, make_uint2(h01, h23));
  const s16x4_t pl = __builtin_bit_cast(s16x4_t, make_uint2(l01, l23));

  uint32_t vr[4][4];
#pragma unroll
  for (int r = 0; r < 4; r++) {
    vr[r][0] = x4[r].x;
    vr[r][1] = x4[r].y;
    vr[r][2] = x4[r].z;
    vr[r][3] = x4[r].w;
  }
  if (valid < kTok) {                                     // rows past the valid tokens must be zero
#pragma unroll
    for (int r = 0; r < 4; r++) {
      if (4 * grp + r >= valid) vr[r][0] = vr[r][1] = vr[r][2] = vr[r][3] = 0u;
    }
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

template <int KT>
__global__ __launch_bounds__(mla::kThreads) void decode_mla_kernel(const DecodeArgs a) {
  using namespace mla;
  using TL = Tiles<KT>;
  constexpr int kTileBytes = TL::kTileBytes;
  load_args(a);
  // the ring, and after the last tile the two groups' states (2 x 16 rows of kMergeRow floats
  // plus their maxima and sums)
  constexpr int kRingBytes = 2 * kRingPairs * kTileBytes;
  constexpr int kMergeBytes = (2 * 16 * kMergeRow + 4 * 16) * 4;
  __shared__ __attribute__((aligned(1024))) unsigned char ring[kRingBytes > kMergeBytes ? kRingBytes : kMergeBytes];
  // [group][wave][lane] partial S^T.  One buffer is enough: a wave writes it for pair t + 1 only
  // after the ring barrier of pair t + 1, which every wave reaches after its reads of pair t.
  __shared__ f32x4_t sx[2][4][kWave];
  const int tid = threadIdx.x, lane = lane_id();
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: scalar branches and waits
  const int tg = w >> 2, wc = w & 3;                      // tile group, channel block
  const int col = lane & 15, grp = lane >> 4;
  const int nload = TL::loads_of_wave(w);
  const int wu = (int)blockIdx.x;
  const int i = wu / a.S;                                 // one KV head: pair == request
  // Q^T operand (head col, channels 32*kk + 8*grp .. +8), loaded first: it depends on nothing
  // else, so it travels with the metadata loads below
  const int kb = ks_begin(wc), kn = ks_count(wc);
  bf16x8_t qv[5];                                         // this wave's k-steps
  {
    const uint16_t* qp = a.q + ((int64_t)i * a.Hq + col) * kD + 8 * grp;
#pragma unroll
    for (int x = 0; x < 5; x++) qv[x] = *reinterpret_cast<const bf16x8_t*>(qp + 32 * min(kb + x, kKSteps - 1));
  }
  // split s covers the fixed slot range [s*max_sel/S, (s+1)*max_sel/S) of the selection row,
  // cut at the selection count
  const int s_ = wu - i * a.S;
  Pages g;
  g.sel = a.sel_pages + (int64_t)i * a.max_sel;
  g.count = a.sel_count + i;
  g.lo = (int)((int64_t)s_ * a.max_sel / a.S);
  g.hi_fixed = (int)((int64_t)(s_ + 1) * a.max_sel / a.S);
  g.L = a.seq_lens[i];
  const int base = a.indptr[i];
  g.indices = a.indices + base;
  g.P = num_pages(g.L, a.bs, (a.indptr[i + 1] - base) * a.r, INT_MAX);
  g.ps = a.ps;
  g.bs = a.bs;
  g.r = a.r;
  g.num_phys = a.num_phys;

  Cursor ic;                                              // issue cursor, kRingPairs - 1 pairs ahead
  bool iok = false;
  if (g.lo < g.hi_fixed) {
    cursor_load(g, g.lo, ic);
    iok = cursor_seek(g, ic, 0);
  }
  if (!iok) {                                             // no token: uniform over the workgroup
    if (a.S == 1) {
      uint16_t* dst = a.out + (int64_t)i * a.Hq * kDv;
      for (int x = tid; x < a.Hq * kDv; x += kThreads) dst[x] = 0;
    } else if (tid < a.g) {
      a.part_lse[(int64_t)wu * a.g + tid] = -INFINITY;
    }
    return;
  }
  Cursor cc = ic;                                         // compute cursor

  // byte offsets (inside a tile) of this lane's chunks: load j = w + 8x fills positions
  // 64 (j % kLoadsPerTile) .. + 63 of its tile, and position q = C r + (c ^ swizzle(r, c)) holds
  // chunk c of token row r
  int goff[TL::kMaxLoads];
#pragma unroll
  for (int x = 0; x < TL::kMaxLoads; x++) {
    const int j = min(w + kWaves * x, TL::kPairLoads - 1);   // clamp: unissued loads
    const int q = (j % TL::kLoadsPerTile) * kWave + lane;
    const int r = q / TL::kChunksPerRow;
    const int c = TL::slot_pos(r, q - r * TL::kChunksPerRow) - r * TL::kChunksPerRow;  // an involution per row
    goff[x] = r * kD * TL::kEB + 16 * c;
  }

  // Consume the query registers before the first direct-to-LDS load: the compiler does not
  // see those loads, so its wait for the query must come here, not inside the tile loop
  // (where it would also wait for every tile in flight).
#pragma unroll
  for (int x = 0; x < 5; x++) asm volatile("" ::"v"(qv[x]));
  f32x4_t acc[8];
#pragma unroll
  for (int j = 0; j < 8; j++) acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, lsum = 0.f;

  const TileOffsets of = tile_offsets<KT>(wc, col, grp);
  const uint32_t ring0 = (uint32_t)(uintptr_t)ring;
  // Issue the next pair of tiles: the cursor's tile and the one after it.  When the split
  // ends after the first, the second slot receives the first tile again, so that every
  // pair costs every wave the same number of loads (its compute is skipped).
  auto issue_next = [&](int slot_pair) {
    const int64_t ta = tile_byte<KT>(ic, a.ps);
    iok = cursor_next(g, ic);
    const int64_t tb = iok ? tile_byte<KT>(ic, a.ps) : ta;
    if (iok) iok = cursor_next(g, ic);
    issue_pair<KT>(static_cast<const unsigned char*>(a.k), ta, tb, ring0 + (uint32_t)(slot_pair * 2 * kTileBytes), w,
                   goff);
  };
  int issued = 0;
  for (; issued < kRingPairs - 1 && iok; issued++) issue_next(issued);
  for (int t = 0;; t++) {
    vm_wait((issued - t - 1) * nload);                    // this wave's loads of pair t landed
    barrier();                                            // ... and every wave's; pair t-1 is free
    if (iok) {
      issue_next(issued % kRingPairs);
      issued++;
    }
    // group tg computes tile 2t + tg of the split when it exists
    Cursor mine = cc;
    bool has = true;
    if (tg == 1) has = cursor_next(g, mine);
    const unsigned char* T = ring + ((t % kRingPairs) * 2 + tg) * kTileBytes;
    if (has) sx[tg][wc][lane] = mla_partial_s<KT>(T, of, kn, qv);
    barrier();                                            // the group's partials are in LDS
    if (has) {
      const f32x4_t p0 = sx[tg][0][lane], p1 = sx[tg][1][lane];
      const f32x4_t p2 = sx[tg][2][lane], p3 = sx[tg][3][lane];
      const f32x4_t st = {((p0[0] + p1[0]) + p2[0]) + p3[0], ((p0[1] + p1[1]) + p2[1]) + p3[1],
                          ((p0[2] + p1[2]) + p2[2]) + p3[2], ((p0[3] + p1[3]) + p2[3]) + p3[3]};
      mla_finish<KT>(T, of, grp, st, min(kTok, mine.n - kTok * mine.tt), a.scale_log2, m, lsum, acc);
    }
    if (!cursor_next(g, cc) || !cursor_next(g, cc)) break;
  }

  float lt = lsum + xor_shfl(lsum, 16);
  lt += xor_shfl(lt, 32);
  // Both groups' states meet in LDS (the ring is free once every wave is here: no load is in
  // flight after the last pair); then every thread combines 4 channels of one head, so the
  // result leaves in row order: 64 lanes store 1 KiB of contiguous partial (or 512 B of bf16
  // output) per instruction, where the accumulator layout (32 channels of one head per lane)
  // would scatter 16-byte pieces over 64 rows.
  __syncthreads();
  float* obuf = reinterpret_cast<float*>(ring);           // [group][head][kMergeRow]
  float* mbuf = obuf + 2 * 16 * kMergeRow;                // [group][head]
  float* lbuf = mbuf + 2 * 16;
  {
    // lane (grp, col) holds channels 128*wc + 8*(4*grp + r) + j of head col in acc[j][r]
    float* row = obuf + (tg * 16 + col) * kMergeRow + 128 * wc + 32 * grp;
#pragma unroll
    for (int r = 0; r < 4; r++) {
      *reinterpret_cast<float4*>(row + 8 * r) = make_float4(acc[0][r], acc[1][r], acc[2][r], acc[3][r]);
      *reinterpret_cast<float4*>(row + 8 * r + 4) = make_float4(acc[4][r], acc[5][r], acc[6][r], acc[7][r]);
    }
    // every wave of a group holds the same (max, sum) per head
    if (wc == 0 && grp == 0) {
      mbuf[tg * 16 + col] = m;
      lbuf[tg * 16 + col] = lt;
    }
  }
  __syncthreads();
  for (int x = tid; x < 16 * kDv / 4; x += kThreads) {
    const int c = x / (kDv / 4), d = 4 * (x - c * (kDv / 4));
    const float m0 = mbuf[c], m1 = mbuf[16 + c];
    const float M = fmaxf(m0, m1);                          // finite: group 0 saw the first tile
    const float w0 = __builtin_amdgcn_exp2f(m0 - M);
    const float w1 = m1 == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m1 - M);
    const float Lt = w0 * lbuf[c] + w1 * lbuf[16 + c];
    const float inv = Lt > 0.f ? a.v_scale / Lt : 0.f;     // V is the latent: its scale is the K scale
    const float4 u = *reinterpret_cast<const float4*>(obuf + c * kMergeRow + d);
    const float4 v = *reinterpret_cast<const float4*>(obuf + (16 + c) * kMergeRow + d);
    const float4 o = make_float4((w0 * u.x + w1 * v.x) * inv, (w0 * u.y + w1 * v.y) * inv,
                                 (w0 * u.z + w1 * v.z) * inv, (w0 * u.w + w1 * v.w) * inv);
    if (a.S == 1) {
      uint16_t* dst = a.out + ((int64_t)i * a.Hq + c) * kDv + d;
      *reinterpret_cast<uint2*>(dst) = make_uint2(f32_to_bf16_rne(o.x) | (f32_to_bf16_rne(o.y) << 16),
                                                  f32_to_bf16_rne(o.z) | (f32_to_bf16_rne(o.w) << 16));
    } else {
      *reinterpret_cast<float4*>(a.part_o + ((int64_t)wu * a.g + c) * kDv + d) = o;
      if (d == 0) a.part_lse[(int64_t)wu * a.g + c] = Lt > 0.f ? M + __log2f(Lt) : -INFINITY;
    }
  }
}

// ------------------------------------------------------------------------------------
// merge: grid (pair, slice of the pair's g*Dv outputs); one thread per 4 output channels
// ------------------------------------------------------------------------------------
__global__ __launch_bounds__(kMergeThreads) void merge_kernel(int S, int H, int g, int Hq, int Dv,
                                                              const float* __restrict__ part_o,
                                                              const float* __restrict__ part_lse,
                                                              uint16_t* __restrict__ out) {
  const int x = (int)blockIdx.y * kMergeThreads + (int)threadIdx.x;
  if (x < g * Dv / 4)
    merge_one(S, S, H, g, Hq, Dv, out, (int)blockIdx.x, x, [&](int64_t u) { return part_lse[u]; },
              [&](int64_t e) { return *reinterpret_cast<const float4*>(part_o + e); });
}

}  // namespace

DecodeLayout decode_layout(int batch, int num_kv_heads, int group, int head_dim_v, int max_sel, bool mla) {
  DecodeLayout L;
  const long long pairs = (long long)batch * num_kv_heads;
  const long long ms = max_sel > 0 ? max_sel : 1;
  const long long cus = device_cus();
  if (mla) {
    // one workgroup per CU: S splits per request over fixed slot ranges, merged by merge_kernel
    long long S = pairs > 0 ? (kMlaTargetWgs + pairs - 1) / pairs : 1;
    S = S < ms ? S : ms;
    S = S < 1 ? 1 : S;
    L.splits = (int)S;
    L.waves = 8;
    L.n_wg = pairs * S;
  } else {
    // S workgroups per pair so that about kGqaTargetWgs fill the chip when every pair selects
    // max_sel pages; split s covers slots [s T, (s + 1) T), and a pair with count cnt runs
    // ceil(cnt / T) of them
    long long S = pairs > 0 ? (kGqaTargetWgs + pairs - 1) / pairs : 1;
    const long long cap = (ms + kDecodeWaves - 1) / kDecodeWaves;  // a slot for every wave
    S = S < cap ? S : cap;
    S = S < 1 ? 1 : S;
    const long long T = (ms + S - 1) / S;
    S = (ms + T - 1) / T;
    // Three-wave workgroups when that makes a grid of one workgroup per pair resident at once
    // (a second round of workgroups would pay the start-up round trips again).
    const long long resident = cus * kGqaWavesPerCu;
    L.waves = (S == 1 && pairs * kDecodeWaves > resident && pairs * 3 <= resident) ? 3 : kDecodeWaves;
    L.splits = (int)S;
    L.split_slots = (int)T;
    L.n_wg = pairs * S;
  }
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const long long rows = pairs * L.splits;
  size_t off = 0;
  L.off_ctr = off;
  off = al(off + sizeof(uint32_t) * (size_t)(mla ? 0 : pairs));
  L.off_lse = off;
  off = al(off + sizeof(float) * (size_t)rows * group);
  L.off_o = off;
  off = al(off + sizeof(float) * (size_t)rows * group * head_dim_v);
  L.total = L.splits > 1 ? off : 256;      // no partials when no pair can be split
  return L;
}

// ---- allocation-free decode: a file-scope scratch buffer -------------------------------------
// For callers that cannot allocate (code under HIP graph capture, tight serving loops):
// vx_sparse_paged_decode_noalloc runs the decode with this per-device array as its workspace.
// Static device memory is zero when the module loads, and every decode call leaves the split
// counters at its start zero again.  The host never names the array itself: its device address
// comes from hipGetSymbolAddress, once per device, with that device current.
constexpr size_t kNoAllocScratchBytes = size_t(12) << 20;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

hipError_t noalloc_scratch(void** ptr, size_t* bytes) {
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  *bytes = kNoAllocScratchBytes;
  return hipSuccess;
}

hipError_t launch_decode(const Geometry& g, const uint16_t* q, int Hq, const int32_t* sel_pages,
                         const int32_t* sel_count, int max_sel, float sm_scale, uint16_t* out, void* ws,
                         const DecodeLayout& lay, hipStream_t stream) {
  if (g.batch == 0) return hipSuccess;
  char* base = reinterpret_cast<char*>(ws);
  uint32_t* ctr = reinterpret_cast<uint32_t*>(base + lay.off_ctr);
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
  a.bs = g.bs;
  a.r = g.r;
  a.num_phys = g.num_phys_pages;
  a.S = lay.splits;
  a.T = lay.split_slots;
  a.ctr = ctr;
  a.scale_log2 = sm_scale * 1.4426950408889634f * g.k_scale;
  a.v_scale = g.v ? g.v_scale : g.k_scale;               // an aliased V carries the K scale
  // One workgroup per pair, more than two per CU, and a batch the ranking covers: balance the
  // CUs by selection count.  The ranking costs every workgroup a round trip and two barriers
  // before its first tile (about 1 us); with two pairs per CU (the bench workload, equal counts)
  // it measured 1.2 us slower, with four (large_gqa, lognormal contexts) 1.4 us faster (E4M3
  // 2.1 us).
  const int cus = device_cus();
  a.order_block = (g.Dqk != 576 && lay.splits == 1 && (long long)g.batch * g.H > 2LL * cus && g.batch > 1 &&
                   g.batch <= kBalanceMaxBatch)
                      ? std::max(1, cus / g.H)
                      : 0;

  const dim3 grid((unsigned)lay.n_wg);
  if (g.Dqk == 576) {
    if (g.kv_dtype == kKvFp8E4M3)
      hipLaunchKernelGGL(decode_mla_kernel<kKvFp8E4M3>, grid, dim3(mla::kThreads), 0, stream, a);
    else if (g.kv_dtype == kKvFp8E5M2)
      hipLaunchKernelGGL(decode_mla_kernel<kKvFp8E5M2>, grid, dim3(mla::kThreads), 0, stream, a);
    else
      hipLaunchKernelGGL(decode_mla_kernel<kKvBf16>, grid, dim3(mla::kThreads), 0, stream, a);
  } else {
    const size_t lds = gqa_merge_lds_bytes(group, g.Dqk, lay.waves);
    const dim3 block(lay.waves * kWave);
#define VX_GQA(D, NW, KT)                                                                      \
  do {                                                                                         \
    if (a.order_block > 0) hipLaunchKernelGGL((decode_gqa_kernel<D, NW, KT, true>), grid, block, lds, stream, a); \
    else hipLaunchKernelGGL((decode_gqa_kernel<D, NW, KT, false>), grid, block, lds, stream, a); \
  } while (0)
#define VX_GQA_KT(D, NW)                                     \
  do {                                                       \
    if (g.kv_dtype == kKvFp8E4M3) VX_GQA(D, NW, kKvFp8E4M3); \
    else if (g.kv_dtype == kKvFp8E5M2) VX_GQA(D, NW, kKvFp8E5M2); \
    else VX_GQA(D, NW, kKvBf16);                             \
  } while (0)
    if (g.Dqk == 128) {
      if (lay.waves == 3) VX_GQA_KT(128, 3);
      else VX_GQA_KT(128, 4);
    } else {
      if (lay.waves == 3) VX_GQA_KT(64, 3);
      else VX_GQA_KT(64, 4);
    }
#undef VX_GQA_KT
#undef VX_GQA
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.S == 1 || g.Dqk != 576) return e;      // GQA merges in the split kernel
  const int slices = (group * g.Dv / 4 + kMergeThreads - 1) / kMergeThreads;
  hipLaunchKernelGGL(merge_kernel, dim3(g.batch * g.H, slices), dim3(kMergeThreads), 0, stream, a.S, g.H, group,
                     Hq, g.Dv, part_o, part_lse, out);
  return hipGetLastError();
}

}  // namespace vx

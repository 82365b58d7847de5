// Indexer stage: page scores (Sec. 3.1 Eq. 2; Sec. 3.2 Quest) and the selection of sink,
// local and top-scoring pages (Sec. 3.1 Eq. 3; Sec. 6.4 setup).
//
// score_kernel   HBM-bound stream over the summaries, on a persistent grid: balanced
//                contiguous ranges of the batch's page references per workgroup (Appendix C
//                template).  A row of 16 lanes owns one (page, KV head) item.  Each lane
//                holds D/16 channels of the summary and of the query view.  Products
//                accumulate in fp64 and reduce across the row with DPP, then round once to
//                fp32.  Output goes to a scratch table scores[h][i][j] (rows padded to 4).
// topk_kernel    One workgroup per (request, KV head).  It runs an exact radix select over
//                an order-preserving uint32 key of the fp32 score.  Passes start at the
//                highest bit where the candidates' smallest and largest keys differ and take
//                up to 8 bits each.  Each pass builds a double-buffered LDS histogram, and
//                one wave scans its bins.  Keys stay cached in LDS, and all score loads are
//                issued in one round trip.  That finds the K_free-th best candidate.
//                Ties at the threshold go to the lowest page index.  Each thread owns a
//                contiguous page range: one block scan ranks the tied pages and a second
//                compacts the forced and chosen pages in ascending order.
#include "summary_task.h"
#include "vx_device.h"
#include "vx_internal.h"

#include <algorithm>

namespace vx {
namespace {

constexpr int kThreads = 256;
constexpr int kRows = kThreads / 16;     // 16-lane rows per workgroup

// Score kinds.  The first three are the ABI's 0..2; kMeanBound is the first pass of the exact
// two-pass block-mean selection (bf16 means give an approximate score and a rigorous bound);
// the envelope flows of the agent-proposed algorithms (Appendix G) are the ABI's 3..5:
//   kQuestConsensus  min over heads of sum_c max(q Max, q Min)   (head-consensus Quest)
//   kEnvLower        max over heads of sum_c min(q Max, q Min)   (pessimistic envelope)
//   kQuestRectified  max over heads of sum_c ReLU(q Max)         (rectified Quest)
// kHeadDot is the first step of the NSA flow: one logit q_r . Mean per query head.
// kQuestBound .. kRectifiedBound are the first passes of the exact two-pass selection for the
// four envelope kinds: fp32 sums of the exact products with a rigorous bound, an interval that
// holds the one-pass score.
enum { kMeanDot = 0, kQuest = 1, kMaxDot = 2, kMeanBound = 3, kQuestConsensus = 4, kEnvLower = 5,
       kQuestRectified = 6, kHeadDot = 7, kQuestBound = 8, kConsensusBound = 9, kEnvLowerBound = 10,
       kRectifiedBound = 11 };
constexpr int kNoRescore = -1;           // two-pass re-scoring kind of a one-pass selection
// ABI kinds beyond the first six: the block mean over the content channels (scored by kMeanDot
// with the other query channels zero), NSA (kHeadDot, then the flow kernel) and positional
// smoothing (kMeanDot, then the flow kernel).
constexpr int kAbiContent = 6, kAbiNsa = 7, kAbiSmooth = 8;
// Envelope kinds (a per-head Max/Min envelope), those that read Min too, and those that read q
// per head (staged as fp32 in row order) instead of the group mean.
constexpr bool is_env(int k) { return k == kQuest || k == kQuestConsensus || k == kEnvLower || k == kQuestRectified; }
constexpr bool is_env_bound(int k) { return k >= kQuestBound && k <= kRectifiedBound; }
// envelope kind of a bound kind, and the bound kind of an envelope kind
constexpr int env_of_bound(int k) {
  return k == kQuestBound ? kQuest : k == kConsensusBound ? kQuestConsensus : k == kEnvLowerBound ? kEnvLower
                                                                                                 : kQuestRectified;
}
constexpr int bound_of_env(int k) {
  return k == kQuest ? kQuestBound : k == kQuestConsensus ? kConsensusBound : k == kEnvLower ? kEnvLowerBound
                                                                                             : kRectifiedBound;
}
constexpr bool needs_min(int k) {
  return k == kQuest || k == kQuestConsensus || k == kEnvLower || k == kQuestBound || k == kConsensusBound ||
         k == kEnvLowerBound;
}
constexpr bool per_head(int k) { return is_env(k) || is_env_bound(k) || k == kHeadDot; }
// Kinds whose scores table holds a lower and an upper plane.
constexpr bool has_bounds(int k) { return k == kMeanBound || is_env_bound(k); }
// Kinds that read fp32 Mean rows.
constexpr bool reads_mean(int k) { return k == kMeanDot || k == kHeadDot; }
// Internal kind of an ABI score kind.
constexpr int internal_kind(int abi) {
  return abi <= 2 ? abi : abi <= 5 ? abi + 1 : abi == kAbiNsa ? kHeadDot : kMeanDot;
}

// Channel mapping of a 16-lane row: lane u owns the chunks u, u+16, u+32, ... of a summary
// row, so every load instruction of a row reads 16 contiguous chunks.  The query
// view uses the same mapping (a dot product does not care about channel order).
template <int D, bool BF16>
struct RowMap {
  // 16-byte chunks, or 8-byte bf16 ones when D is not a multiple of 128 (D = 64, 576)
  static constexpr int kElemsPerChunk = BF16 ? (D % 128 == 0 ? 8 : 4) : 4;
  static constexpr int kChunks = D / kElemsPerChunk / 16;     // chunks per lane
  static constexpr int E = kChunks * kElemsPerChunk;          // channels per lane
  static_assert(E * 16 == D, "a row of 16 lanes must cover every channel");
  __device__ static int channel(int u, int c, int e) { return (u + 16 * c) * kElemsPerChunk + e; }
};

// Raw words of one summary row held by one lane: W 32-bit words (fp32 values, or bf16 pairs).
template <int D, bool BF16>
struct RowWords {
  using M = RowMap<D, BF16>;
  static constexpr int W = BF16 ? M::E / 2 : M::E;
  static constexpr int kWordsPerChunk = W / M::kChunks;
};

template <int D, bool BF16>
__device__ __forceinline__ void load_row_words(const void* base, int u, uint32_t (&w)[RowWords<D, BF16>::W]) {
  using M = RowMap<D, BF16>;
  using R = RowWords<D, BF16>;
  const char* b = reinterpret_cast<const char*>(base);
  constexpr int kBytesPerElem = BF16 ? 2 : 4;
#pragma unroll
  for (int c = 0; c < M::kChunks; c++) {
    const char* src = b + (size_t)M::channel(u, c, 0) * kBytesPerElem;
    if constexpr (R::kWordsPerChunk == 4) {
      const uint4 v = load_stream_u4(src);
      w[4 * c] = v.x;
      w[4 * c + 1] = v.y;
      w[4 * c + 2] = v.z;
      w[4 * c + 3] = v.w;
    } else {
      const uint2 v = load_stream_u2(src);
      w[2 * c] = v.x;
      w[2 * c + 1] = v.y;
    }
  }
}

// Channel value e of a lane's row from its raw words.
template <int D, bool BF16>
__device__ __forceinline__ float row_value(const uint32_t (&w)[RowWords<D, BF16>::W], int e) {
  if constexpr (BF16) return (e & 1) ? bf16hi(w[e >> 1]) : bf16lo(w[e >> 1]);
  else return __uint_as_float(w[e]);
}

// Items (page, KV head) per row in one pipeline stage: about 128 bytes of loads per lane
// (64 for the envelope kinds, one-pass and bound pass), in two stages, one loading while the
// other computes.  Measured on the bench workload: 128 bytes per lane beat 64 and 256 (fewer
// waves fit per SIMD at 256), also for the per-head logits.  The envelope bound passes keep four
// waves per SIMD at 64 bytes (115 VGPRs, 149 at 128): Quest on the long-generation workload
// takes 53.4 us at 64 bytes, 54.2 at 128.
template <int D, int KIND>
constexpr int items_per_stage() {
  constexpr int bytes_per_item = (reads_mean(KIND) || needs_min(KIND) ? 4 : 2) * D / 16;
  constexpr int u = (is_env(KIND) || is_env_bound(KIND) ? 64 : 128) / bytes_per_item;
  return u < 1 ? 1 : (u > 8 ? 8 : u);
}

// Row stride of the scores table: a multiple of 4 floats, so that rows can be read as float4.
constexpr int score_stride(int max_pages) { return (max_pages + 3) & ~3; }

constexpr int kChunk = 256;           // page ids staged per chunk (one per thread)
constexpr int kMaxLdsBatch = 4096;    // page_indptr staged in LDS up to this batch
constexpr size_t kLdsPerCu = 160 * 1024;
// Balanced ranges per resident workgroup slot.  Above 1, workgroups queue for slots and the
// dispatcher hands them out as slots free up.
constexpr int kScoreGridFactor = 1;

// The block-mean (or Max) score of one (page, head) row: fp64 products of the lane's
// channels in RowMap order, then the fp64 DPP sum over the 16-lane row, rounded to fp32.
// The one-pass kernel and the two-pass re-scoring both call this, so the two selections
// see bit-identical scores.
template <int D, bool BF16>
__device__ __forceinline__ float exact_row_score(const double (&qb)[D / 16],
                                                 const uint32_t (&w)[RowWords<D, BF16>::W]) {
  double acc = 0.0;
#pragma unroll
  for (int e = 0; e < D / 16; e++) acc = fma(qb[e], (double)row_value<D, BF16>(w, e), acc);
  return (float)row16_sum_f64(acc);
}

// Group-mean query view in RowMap order: fp64 sums of the group's bf16 query values (exact),
// then one division (a multiplication by 1/g when g is a power of two, also exact).
__device__ __forceinline__ double finish_qbar_one(double sum, int g) {
  return (g & (g - 1)) == 0 ? sum * (1.0 / (double)g) : sum / (double)g;
}

// First four 16-byte chunks of each thread (chunks tid + kThreads*t) of request i's Hq x D
// bf16 query block, loaded early so that they travel with other loads.
struct QueryPrefetch {
  uint4 v[4];
  int req = -1;
};
__device__ __forceinline__ void query_prefetch(const uint16_t* __restrict__ q, int i, int n8, QueryPrefetch& p) {
  const uint4* src = reinterpret_cast<const uint4*>(q + (int64_t)i * n8 * 8);
#pragma unroll
  for (int t = 0; t < 4; t++) p.v[t] = src[min((int)threadIdx.x + kThreads * t, n8 - 1)];
  p.req = i;
}

// Request i's query block (n8 chunks) into LDS through put(chunk, index): the prefetched
// chunks when they are request i's, the rest loaded four per thread per round trip.  Indices
// past the end are clamped (a duplicate rewrites the same value), so no load waits behind a
// branch.
template <class Put>
__device__ __forceinline__ void stage_query_block(const uint16_t* __restrict__ q, int i, int n8,
                                                  const QueryPrefetch& pre, Put put) {
  const uint4* src = reinterpret_cast<const uint4*>(q + (int64_t)i * n8 * 8);
  int x0 = threadIdx.x;
  if (pre.req == i) {
#pragma unroll
    for (int t = 0; t < 4; t++) put(pre.v[t], min(x0 + kThreads * t, n8 - 1));
    x0 += 4 * kThreads;
  }
  for (; x0 < n8; x0 += 4 * kThreads) {
    uint4 v[4];
#pragma unroll
    for (int t = 0; t < 4; t++) v[t] = src[min(x0 + kThreads * t, n8 - 1)];
#pragma unroll
    for (int t = 0; t < 4; t++) put(v[t], min(x0 + kThreads * t, n8 - 1));
  }
}

// Request i's raw bf16 query block (n8 16-byte chunks) into LDS.  Issued where no summary load
// is in flight, so that waiting for it waits for nothing else.
__device__ __forceinline__ void load_query_raw(const uint16_t* __restrict__ q, int i, int n8, const QueryPrefetch& pre,
                                               uint4* __restrict__ qraw) {
  stage_query_block(q, i, n8, pre, [&](uint4 w, int x) { qraw[x] = w; });
}

// Barrier over LDS only: the wave's LDS accesses complete, global loads stay in flight.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Per-head kinds: the raw query block (LDS) as fp32 in each row's channel order,
// qs[(r * 16 + u) * E + e].  Ends with an LDS barrier.
template <int D, bool BF16>
__device__ __forceinline__ void convert_query(const uint4* __restrict__ qraw, int Hq, float* __restrict__ qs) {
  using M = RowMap<D, BF16>;
  constexpr int E = D / 16;
  const int n8 = Hq * D / 8;
  for (int x = threadIdx.x; x < n8; x += kThreads) {
    const uint4 w = qraw[x];
    const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int t = 0; t < 8; t++) {
      const int flat = 8 * x + t, r = flat / D, c = flat - r * D;
      const int chunk = c / M::kElemsPerChunk, e_in = c - chunk * M::kElemsPerChunk;
      const int uu = chunk % 16, cc = chunk / 16;              // inverse of RowMap::channel
      qs[(r * 16 + uu) * E + cc * M::kElemsPerChunk + e_in] = (t & 1) ? bf16hi(ws[t >> 1]) : bf16lo(ws[t >> 1]);
    }
  }
  lds_barrier();
}

// Group-mean query of every KV head from the raw query block (LDS): qbar[h][c] = (sum over
// r < g of q[h*g + r][c]) / g, the sum in fp64 in head order (exact for bf16 values), then
// finish_qbar's division; channels c >= qdims are zero (the content-channel score leaves the
// rope channels out).  Ends with an LDS barrier.
template <int D>
__device__ __forceinline__ void finish_qbar(const uint4* __restrict__ qraw, int Hq, int H, int qdims,
                                            double* __restrict__ qbar) {
  const int g = Hq / H;
  const uint16_t* qh = reinterpret_cast<const uint16_t*>(qraw);
  for (int t = threadIdx.x; t < H * D; t += kThreads) {
    const int h = t / D, c = t - h * D;
    double acc = 0.0;
    for (int r = 0; r < g; r++) acc += (double)bf16_to_f32(qh[(h * g + r) * D + c]);
    qbar[t] = c < qdims ? finish_qbar_one(acc, g) : 0.0;
  }
  lds_barrier();
}


// Float nearest to x in the given direction (x finite).
__device__ __forceinline__ float f64_to_f32_down(double x) {
  float f = (float)x;
  return (double)f > x ? nextafterf(f, -INFINITY) : f;
}
__device__ __forceinline__ float f64_to_f32_up(double x) {
  float f = (float)x;
  return (double)f < x ? nextafterf(f, INFINITY) : f;
}

// The four heads' per-lane partial sums p[0..3] over the 16 lanes of a row, scattered:
// lanes u and u ^ 8 (row rotation by 8) trade halves so that the lower half keeps heads 0
// and 1 and the upper half 2 and 3; lanes u and 7 - u (half-row mirror) then keep one head
// each; the quad sums the rest.  Lane u returns the total of head u / 4.
template <class T, int CTRL>
__device__ __forceinline__ T dpp_t(T x) {
  if constexpr (sizeof(T) == 8) return dpp_f64<CTRL>(x);
  else return dpp_f32<CTRL>(x);
}
template <class T>
__device__ __forceinline__ T reduce_scatter4(const T (&p)[4], int u) {
  const bool up = (u & 8) != 0;
  const T s0 = up ? p[0] : p[2], s1 = up ? p[1] : p[3];
  const T k0 = (up ? p[2] : p[0]) + dpp_t<T, 0x128>(s0);
  const T k1 = (up ? p[3] : p[1]) + dpp_t<T, 0x128>(s1);
  const bool odd = (u & 4) != 0;
  const T s = odd ? k0 : k1;
  T z = (odd ? k1 : k0) + dpp_t<T, 0x141>(s);
  z += dpp_t<T, 0x4E>(z);                          // quad lanes u ^ 2
  z += dpp_t<T, 0xB1>(z);                          // quad lanes u ^ 1
  return z;
}

// Exact score of an envelope kind for one (page, KV head) item held by a 16-lane row: lane u
// has the RowMap channels of the item's Max row in wa and Min row in wb (wa again when the kind
// reads no Min).  For each query head r of the group, the lane adds its channels' terms in
// channel order in fp64 (each term, a product of two bf16 values or its max / min / ReLU, is
// exact in fp32), the row reduces the sums, and the heads combine by max (head consensus: min).
// Every lane of the row returns the fp64 score.  qs holds the query rows as fp32 in row order:
// head h g + r at qs + ((h g + r) 16 + u) E.  The one-pass score kernel and the two-pass
// re-scoring both call this, so the two selections see bit-identical scores.
template <int KIND, int D>
__device__ __forceinline__ double env_exact(const float* qs, int h, int g, int u,
                                            const uint32_t (&wa)[RowWords<D, true>::W],
                                            const uint32_t (&wb)[RowWords<D, true>::W]) {
  constexpr int E = D / 16;
  if (g == 4) {
    // the four heads' sums reduced together, then the max (min) over the quads that hold them:
    // half-row mirror (quads 0 and 1, 2 and 3), then rotation by 8
    double p[4];
#pragma unroll
    for (int r = 0; r < 4; r++) {
      const float* qr = qs + ((h * 4 + r) * 16 + u) * E;
      double acc = 0.0;
#pragma unroll
      for (int e = 0; e < E; e++) {
        const float x = qr[e] * row_value<D, true>(wa, e);     // exact
        if constexpr (KIND == kQuestRectified) {
          acc += (double)fmaxf(x, 0.f);
        } else {
          const float y = qr[e] * row_value<D, true>(wb, e);   // exact
          acc += (double)(KIND == kEnvLower ? fminf(x, y) : fmaxf(x, y));
        }
      }
      p[r] = acc;
    }
    double z = reduce_scatter4(p, u);
    if constexpr (KIND == kQuestConsensus) {
      z = fmin(z, dpp_f64<0x141>(z));
      z = fmin(z, dpp_f64<0x128>(z));
    } else {
      z = fmax(z, dpp_f64<0x141>(z));
      z = fmax(z, dpp_f64<0x128>(z));
    }
    return z;
  }
  double s = KIND == kQuestConsensus ? INFINITY : -INFINITY;
  for (int r = 0; r < g; r++) {
    const float* qr = qs + ((h * g + r) * 16 + u) * E;
    double acc = 0.0;
#pragma unroll
    for (int e = 0; e < E; e++) {
      const float x = qr[e] * row_value<D, true>(wa, e);     // exact
      if constexpr (KIND == kQuestRectified) {
        acc += (double)fmaxf(x, 0.f);
      } else {
        const float y = qr[e] * row_value<D, true>(wb, e);   // exact
        acc += (double)(KIND == kEnvLower ? fminf(x, y) : fmaxf(x, y));
      }
    }
    acc = row16_sum_f64(acc);
    if constexpr (KIND == kQuestConsensus) s = acc < s ? acc : s;
    else s = acc > s ? acc : s;
  }
  return s;
}

// Maximum over the 16 lanes of a DPP row; every lane of the row receives it.
__device__ __forceinline__ float row16_max_f32(float x) {
  x = fmaxf(x, dpp_f32<0x128>(x));
  x = fmaxf(x, dpp_f32<0x124>(x));
  x = fmaxf(x, dpp_f32<0x122>(x));
  x = fmaxf(x, dpp_f32<0x121>(x));
  return x;
}
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xf, 0xf, false);
}
__device__ __forceinline__ uint32_t row16_max_u32(uint32_t x) {
  x = max(x, dpp_u32<0x128>(x));
  x = max(x, dpp_u32<0x124>(x));
  x = max(x, dpp_u32<0x122>(x));
  x = max(x, dpp_u32<0x121>(x));
  return x;
}

// Packed pairs of bf16 values in a 32-bit word (channel 2k in the low half, 2k + 1 in the high).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef unsigned short u16x2_t __attribute__((ext_vector_type(2)));
typedef short i16x2_t __attribute__((ext_vector_type(2)));
// a.lo b.lo + a.hi b.hi + c (v_dot2c_f32_bf16).  Its rounding is not that of an fp32 fma chain:
// the terms are aligned to the largest one and the sum rounded, which a probe of 4 M operand
// triples (products and accumulators from 2^-30 to 2^30, near cancellations, subnormals) measured
// at no more than 2.9 units of 2^-24 (|a.lo b.lo| + |a.hi b.hi| + |c|) per instruction, with
// subnormal products and results flushed to zero.
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), c, false);
}
// Per-half unsigned maximum of two packed words.
__device__ __forceinline__ uint32_t pk_max_u16(uint32_t a, uint32_t b) {
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(u16x2_t, a),
                                                                __builtin_bit_cast(u16x2_t, b)));
}
// 0xffff in each half whose sign bit is set, else 0.
__device__ __forceinline__ uint32_t pk_sign_mask(uint32_t a) {
  return __builtin_bit_cast(uint32_t, __builtin_bit_cast(i16x2_t, a) >> (i16x2_t)15);
}

// ------------------------------------------------------------------------------------
// Score policies.  MEAN_DOT / MAX_DOT: s_j = (mean_r q_r) . S_j (equal to the mean over the
// group's heads of q_r . S_j by linearity); the group-mean query is formed in fp64 from the
// staged query (exact for bf16 inputs) and kept in registers (a row always serves one head).
// QUEST: s_j = max_r sum_c max(q_rc Max_jc, q_rc Min_jc); each product of two bf16 values is
// exact in fp32, the per-head sums run in fp64, and q is read from LDS.
// ------------------------------------------------------------------------------------
template <int KIND, int D>
struct ScorePolicy {
  static constexpr bool kBf16 = !reads_mean(KIND);    // Max, Min, or the bf16 copy of Mean
  static constexpr int E = D / 16;
  static constexpr int U = items_per_stage<D, KIND>();
  static constexpr int W = RowWords<D, kBf16>::W;
  struct Stage {
    uint32_t a[U][W];                     // Mean / Max rows
    uint32_t b[needs_min(KIND) ? U : 1][needs_min(KIND) ? W : 1];   // Min rows
  };
  // kHeadDot with groups of 1, 2 or 4 query heads and D <= 128 keeps the row's channels of the
  // group's query heads in registers as fp64 (the other geometries read them from LDS per item)
  static constexpr bool kHeadRegs = KIND == kHeadDot && D <= 128;
  double qb[KIND == kMeanBound || per_head(KIND) ? 1 : E];  // the row's channels of qbar (exact, fp64)
  float qf[KIND == kMeanBound ? E : 1];   // kMeanBound: the same channels rounded to fp32
  float qabs;                             // kMeanBound: sum over the row of |qf_c|
  double qh[kHeadRegs ? 4 : 1][kHeadRegs ? E : 1];
  // bound kinds: the row's channels of the group's (at most four) query heads as packed bf16
  // pairs split by sign (qp: the channels with q >= 0, the others zero; qn: those with q < 0),
  // zero for heads past g, and the 1-norm over all D channels of this lane's head u / 4
  static constexpr bool kBound = is_env_bound(KIND);
  uint32_t qp[kBound ? 4 : 1][kBound ? E / 2 : 1], qn[kBound ? 4 : 1][kBound ? E / 2 : 1];
  float qnorm;

  static __device__ __forceinline__ bool head_regs(int g) { return kHeadRegs && (g == 1 || g == 2 || g == 4); }

  // kHeadDot: the row's channels of query heads h g + r (qs: the request's query block in LDS,
  // fp32 in row order), exact as fp64.
  __device__ __forceinline__ void on_new_request_heads(const float* qs, int h, int g, int u) {
    if constexpr (kHeadRegs) {
      if (!head_regs(g)) return;
#pragma unroll
      for (int r = 0; r < 4; r++)
#pragma unroll
        for (int e = 0; e < E; e++) qh[r][e] = r < g ? (double)qs[((h * g + r) * 16 + u) * E + e] : 0.0;
    }
  }

  // kHeadDot, G = g query heads per KV head: the G logits z_r = q_r . Mean of one item from
  // registers.  Each lane forms its G partial sums (fp64 products, exact), then the row
  // reduces them with a reduce-scatter: at each of the first log2(G) levels a lane keeps half
  // of its heads and adds its partner's half (row rotation by 8, then the half-row mirror), and
  // the lanes left holding the same head sum their partials over the quad.  Lanes 16/G apart
  // then hold the G totals; one of each writes its logit, rounded once to fp32.
  template <int G>
  __device__ __forceinline__ void head_logits(const uint32_t (&w)[W], int h, int u, int jj, float* __restrict__ out,
                                              int64_t plane) const {
    double p[G];
#pragma unroll
    for (int r = 0; r < G; r++) p[r] = 0.0;
#pragma unroll
    for (int e = 0; e < E; e++) {
      const double m = (double)row_value<D, false>(w, e);
#pragma unroll
      for (int r = 0; r < G; r++) p[r] = fma(qh[r][e], m, p[r]);
    }
    double z;
    if constexpr (G == 1) {
      z = row16_sum_f64(p[0]);
    } else if constexpr (G == 4) {
      z = reduce_scatter4(p, u);
    } else {
      const bool up = (u & 8) != 0;                // lanes u and u ^ 8 keep one head each
      const double s = up ? p[0] : p[1];
      z = (up ? p[1] : p[0]) + dpp_f64<0x128>(s);
      z += dpp_f64<0x141>(z);                      // lanes u and 7 - u of the half row
      z += dpp_f64<0x4E>(z);                       // quad lanes u ^ 2
      z += dpp_f64<0xB1>(z);                       // quad lanes u ^ 1
    }
    constexpr int span = 16 / G;                   // lanes holding one head's total
    if (u % span == 0) out[(int64_t)(h * (G - 1) + u / span) * plane + jj] = (float)z;
  }

  // Bound kinds: the row's query registers and the head norms (qs: the request's query block in
  // LDS, fp32 in row order; g <= 4).
  __device__ __forceinline__ void on_new_request_bound(const float* qs, int h, int g, int u) {
    if constexpr (kBound) {
      float nrm[4];
#pragma unroll
      for (int r = 0; r < 4; r++) {
        float a = 0.f;
#pragma unroll
        for (int k = 0; k < E / 2; k++) {
          uint32_t pos = 0u, neg = 0u;
#pragma unroll
          for (int half = 0; half < 2; half++) {
            const float x = r < g ? qs[((h * g + r) * 16 + u) * E + 2 * k + half] : 0.f;
            a += fabsf(x);
            const uint32_t bits = (__float_as_uint(x) >> 16) << (16 * half);   // x is a bf16 value
            if (x >= 0.f) pos |= bits;
            else neg |= bits;
          }
          qp[r][k] = pos;
          qn[r][k] = neg;
        }
        nrm[r] = row16_sum_f32(a);
      }
      const int mh = u >> 2;
      qnorm = mh == 0 ? nrm[0] : mh == 1 ? nrm[1] : mh == 2 ? nrm[2] : nrm[3];
    }
  }

  // The row's view of the group-mean query of KV head h (qbar: [H][D] fp64 in LDS).
  __device__ __forceinline__ void on_new_request(const double* qbar, int h, int u) {
    using MQ = RowMap<D, kBf16>;
    if constexpr (KIND == kMeanBound) {
      float a = 0.f;
#pragma unroll
      for (int c = 0; c < MQ::kChunks; c++)
#pragma unroll
        for (int e = 0; e < MQ::kElemsPerChunk; e++) {
          qf[c * MQ::kElemsPerChunk + e] = (float)qbar[h * D + MQ::channel(u, c, e)];
          a += fabsf(qf[c * MQ::kElemsPerChunk + e]);
        }
      qabs = row16_sum_f32(a);
    } else if constexpr (!per_head(KIND)) {
#pragma unroll
      for (int c = 0; c < MQ::kChunks; c++)
#pragma unroll
        for (int e = 0; e < MQ::kElemsPerChunk; e++)
          qb[c * MQ::kElemsPerChunk + e] = qbar[h * D + MQ::channel(u, c, e)];
    }
  }

  __device__ __forceinline__ void load(Stage& st, const float* __restrict__ mean, const uint16_t* __restrict__ maxs,
                                       const uint16_t* __restrict__ mins, const int* pid, int H, int h, int u,
                                       int j0, int slots, int nj) {
#pragma unroll
    for (int v = 0; v < U; v++) {
      // items past the chunk's end load nothing (compute skips them): every load costs the CU
      // an issue slot, cached or not.  The row's slot is the same for the wave's rows, so the
      // branch is uniform.
      const int jj = j0 + v * slots;
      if (jj >= nj) continue;
      const int64_t o = ((int64_t)pid[jj] * H + h) * D;
      if constexpr (reads_mean(KIND)) {
        load_row_words<D, false>(mean + o, u, st.a[v]);
      } else {
        load_row_words<D, true>(maxs + o, u, st.a[v]);      // Max, or the bf16 Mean copy
        if constexpr (needs_min(KIND)) load_row_words<D, true>(mins + o, u, st.b[v]);
      }
    }
  }

  // Scores of the stage's items; lane v of the row keeps item v's score, and one store per
  // plane writes them all: out[jj] (and, for the bounds, the upper one at out[plane + jj]).
  // kHeadDot writes one logit per query head r of the group instead, lane r storing it to
  // out[(h (g - 1) + r) plane + jj], the row of query head h g + r.
  __device__ __forceinline__ void compute(const Stage& st, const float* qs, int h, int g, int u, int j0, int slots,
                                          int nj, float* __restrict__ out, int64_t plane) const {
    float mine = 0.f, mine_up = 0.f;
#pragma unroll
    for (int v = 0; v < U; v++) {
      const int jj = j0 + v * slots;
      if (jj < nj) {
        double s;
        if constexpr (is_env(KIND)) {
          double z;
          if constexpr (needs_min(KIND)) z = env_exact<KIND, D>(qs, h, g, u, st.a[v], st.b[v]);
          else z = env_exact<KIND, D>(qs, h, g, u, st.a[v], st.a[v]);
          if (u == v) mine = (float)z;
          continue;
        } else if constexpr (kBound) {
          // Per head, the sum of the exact terms t_c = q_c (q_c >= 0 ? a_c : b_c), with a, b = Max,
          // Min for Quest and the head consensus (max(q Max, q Min) is q Max for q >= 0, q Min
          // below), Min, Max for the pessimistic envelope, and max(Max, 0), min(Max, 0) for
          // rectified Quest: t_c = q+_c a_c + q-_c b_c with q+ = q where q >= 0 (else 0) and q- the
          // rest, two chains of bf16 pair dot products (dot2_bf16) per head, two channels per
          // step, added at the end; the row then reduces over 4 levels of fp32 additions.  Error:
          // each of a chain's n = E/2 steps is off by at most K 2^-24 (|its two products| + |the
          // running sum|); with K = 8 (the instruction measured at most 2.9) a chain is off by at
          // most n K 2^-24 sum |t_c| over its terms, so the fp32 sum differs from the exact one by
          // at most (4 K + 5) 2^-24 sum |t_c| < 2^-18.7 sum |t_c| (D = 128; less for D = 64), and
          // sum |t_c| <= |q_h|_1 m with m the largest |Max_c|, |Min_c| of the item.  The one-pass
          // fp64 sum is within 2^-40 sum |t_c| of the exact one, rounding the interval ends adds
          // at most 2^-23 |q_h|_1 m, and the fp32 norm and product fall short of |q_h|_1 m by a
          // factor of at most 1 - 2^-19: b = |q_h|_1 m 2^-18 covers all of these.  Subnormal
          // operands, products and sums flushed to zero lose at most 2^-126 (|q_h|_1 + D m) plus
          // 2^-126 per step over the row, which (|q_h|_1 + m) 2^-110 + 2^-110 covers.  So every
          // head's one-pass sum lies in [s_h - b, s_h + b].  The max (min) over the heads of the
          // ends then brackets the one-pass score, before and after its rounding to fp32
          // (monotone).  m is taken on the bf16 bit patterns (magnitudes order as integers); an
          // item with an infinite or NaN Max / Min gets the interval (-inf, inf), so its exact
          // score decides.
          float ax[4] = {0.f, 0.f, 0.f, 0.f}, ay[4] = {0.f, 0.f, 0.f, 0.f};
          uint32_t mb = 0u;
#pragma unroll
          for (int k = 0; k < E / 2; k++) {
            const uint32_t wa = st.a[v][k];
            uint32_t wb = wa;
            if constexpr (needs_min(KIND)) wb = st.b[v][k];
            mb = pk_max_u16(mb, wa & 0x7fff7fffu);
            if constexpr (needs_min(KIND)) mb = pk_max_u16(mb, wb & 0x7fff7fffu);
            uint32_t pa = wa, pb = wb;                   // paired with q >= 0, with q < 0
            if constexpr (KIND == kEnvLowerBound) {
              pa = wb;
              pb = wa;
            } else if constexpr (KIND == kRectifiedBound) {
              const uint32_t neg = pk_sign_mask(wa);
              pa = wa & ~neg;
              pb = wa & neg;
            }
#pragma unroll
            for (int r = 0; r < 4; r++) {
              ax[r] = dot2_bf16(qp[r][k], pa, ax[r]);
              ay[r] = dot2_bf16(qn[r][k], pb, ay[r]);
            }
          }
          float acc[4];
#pragma unroll
          for (int r = 0; r < 4; r++) acc[r] = ax[r] + ay[r];
          const float z = reduce_scatter4(acc, u);           // lane u: head u / 4
          const uint32_t mbits = row16_max_u32(max(mb << 16, mb & 0xffff0000u));
          const float m = __uint_as_float(mbits);
          const bool finite = mbits < 0x7f800000u;             // uniform over the row
          const float b = qnorm * m * 0x1p-18f + (qnorm + m) * 0x1p-110f + 0x1p-110f;
          constexpr float kNone = KIND == kConsensusBound ? INFINITY : -INFINITY;
          float lo = (u >> 2) < g ? (finite ? z - b : -INFINITY) : kNone;
          float hi = (u >> 2) < g ? (finite ? z + b : INFINITY) : kNone;
          if constexpr (KIND == kConsensusBound) {
            lo = fminf(lo, dpp_f32<0x141>(lo));
            hi = fminf(hi, dpp_f32<0x141>(hi));
            lo = fminf(lo, dpp_f32<0x128>(lo));
            hi = fminf(hi, dpp_f32<0x128>(hi));
          } else {
            lo = fmaxf(lo, dpp_f32<0x141>(lo));
            hi = fmaxf(hi, dpp_f32<0x141>(hi));
            lo = fmaxf(lo, dpp_f32<0x128>(lo));
            hi = fmaxf(hi, dpp_f32<0x128>(hi));
          }
          if (u == v) {
            mine = lo;
            mine_up = hi;
          }
          continue;
        } else if constexpr (KIND == kHeadDot) {
          if constexpr (kHeadRegs) {
            if (g == 4) { head_logits<4>(st.a[v], h, u, jj, out, plane); continue; }
            if (g == 2) { head_logits<2>(st.a[v], h, u, jj, out, plane); continue; }
            if (g == 1) { head_logits<1>(st.a[v], h, u, jj, out, plane); continue; }
          }
          // z_r = q_r . Mean: fp64 products (q is a bf16 value held in fp32) and sums, one
          // rounding to fp32
          double mine_z = 0.0;
          for (int r = 0; r < g; r++) {
            const float* qr = qs + ((h * g + r) * 16 + u) * E;
            double acc = 0.0;
#pragma unroll
            for (int e = 0; e < E; e++) acc = fma((double)qr[e], (double)row_value<D, false>(st.a[v], e), acc);
            acc = row16_sum_f64(acc);
            if (u == r) mine_z = acc;
          }
          if (u < g) out[(int64_t)(h * (g - 1) + u) * plane + jj] = (float)mine_z;
          continue;
        } else if constexpr (KIND == kMeanBound) {
          // In fp32: s' = qf . m and A' = sum |qf_c| |m_c| with m = bf16(Mean) and qf = fp32(qbar).
          // The exact score s (fp64 products of qbar and the fp32 Mean, one rounding to fp32)
          // differs from s' by at most
          //   2^-8 A    RNE to bf16 moves a normal channel by at most 2^-8 of its bf16 value
          //             (a subnormal one by 2^-134: the qabs * 2^-133 term)
          //   2^-24 A   rounding qbar to fp32
          //   40 u A    the fp32 evaluation (D/16 <= 36 fused steps per lane, 4 tree levels;
          //             u = 2^-24)
          //   2^-40 A   the fp64 evaluation of s, and its final rounding (monotone, so it keeps
          //             any fp32 bound on the fp64 value)
          // with A = sum |qbar_c m_c| <= A' (1 + 2^-18).  b = A' (2^-8 + 2^-16) covers all of
          // these plus the fp32 rounding of s' -/+ b itself (at most u (|s'| + b) <= 2^-23 A');
          // 2^-120 covers products that underflow.  So L = s' - b <= s <= s' + b = U.
          float acc = 0.f, aab = 0.f;
#pragma unroll
          for (int e = 0; e < E; e++) {
            const float x = row_value<D, true>(st.a[v], e);
            acc = fmaf(qf[e], x, acc);
            aab = fmaf(fabsf(qf[e]), fabsf(x), aab);
          }
          acc = row16_sum_f32(acc);
          aab = row16_sum_f32(aab);
          const float b = aab * (0x1p-8f + 0x1p-16f) + qabs * 0x1p-133f + 0x1p-120f;
          if (u == v) {
            mine = acc - b;
            mine_up = acc + b;
          }
          continue;
        } else {
          s = exact_row_score<D, kBf16>(qb, st.a[v]);
        }
        if (u == v) mine = (float)s;
      }
    }
    const int jj = j0 + u * slots;
    if constexpr (KIND != kHeadDot) {
      if (u < U && jj < nj) {
        out[jj] = mine;
        if constexpr (has_bounds(KIND)) out[plane + jj] = mine_up;
      }
    }
  }
};

// Byte offsets of the score kernel's dynamic LDS regions (16-byte aligned) and its size.
struct ScoreLds {
  int ind, raw, q, qbar, total;
};
template <int KIND, int D>
__host__ __device__ inline ScoreLds score_lds(int batch, int Hq, int H) {
  ScoreLds L;
  L.ind = 0;
  L.raw = batch <= kMaxLdsBatch ? ((2 * batch + 1) * 4 + 15) & ~15 : 0;   // page_indptr, seq_lens
  L.q = L.raw + Hq * D * 2;
  L.qbar = L.q + (per_head(KIND) ? Hq * D * 4 : 0);
  L.total = L.qbar + (per_head(KIND) ? 0 : H * D * 8);
  return L;
}

struct ScoreArgs {
  const uint16_t* q;
  const int32_t* indptr;
  const int32_t* indices;
  const int32_t* seq_lens;
  const float* mean;
  const uint16_t* maxs;
  const uint16_t* mins;
  float* scores;
  int64_t plane;                       // kMeanBound: floats per scores plane (H * B * stride);
                                       // kHeadDot: floats per query head's rows (B * stride)
  int Hq, H, ps, num_phys, max_pages, batch;   // ps: block size; max_pages: blocks per request
  int r;                               // blocks per page
  int qdims;                           // query channels that enter the group-mean scores
  int stride;                          // row stride of the scores table (max_pages rounded up to 4)
};

// Persistent score kernel following the sequence-local template (Appendix C): the page
// references of the whole batch, in page_indptr order, are split into one balanced
// contiguous range per workgroup.  A workgroup walks its range in chunks of up to 256 pages
// that never cross a request, with one barrier per chunk.  The next chunk's page ids load
// while the current chunk's summaries stream through each row's two-stage pipeline, and
// every row stores its own scores.  The query work of a new request runs while the chunk's
// first loads are in flight.
template <int KIND, int D, bool LDS_IND>
__global__ __launch_bounds__(kThreads) void score_kernel(const ScoreArgs a) {
  using P = ScorePolicy<KIND, D>;

  __shared__ int pid[2][kChunk];
  // dynamic LDS: page_indptr (batch <= kMaxLdsBatch), the raw bf16 query block of the next
  // request to stage, then the per-head kinds' fp32 query in row order [Hq][16][E], or the
  // other kinds' qbar [H][D] fp64
  extern __shared__ uint4 dyn_lds[];
  const ScoreLds L = score_lds<KIND, D>(a.batch, a.Hq, a.H);
  int* ind_lds = reinterpret_cast<int*>(reinterpret_cast<char*>(dyn_lds) + L.ind);
  uint4* qraw = reinterpret_cast<uint4*>(reinterpret_cast<char*>(dyn_lds) + L.raw);
  float* qs = reinterpret_cast<float*>(reinterpret_cast<char*>(dyn_lds) + L.q);
  double* qbar = reinterpret_cast<double*>(reinterpret_cast<char*>(dyn_lds) + L.qbar);
  const int tid = threadIdx.x;
  const int B = a.batch;
  if constexpr (LDS_IND) {
    for (int x = tid; x <= B; x += kThreads) ind_lds[x] = a.indptr[x];
    for (int x = tid; x < B; x += kThreads) ind_lds[B + 1 + x] = a.seq_lens[x];
  }
  __syncthreads();
  // block references: request i's blocks are [indptr[i] * r, indptr[i + 1] * r).  With the
  // page_indptr and the lengths in LDS, the cursor waits on LDS only, never on the summary loads
  // in flight (a wait for a global load issued after them would wait for them too).
  auto ind = [&](int x) -> int { return (LDS_IND ? ind_lds[x] : a.indptr[x]) * a.r; };
  auto len = [&](int i) -> int { return LDS_IND ? ind_lds[B + 1 + i] : a.seq_lens[i]; };
  const int T = ind(B);
  int k0, k1;
  {
    const int n = T, prog = (int)blockIdx.x, nprog = (int)gridDim.x;
    const int per = n / nprog, rem = n % nprog;
    k0 = prog * per + min(prog, rem);
    k1 = k0 + per + (prog < rem ? 1 : 0);
  }
  if (k0 >= k1) return;                                  // uniform over the block
  // request holding k0: the last i with ind(i) <= k0
  int lo = 0, hi = B - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (ind(mid) <= k0) lo = mid;
    else hi = mid - 1;
  }

  const int row = tid >> 4, u = tid & 15;
  const int h = row % a.H, slot = row / a.H, slots = kRows / a.H;
  const int g = a.Hq / a.H;

  // Chunk cursor: request ci, refs [ck, cend), of which the first cn are pages (logical pages
  // from cj).  A chunk's end needs only the page-list bounds; its page count needs the request's
  // length, a global load that is issued with the chunk's page ids and read after them.
  auto advance = [&](int& i, int k) {
    while (i < B - 1 && ind(i + 1) <= k) i++;
    return min(k1, min(k + kChunk, ind(i + 1)));
  };
  auto pages_in = [&](int i, int k, int end, int L, int& j0) {
    const int base = ind(i);
    const int P = num_pages(L, a.ps, ind(i + 1) - base, a.max_pages);
    j0 = k - base;
    return max(0, min(end, base + P) - k);               // refs past P_i are not pages
  };

  int ci = lo, ck = k0;
  int cend = advance(ci, ck);
  // The first request's query rows, the chunk's page ids and the request's length load
  // together: every reference of [ck, cend) lies in the request's page list, so the ids past its
  // last page are read (in bounds) and never used.  The raw query block reaches LDS before any
  // summary load is issued, so the staging below waits on LDS only (a wait for a query register
  // after the summary loads would wait for those too).
  const int n8 = a.Hq * D / 8;
  int cn, cj;
  {
    QueryPrefetch pre;
    query_prefetch(a.q, ci, n8, pre);
    if (tid < cend - ck) pid[0][tid] = (int)block_row(a.indices, ck + tid, a.r, a.num_phys);
    load_query_raw(a.q, ci, n8, pre, qraw);
    cn = pages_in(ci, ck, cend, len(ci), cj);
  }
  QueryPrefetch none;                                   // req -1: nothing prefetched
  int buf = 0, cur_req = -1, raw_req = ci;
  int next_raw = 0;                                      // the next chunk's page id (raw), per thread
  P pol;
  while (true) {
    __syncthreads();                                     // pid[buf] and qraw ready; last chunk's q reads done
    // the chunk's first stage is in flight while the query work below runs
    const bool active = cn > 0 && slot < cn;
    const int step = P::U * slots;
    const int* pc = pid[buf];
    typename P::Stage sa, sb;
    if (active) pol.load(sa, a.mean, a.maxs, a.mins, pc, a.H, h, u, slot, slots, cn);
    if (ci != cur_req && cn > 0) {                       // uniform over the block; qraw holds ci's block
      if constexpr (per_head(KIND)) {
        convert_query<D, P::kBf16>(qraw, a.Hq, qs);
        if constexpr (KIND == kHeadDot) pol.on_new_request_heads(qs, h, g, u);
        if constexpr (is_env_bound(KIND)) pol.on_new_request_bound(qs, h, g, u);
      } else {
        finish_qbar<D>(qraw, a.Hq, a.H, a.qdims, qbar);
        pol.on_new_request(qbar, h, u);
      }
      cur_req = ci;
    }
    // next chunk: its end, and its raw page ids into a register, consumed after this chunk's
    // summaries (the block rows are formed there, so nothing waits for the load before)
    int ni = ci, nk = cend, nend = cend;
    const bool more = nk < k1;
    if (more) {
      nend = advance(ni, nk);
      if (tid < nend - nk) next_raw = a.indices[(nk + tid) / a.r];
    }
    if (active) {
      float* out = a.scores + ((int64_t)h * B + ci) * a.stride + cj;    // this chunk's pages, head h
      int j0 = slot;
      while (true) {
        int jn = j0 + step;
        if (jn < cn) pol.load(sb, a.mean, a.maxs, a.mins, pc, a.H, h, u, jn, slots, cn);
        pol.compute(sa, qs, h, g, u, j0, slots, cn, out, a.plane);
        if (jn >= cn) break;
        j0 = jn;
        jn = j0 + step;
        if (jn < cn) pol.load(sa, a.mean, a.maxs, a.mins, pc, a.H, h, u, jn, slots, cn);
        pol.compute(sb, qs, h, g, u, j0, slots, cn, out, a.plane);
        if (jn >= cn) break;
        j0 = jn;
      }
    }
    if (!more) break;
    int nj0;
    const int nn = pages_in(ni, nk, nend, len(ni), nj0);
    // The empty asm consumes the raw id here, on every lane: the compiler can neither fold the
    // clamp into the load's branch nor leave the load pending into the next chunk, and either
    // would make it wait for the load, and for every summary load issued before it, ahead of
    // a chunk's work.
    asm volatile("" : "+v"(next_raw));
    if (tid < nn) {                                    // read after the next loop-top barrier
      const int jb = nk + tid, qb = jb / a.r;
      pid[buf ^ 1][tid] = (int)(clamp_page(next_raw, a.num_phys) * a.r + (jb - qb * a.r));
    }
    // the next request's raw query block, after this chunk's loads (no reader of qraw is left:
    // the staging above ended with a barrier)
    if (ni != raw_req) {                                 // uniform over the block
      load_query_raw(a.q, ni, n8, none, qraw);
      raw_req = ni;
    }
    buf ^= 1;
    ci = ni;
    ck = nk;
    cn = nn;
    cj = nj0;
    cend = nend;
  }
}

// ------------------------------------------------------------------------------------
// top-K selection, one workgroup per (request, KV head)
// ------------------------------------------------------------------------------------
__device__ __forceinline__ bool is_forced(int j, int P, int n_sink, int n_local) {
  return j < n_sink || j >= P - n_local;
}

constexpr int kMaxLdsKeys = 8192;      // candidates kept in LDS; longer requests re-read scores

// Wave-wide inclusive scans in lane order through DPP moves, with no LDS round trip: shifts by 1,
// 2, 4 and 8 lanes within each row of 16, then the row totals carried forward by the broadcasts of
// lane 15 (into rows 1 and 3) and lane 31 (into rows 2 and 3).  A lane that a move leaves without
// a source takes the operation's identity.  Lane 63 ends with the whole wave's value.  The whole
// wave must be active.
template <int CTRL, int ROWS = 0xf>
__device__ __forceinline__ uint32_t dpp_move(uint32_t x, uint32_t identity) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)identity, (int)x, CTRL, ROWS, 0xf, false);
}
template <typename Op>
__device__ __forceinline__ uint32_t wave_scan_bits(uint32_t x, uint32_t identity, Op op) {
  x = op(x, dpp_move<0x111>(x, identity));          // row_shr:1
  x = op(x, dpp_move<0x112>(x, identity));          // row_shr:2
  x = op(x, dpp_move<0x114>(x, identity));          // row_shr:4
  x = op(x, dpp_move<0x118>(x, identity));          // row_shr:8
  x = op(x, dpp_move<0x142, 0xa>(x, identity));     // row_bcast:15
  x = op(x, dpp_move<0x143, 0xc>(x, identity));     // row_bcast:31
  return x;
}
__device__ __forceinline__ int wave_incl_sum(int x) {
  return (int)wave_scan_bits((uint32_t)x, 0u, [](uint32_t a, uint32_t b) { return a + b; });
}
__device__ __forceinline__ uint32_t wave_last(uint32_t x) { return (uint32_t)__builtin_amdgcn_readlane((int)x, 63); }
__device__ __forceinline__ float wave_min_f32(float x) {
  return __uint_as_float(wave_last(wave_scan_bits(__float_as_uint(x), 0x7f800000u, [](uint32_t a, uint32_t b) {
    return __float_as_uint(fminf(__uint_as_float(a), __uint_as_float(b)));
  })));
}
__device__ __forceinline__ float wave_max_f32(float x) {
  return __uint_as_float(wave_last(wave_scan_bits(__float_as_uint(x), 0xff800000u, [](uint32_t a, uint32_t b) {
    return __float_as_uint(fmaxf(__uint_as_float(a), __uint_as_float(b)));
  })));
}

// Inclusive scan of one int per thread over the kThreads threads of the block, in thread order.
__device__ __forceinline__ int block_incl_scan(int x, int* wave_tot, int* total) {
  const int lane = lane_id(), w = threadIdx.x >> 6;
  x = wave_incl_sum(x);
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

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x) {
  return wave_last(wave_scan_bits(x, 0xffffffffu, [](uint32_t a, uint32_t b) { return min(a, b); }));
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
  return wave_last(wave_scan_bits(x, 0u, [](uint32_t a, uint32_t b) { return max(a, b); }));
}

constexpr int kRegKeys = kMaxLdsKeys / kThreads;    // 32 pages per thread held in registers

// Options of the radix selection beyond the exact one (Sec. 5.2 approximate top-k):
//   remap 1: keys are the affine map of the candidates' [min, max] onto 32-bit fixed point,
//            floor((s - min) * scale), scale = 4294967295 / (max - min) in fp64;
//   tau_q:   tolerate ratio in 16-bit fixed point; after a pass with key bits left, refinement
//            stops once certain * 65536 >= (65536 - tau_q) * K_free members lie in higher bins,
//            and the rest is a random sample of the threshold bin: its members ordered by the
//            8-bit hash h8(j) = lowbias32(z ^ j) >> 24, larger first, equal hashes by page,
//            z = lowbias32(seed ^ lowbias32(i * H + h)).  One more radix pass, over h8 instead
//            of the next key digit, finds the hash threshold.
// remap 0 and tau_q 0 is the exact selection.
struct TopkOptions {
  int remap, tau_q;
  uint32_t seed;
};

__device__ __forceinline__ uint32_t lowbias32(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}

// Block-wide min and max of one float per thread (NaN-free inputs; +inf/-inf when empty).
__device__ __forceinline__ void block_fminmax(float& mn, float& mx, float (*wave_fm)[kThreads / kWave]) {
  const int lane = lane_id(), w = threadIdx.x >> 6;
  mn = wave_min_f32(mn);
  mx = wave_max_f32(mx);
  if (lane == 0) {
    wave_fm[0][w] = mn;
    wave_fm[1][w] = mx;
  }
  __syncthreads();
#pragma unroll
  for (int x = 0; x < kThreads / kWave; x++) {
    mn = fminf(mn, wave_fm[0][x]);
    mx = fmaxf(mx, wave_fm[1][x]);
  }
}

// items == nullptr: the request's page count from seq_lens and the page list; else items[i]
// (capped at the row stride).
//
// Thread t owns the contiguous pages [t*R, t*R + R), R = ceil(P / kThreads).  Up to
// kMaxLdsKeys pages (R <= 32) their keys stay in registers for every radix pass and for the
// compaction; longer rows recompute the keys from the scores (L2-resident after the first read).
__global__ __launch_bounds__(kThreads) void topk_kernel(
    const float* __restrict__ scores, int H, int ps, int r, int max_pages, int stride, int batch,
    const int32_t* __restrict__ indptr, const int32_t* __restrict__ seq_lens, const int32_t* __restrict__ items,
    const int32_t* __restrict__ budget, int n_sink, int n_local, int max_sel, const TopkOptions opt,
    int32_t* __restrict__ sel_pages, int32_t* __restrict__ sel_count) {
  __shared__ int hist[2][256];
  __shared__ int wave_tot[kThreads / kWave];
  __shared__ uint32_t wave_mm[2][kThreads / kWave];
  __shared__ float wave_fm[2][kThreads / kWave];
  __shared__ int pick[2][3];           // digit, count above the digit's bin, bin count

  const int tid = threadIdx.x, lane = lane_id(), w = tid >> 6;
  const int i = blockIdx.x / H, h = blockIdx.x % H;
  const int P = items ? min(max(items[i], 0), stride)
                      : num_pages(seq_lens[i], ps, (indptr[i + 1] - indptr[i]) * r, max_pages);
  int Ktot = budget[i];
  Ktot = Ktot < max_sel ? Ktot : max_sel;
  Ktot = Ktot < 0 ? 0 : Ktot;
  const float* s = scores + ((int64_t)h * batch + i) * stride;
  int32_t* out = sel_pages + ((int64_t)i * H + h) * max_sel;

  const bool all = Ktot >= P;
  const int nS = min(n_sink, P), nL = min(n_local, P);
  const int nF = all ? P : nS + nL - max(0, nS - (P - nL));
  const int Kfree = all ? 0 : max(0, Ktot - nF);
  const int R = (P + kThreads - 1) / kThreads;
  const int j_lo = min(P, tid * R), n_mine = min(P, j_lo + R) - j_lo;
  const bool in_regs = R <= kRegKeys;

  // scores of the own range (registers), and the candidate mask (bit x: page j_lo + x)
  float sv[kRegKeys];
  uint32_t kr[kRegKeys], cand = 0;
  if (Kfree > 0 && in_regs) {
#pragma unroll
    for (int x = 0; x < kRegKeys; x++) {
      if (x < R) sv[x] = s[x < n_mine ? j_lo + x : 0];     // all loads issued before any use
    }
#pragma unroll
    for (int x = 0; x < kRegKeys; x++)
      if (x < n_mine && !is_forced(j_lo + x, P, nS, nL)) cand |= 1u << x;
  }

  double rmin = 0.0, rscale = 0.0;                       // remap 1: min and scale of the affine map
  auto make_key = [&](float x) -> uint32_t {
    if (opt.remap == 0) return float_key(x);
    if (x != x) return 0u;
    // in [0, 2^32 - 1] for candidates; forced pages (never ranked) may fall outside: clamp
    return (uint32_t)fmin(fmax(floor(((double)x - rmin) * rscale), 0.0), 4294967295.0);
  };
  // f(key) for every candidate of this thread
  auto each_candidate = [&](auto&& f) {
    if (in_regs) {
#pragma unroll
      for (int x = 0; x < kRegKeys; x++)
        if ((cand >> x) & 1u) f(kr[x]);
    } else {
      for (int j = j_lo; j < j_lo + n_mine; j++)
        if (!is_forced(j, P, nS, nL)) f(make_key(s[j]));
    }
  };
  // f(j, key) for every candidate of this thread
  auto each_candidate_j = [&](auto&& f) {
    if (in_regs) {
#pragma unroll
      for (int x = 0; x < kRegKeys; x++)
        if ((cand >> x) & 1u) f(j_lo + x, kr[x]);
    } else {
      for (int j = j_lo; j < j_lo + n_mine; j++)
        if (!is_forced(j, P, nS, nL)) f(j, make_key(s[j]));
    }
  };
  // f(j, key) for every page of this thread in ascending order (key meaningful for candidates)
  auto each_own = [&](auto&& f) {
    if (in_regs) {
#pragma unroll
      for (int x = 0; x < kRegKeys; x++)
        if (x < n_mine) f(j_lo + x, kr[x]);
    } else {
      for (int j = j_lo; j < j_lo + n_mine; j++) f(j, Kfree > 0 ? make_key(s[j]) : 0u);
    }
  };

  // Radix select over the candidates' keys.  Threshold prefix: a candidate is chosen when
  // (key & pmask) > prefix, or when it equals the prefix and its rank among equals (by page
  // index; after an early stop by (h8 desc, page)) is below `remaining`.
  uint32_t prefix = 0, pmask = 0;
  int remaining = Kfree;
  int hthr = -1;                                         // stopped early: hash threshold h8
  uint32_t hz = 0;                                       // hash salt z of this (request, head)
  // Wave 0 finds the bin of histogram hb holding the remaining-th largest digit (lane l owns
  // bins 255-4l .. 252-4l, descending): pick[hb] = {bin, count above it, bin count}.
  auto pick_bin = [&](int hb) {
    if (w == 0) {
      int c[4], tot = 0;
#pragma unroll
      for (int e = 0; e < 4; e++) {
        c[e] = hist[hb][255 - 4 * lane - e];
        tot += c[e];
      }
      int above = wave_incl_sum(tot) - tot;
#pragma unroll
      for (int e = 0; e < 4; e++) {
        if (above < remaining && above + c[e] >= remaining) {
          pick[hb][0] = 255 - 4 * lane - e;
          pick[hb][1] = above;
          pick[hb][2] = c[e];
        }
        above += c[e];
      }
    }
    __syncthreads();
  };
  if (Kfree > 0) {
    if (opt.remap != 0) {
      // the candidates' score range (NaN excluded) fixes the affine map
      float fmn = INFINITY, fmx = -INFINITY;
      if (in_regs) {
#pragma unroll
        for (int x = 0; x < kRegKeys; x++) {
          if (((cand >> x) & 1u) && sv[x] == sv[x]) {
            fmn = fminf(fmn, sv[x]);
            fmx = fmaxf(fmx, sv[x]);
          }
        }
      } else {
        for (int j = j_lo; j < j_lo + n_mine; j++) {
          const float x = s[j];
          if (!is_forced(j, P, nS, nL) && x == x) {
            fmn = fminf(fmn, x);
            fmx = fmaxf(fmx, x);
          }
        }
      }
      block_fminmax(fmn, fmx, wave_fm);
      rmin = (double)fmn;
      rscale = fmx > fmn ? 4294967295.0 / ((double)fmx - (double)fmn) : 0.0;
    }
    if (in_regs) {
#pragma unroll
      for (int x = 0; x < kRegKeys; x++) kr[x] = x < n_mine ? make_key(sv[x]) : 0u;
    }
    // bits above the highest bit where the smallest and largest candidate key differ are
    // common to every candidate and need no pass
    uint32_t kmin = 0xffffffffu, kmax = 0u;
    each_candidate([&](uint32_t key) {
      kmin = min(kmin, key);
      kmax = max(kmax, key);
    });
    kmin = wave_min_u32(kmin);
    kmax = wave_max_u32(kmax);
    if (lane == 0) {
      wave_mm[0][w] = kmin;
      wave_mm[1][w] = kmax;
    }
    hist[0][tid] = 0;
    __syncthreads();
#pragma unroll
    for (int x = 0; x < kThreads / kWave; x++) {
      kmin = min(kmin, wave_mm[0][x]);
      kmax = max(kmax, wave_mm[1][x]);
    }
    const uint32_t diff = kmin ^ kmax;
    int top = diff ? 31 - __clz((int)diff) : -1;           // highest differing bit
    pmask = top >= 31 ? 0u : ~((2u << top) - 1u);           // common high bits
    if (top < 0) pmask = 0xffffffffu;                        // all candidate keys equal
    prefix = kmin & pmask;

    int hb = 0, certain = 0;
    while (top >= 0) {
      const int shift = top >= 7 ? top - 7 : 0;
      const uint32_t dmask = (1u << (top - shift + 1)) - 1u;   // 1..8 bits
      hist[hb ^ 1][tid] = 0;                                   // next pass's histogram
      each_candidate([&](uint32_t key) {
        if ((key & pmask) == prefix) atomicAdd(&hist[hb][(key >> shift) & dmask], 1);
      });
      __syncthreads();
      pick_bin(hb);
      remaining -= pick[hb][1];
      certain += pick[hb][1];
      prefix |= (uint32_t)pick[hb][0] << shift;
      pmask |= dmask << shift;
      const bool done = pick[hb][2] == remaining;   // every key with this prefix is chosen
      top = shift - 1;
      hb ^= 1;
      if (done) break;
      if (top >= 0 && (int64_t)certain * 65536 >= (int64_t)(65536 - opt.tau_q) * Kfree) {
        // early termination: one pass over the threshold bin's hashes (histogram hb was
        // cleared during the last pass) orders the rest at random
        hz = lowbias32(opt.seed ^ lowbias32((uint32_t)(i * H + h)));
        each_candidate_j([&](int j, uint32_t key) {
          if ((key & pmask) == prefix) atomicAdd(&hist[hb][lowbias32(hz ^ (uint32_t)j) >> 24], 1);
        });
        __syncthreads();
        pick_bin(hb);
        remaining -= pick[hb][1];
        hthr = pick[hb][0];
        break;
      }
    }
  }

  // Compaction: one scan gives each tied candidate its rank by page index, a second gives each
  // chosen page its slot.
  // After an early stop a bin member ranks above the tie class by its hash, else ties.
  auto hash_cmp = [&](int j) -> int {
    if (hthr < 0) return 0;
    const int hv = (int)(lowbias32(hz ^ (uint32_t)j) >> 24);
    return (hv > hthr) - (hv < hthr);
  };
  int n_eq = 0;
  if (Kfree > 0) {
    each_candidate_j([&](int j, uint32_t key) { n_eq += (key & pmask) == prefix && hash_cmp(j) == 0; });
  }
  int tot_eq;
  const int eq_rank = block_incl_scan(n_eq, wave_tot, &tot_eq) - n_eq;
  // the tie class's chosen members are its `remaining` lowest page indices
  auto chosen_at = [&](int j, uint32_t key, int& r) -> bool {
    if (all || is_forced(j, P, nS, nL)) return true;
    if (Kfree <= 0) return false;
    const uint32_t mk = key & pmask;
    if (mk != prefix) return mk > prefix;
    const int hc = hash_cmp(j);
    if (hc != 0) return hc > 0;
    const bool in = r < remaining;
    r++;
    return in;
  };
  int n_chosen = 0;
  {
    int r = eq_rank;
    each_own([&](int j, uint32_t key) { n_chosen += chosen_at(j, key, r); });
  }
  int tot_sel;
  int pos = block_incl_scan(n_chosen, wave_tot, &tot_sel) - n_chosen;
  {
    int r = eq_rank;
    each_own([&](int j, uint32_t key) {
      if (chosen_at(j, key, r)) {
        if (pos < max_sel) out[pos] = j;
        pos++;
      }
    });
  }
  for (int m = tot_sel + tid; m < max_sel; m += kThreads) out[m] = -1;
  if (h == 0 && tid == 0) sel_count[i] = min(tot_sel, max_sel);
}

// ------------------------------------------------------------------------------------
// Two-pass selection for the block-mean score (first pass: kMeanBound).  For each
// (request, KV head), with K = K_free and B a monotone bucket map of the bounds:
//   T_lo = K-th largest B(lower), T_hi = (K+1)-th largest B(upper) (over candidates);
//   B(upper) < T_lo  -> out: K candidates score strictly higher (their fp32 keys too);
//   B(lower) > T_hi  -> in:  at most K candidates, itself included, can score >= it;
//   otherwise undecided: re-scored from the fp32 Mean with exact_row_score (the one-pass
//   arithmetic); the best K - |in| of them by (score desc, page asc) complete the set.
// Both thresholds come out of one radix walk (two histograms per pass).  Every load of the
// prologue (both bounds of every page and the group's query rows) is issued before any is
// used, and the keys stay in registers.
// ------------------------------------------------------------------------------------
constexpr int kFusedAppendMaxElems = 8192;  // block rows x channels refreshed in the top-K launch
constexpr int kTwoPassKeys = 4096;     // = kTwoPassMaxPages
constexpr int kRounds2 = kTwoPassKeys / (4 * kThreads);  // float4 rounds per thread
constexpr int kPerThread2 = 4 * kRounds2;                  // 16 pages per thread
constexpr int kMaxUndecided = 1024;

// Page of this thread's key slot x: four consecutive pages per float4 round, rounds 4*kThreads
// pages apart.
__device__ __forceinline__ int slot_page(int x) { return 4 * (int)threadIdx.x + (x & 3) + 4 * kThreads * (x >> 2); }

// Both bound rows of N rounds, every load issued before any is used.  Slots past the
// request's pages re-read its last float4 (never used), so no row padding is fetched.
template <int N, bool BOTH>
__device__ __forceinline__ void load_bounds(const float* lo, const float* up, int P, float4 (&lv)[kRounds2],
                                            float4 (&uv)[kRounds2]) {
  const int last4 = ((P + 3) & ~3) - 4;           // P >= 1; the row stride is a multiple of 4 >= P
#pragma unroll
  for (int y = 0; y < N; y++) {
    const int j = min(4 * (int)threadIdx.x + 4 * kThreads * y, last4);
    lv[y] = *reinterpret_cast<const float4*>(lo + j);
    if constexpr (BOTH) uv[y] = *reinterpret_cast<const float4*>(up + j);
  }
}

struct RadixState {
  uint32_t prefix, pmask;   // resolved high bits of the k-th largest key
  int top;                  // highest unresolved bit, -1 when done
  int remaining;            // rank of the target among keys that share the prefix
};

// Start from the candidates' smallest and largest keys: bits above the highest differing bit
// are common to every candidate.
__device__ __forceinline__ RadixState radix_init(uint32_t kmin, uint32_t kmax, int k) {
  RadixState r;
  const uint32_t diff = kmin ^ kmax;
  r.top = diff ? 31 - __clz((int)diff) : -1;
  r.pmask = r.top < 0 ? 0xffffffffu : (r.top >= 31 ? 0u : ~((2u << r.top) - 1u));
  r.prefix = kmin & r.pmask;
  r.remaining = k;
  return r;
}
__device__ __forceinline__ int radix_shift(const RadixState& r) { return r.top >= 7 ? r.top - 7 : 0; }
__device__ __forceinline__ uint32_t radix_dmask(const RadixState& r) {
  return r.top >= 0 ? (1u << (r.top - radix_shift(r) + 1)) - 1u : 0u;
}

// One wave: lane l owns the bins 255-4l .. 252-4l (descending).  Writes the bin that holds the
// remaining-th largest key and the number of keys in the bins above it.
__device__ __forceinline__ void wave_pick_bin(const int* hist, int remaining, int* pick) {
  const int lane = lane_id();
  int c[4], tot = 0;
#pragma unroll
  for (int e = 0; e < 4; e++) {
    c[e] = hist[255 - 4 * lane - e];
    tot += c[e];
  }
  int above = wave_incl_sum(tot) - tot;
#pragma unroll
  for (int e = 0; e < 4; e++) {
    if (above < remaining && above + c[e] >= remaining) {
      pick[0] = 255 - 4 * lane - e;
      pick[1] = above;
    }
    above += c[e];
  }
}

__device__ __forceinline__ void radix_advance(RadixState& r, const int* pick) {
  const int sh = radix_shift(r);
  r.remaining -= pick[1];
  r.prefix |= (uint32_t)pick[0] << sh;
  r.pmask |= radix_dmask(r) << sh;
  r.top = sh - 1;
}

// The k-th largest keys of two key sets held in registers (key x of this thread counts when
// bit x of `cand` is set); both selects share each pass and its barriers.  sb.top < 0 on
// entry runs the first select alone.
__device__ __forceinline__ void dual_radix_select(const uint32_t (&ka)[kPerThread2], const uint32_t (&kb)[kPerThread2],
                                                  uint32_t cand, RadixState& sa, RadixState& sb,
                                                  int (*hist)[2][256], int (*pick)[2][2]) {
  const int tid = threadIdx.x, w = tid >> 6;
  int hb = 0;
  hist[0][0][tid] = 0;
  hist[0][1][tid] = 0;
  __syncthreads();
  while (sa.top >= 0 || sb.top >= 0) {
    const int sha = radix_shift(sa), shb = radix_shift(sb);
    const uint32_t dma = radix_dmask(sa), dmb = radix_dmask(sb);
    hist[hb ^ 1][0][tid] = 0;
    hist[hb ^ 1][1][tid] = 0;
#pragma unroll
    for (int x = 0; x < kPerThread2; x++) {
      if ((cand >> x) & 1u) {
        if (sa.top >= 0 && (ka[x] & sa.pmask) == sa.prefix) atomicAdd(&hist[hb][0][(ka[x] >> sha) & dma], 1);
        if (sb.top >= 0 && (kb[x] & sb.pmask) == sb.prefix) atomicAdd(&hist[hb][1][(kb[x] >> shb) & dmb], 1);
      }
    }
    __syncthreads();
    if (w == 0 && sa.top >= 0) wave_pick_bin(hist[hb][0], sa.remaining, pick[hb][0]);
    if (w == 1 && sb.top >= 0) wave_pick_bin(hist[hb][1], sb.remaining, pick[hb][1]);
    __syncthreads();
    if (sa.top >= 0) radix_advance(sa, pick[hb][0]);
    if (sb.top >= 0) radix_advance(sb, pick[hb][1]);
    hb ^= 1;
  }
}

// The decode step's append inside the selection launch: the workgroup of (request i, KV head h)
// writes the step's K/V rows of head h at token L - 1 and refreshes that block's summaries with
// the cache stage's own task code (4 lanes per 8-channel task, as in the decode-step summary
// launch), so the cache and the summaries are bit-identical to a separate append.  The block is
// request i's last one, a forced local block, so the selection never reads its new summary.
struct AppendStep {
  summ::AppendArgs app;      // app.knew == nullptr: nothing to append
  const void* k;             // the K cache (read)
  float k_scale;
  int kt, ps, D, num_phys;
  int wgs;                   // one-wave selection launch: 0, the selection workgroup appends its
                             // head; > 0, this many workgroups per request past the selection's
                             // append all of the request's heads
  int max_pages;             // blocks per request bound
  float* mean;
  uint16_t* mean_bf;
  uint16_t* maxo;
  uint16_t* mino;
};
template <int KT, int NT>
__device__ __forceinline__ void append_head_kt(const AppendStep& ap, int i, int h, int H, int bs, int r, int base,
                                               int L, const int32_t* __restrict__ indices) {
  const int chunks = ap.D / 8, j = (L - 1) / bs, slice = (int)threadIdx.x & 3;
  for (int t0 = 0; t0 < chunks; t0 += NT / 4) {             // uniform: full quads
    const int c8 = t0 + (int)threadIdx.x / 4;
    const bool active = c8 < chunks;
    summ::task<4, KT, true>(ap.k, ap.k_scale, ap.num_phys, H, ap.ps, bs, r, ap.D, indices, base, L, i, j, h,
                            active ? c8 : 0, active, slice, ap.mean, ap.mean_bf, ap.maxo, ap.mino, ap.app);
  }
}
// NT: the workgroup's thread count.  P: the request's block count; a request whose token L - 1
// lies in no listed block (L = 0, a short page list) appends nothing, as in the cache stage's
// own append launch.
template <int NT = kThreads>
__device__ __forceinline__ void append_head(const AppendStep& ap, int i, int h, int H, int bs, int r, int base, int L,
                                            int P, const int32_t* __restrict__ indices) {
  if (L < 1 || (L - 1) / bs >= P) return;
  if (ap.kt == kKvFp8E4M3) append_head_kt<kKvFp8E4M3, NT>(ap, i, h, H, bs, r, base, L, indices);
  else if (ap.kt == kKvFp8E5M2) append_head_kt<kKvFp8E5M2, NT>(ap, i, h, H, bs, r, base, L, indices);
  else append_head_kt<kKvBf16, NT>(ap, i, h, H, bs, r, base, L, indices);
}

// The one-wave selection launch's append workgroups (blocks of more than kFusedAppendMaxElems
// elements): ap.wgs workgroups per request share the tasks (KV head, 8-channel chunk) of the
// request's block L - 1, kWave / 4 tasks each, with the cache stage's task code and load batch,
// so the summaries are bit-identical to its append launch.
template <int KT, int KB>
__device__ __forceinline__ void append_spread_kt(const AppendStep& ap, int a, int H, int bs, int r,
                                                 const int32_t* __restrict__ indptr,
                                                 const int32_t* __restrict__ indices,
                                                 const int32_t* __restrict__ seq_lens) {
  const int i = a / ap.wgs;
  const int L = seq_lens[i], base = indptr[i];
  const int P = num_pages(L, bs, (indptr[i + 1] - base) * r, ap.max_pages);
  if (L < 1 || (L - 1) / bs >= P) return;
  const int chunks = ap.D / 8;
  const int t = (a - i * ap.wgs) * (kWave / 4) + (int)threadIdx.x / 4;   // the same for a quad's lanes
  const bool active = t < H * chunks;
  const int tk = active ? t : 0, h = tk / chunks;
  summ::task<4, KT, true, KB>(ap.k, ap.k_scale, ap.num_phys, H, ap.ps, bs, r, ap.D, indices, base, L, i,
                              (L - 1) / bs, h, tk - h * chunks, active, (int)threadIdx.x & 3, ap.mean, ap.mean_bf,
                              ap.maxo, ap.mino, ap.app);
}
__device__ __forceinline__ void append_spread(const AppendStep& ap, int a, int H, int bs, int r,
                                              const int32_t* __restrict__ indptr, const int32_t* __restrict__ indices,
                                              const int32_t* __restrict__ seq_lens) {
  // blocks of 64 tokens: a lane's 16 rows in one round trip, as in the append launch
  if (bs > 4 * summ::kBatch) {
    if (ap.kt == kKvFp8E4M3) append_spread_kt<kKvFp8E4M3, 2 * summ::kBatch>(ap, a, H, bs, r, indptr, indices, seq_lens);
    else if (ap.kt == kKvFp8E5M2) append_spread_kt<kKvFp8E5M2, 2 * summ::kBatch>(ap, a, H, bs, r, indptr, indices, seq_lens);
    else append_spread_kt<kKvBf16, 2 * summ::kBatch>(ap, a, H, bs, r, indptr, indices, seq_lens);
  } else {
    if (ap.kt == kKvFp8E4M3) append_spread_kt<kKvFp8E4M3, summ::kBatch>(ap, a, H, bs, r, indptr, indices, seq_lens);
    else if (ap.kt == kKvFp8E5M2) append_spread_kt<kKvFp8E5M2, summ::kBatch>(ap, a, H, bs, r, indptr, indices, seq_lens);
    else append_spread_kt<kKvBf16, summ::kBatch>(ap, a, H, bs, r, indptr, indices, seq_lens);
  }
}

// RK = kMeanDot: the two-pass block-mean selection (bounds in, fp32 Mean rows of D channels for
// the re-scoring).  RK = an envelope kind: the two-pass selection of that kind (bounds in, bf16
// Max and Min rows of D channels for the re-scoring, g <= 4).  RK = kNoRescore: exact scores
// (lower == upper == the scores); the pages of the threshold buckets are ranked by their own
// scores and nothing is re-scored.
template <int RK, int D>
__global__ __launch_bounds__(kThreads) void topk_bucket_kernel(
    const float* __restrict__ lower, const float* __restrict__ upper, const float* __restrict__ mean,
    const uint16_t* __restrict__ maxs, const uint16_t* __restrict__ mins, const uint16_t* __restrict__ q, int Hq,
    int H, int qdims, int ps, int r, int max_pages, int stride, int batch, int num_phys,
    const int32_t* __restrict__ indptr, const int32_t* __restrict__ indices, const int32_t* __restrict__ seq_lens,
    const int32_t* __restrict__ budget, int n_sink, int n_local, int max_sel, int32_t* __restrict__ sel_pages,
    int32_t* __restrict__ sel_count, const AppendStep ap) {
  constexpr bool kMeanRescore = RK == kMeanDot;
  constexpr bool kEnvRescore = is_env(RK);
  constexpr bool kRescore = kMeanRescore || kEnvRescore;
  constexpr int DD = kRescore ? D : 64;                      // shapes of the unused re-scoring parts
  using M = RowMap<DD, false>;                               // fp32 Mean rows
  using ME = RowMap<DD, true>;                               // bf16 Max / Min rows
  constexpr int E = DD / 16;
  // 16-byte query chunks of a group: g <= 16 heads (block mean), g <= 4 (envelope kinds)
  constexpr int kQChunks = kMeanRescore ? 16 * D / 8 : kEnvRescore ? 4 * D / 8 : 1;
  constexpr int kQRounds = (kQChunks + kThreads - 1) / kThreads;
  __shared__ uint32_t exact_keys[kTwoPassKeys];   // only after a bound overflow
  __shared__ __align__(16) uint8_t status[kTwoPassKeys];   // 0 out, 1 chosen, 2 undecided
  __shared__ int und[kMaxUndecided];              // undecided pages
  __shared__ uint32_t und_key[kMaxUndecided];     // their exact keys
  __shared__ uint4 qraw[kMeanRescore ? kQChunks : 1];   // the group's bf16 query rows
  __shared__ double qbar[kMeanRescore ? D : 1];   // group-mean query, channel order
  __shared__ float qs[kEnvRescore ? 4 * D : 1];   // the group's query rows, fp32 in row order
  __shared__ int hist[2][2][256];
  __shared__ int pick[2][2][2];
  __shared__ uint32_t mm[4][kThreads / kWave];
  __shared__ int wave_tot[kThreads / kWave];
  __shared__ int counters[2];                     // |in|, |undecided|

  const int tid = threadIdx.x, lane = lane_id(), w = tid >> 6;
  const int i = blockIdx.x / H, h = blockIdx.x % H;
  const int base = indptr[i];
  const int P = num_pages(seq_lens[i], ps, (indptr[i + 1] - base) * r, min(max_pages, kTwoPassKeys));
  if (ap.app.knew) append_head(ap, i, h, H, ps, r, base, seq_lens[i], P, indices);
  int Ktot = budget[i];
  Ktot = Ktot < max_sel ? Ktot : max_sel;
  Ktot = Ktot < 0 ? 0 : Ktot;
  int32_t* out = sel_pages + ((int64_t)i * H + h) * max_sel;
  const bool all = Ktot >= P;
  const int nS = min(n_sink, P), nL = min(n_local, P);
  const int nF = all ? P : nS + nL - max(0, nS - (P - nL));
  const int Kfree = all ? 0 : max(0, Ktot - nF);
  const int g = Hq / H;

  for (int j = tid; j < P; j += kThreads) status[j] = (all || is_forced(j, P, nS, nL)) ? 1 : 0;
  if (tid < 2) counters[tid] = 0;
  int need = 0, n_und = 0;
  bool rescore_all = false;
  uint32_t cand = 0;                               // bit x: slot_page(x) is a candidate
  if (Kfree > 0) {
    // every prologue load in one round trip: both bound rows and the group's query rows
    const float* lo = lower + ((int64_t)h * batch + i) * stride;
    const float* up = upper + ((int64_t)h * batch + i) * stride;
    float4 lv[kRounds2], uv[kRounds2];
    const int rounds = (P + 4 * kThreads - 1) / (4 * kThreads);
    if (rounds <= 1) load_bounds<1, kRescore>(lo, up, P, lv, uv);
    else if (rounds <= 2) load_bounds<2, kRescore>(lo, up, P, lv, uv);
    else load_bounds<kRounds2, kRescore>(lo, up, P, lv, uv);
    if constexpr (!kRescore) {
#pragma unroll
      for (int y = 0; y < kRounds2; y++) uv[y] = lv[y];
    }
    const int nq = g * DD / 8;
    uint4 qv[kQRounds];
    if constexpr (kRescore) {
      const uint4* qsrc = reinterpret_cast<const uint4*>(q + ((int64_t)i * Hq + (int64_t)h * g) * D);
#pragma unroll
      for (int t = 0; t < kQRounds; t++) qv[t] = qsrc[min(tid + kThreads * t, nq - 1)];
    }

    // Bucket keys: B(x) = floor((x - lo) * 65535 / (hi - lo)), clamped to [0, 65535], with lo
    // the smallest candidate lower bound and hi the largest upper bound.  B is monotone
    // (non-decreasing) in x, so the classification below is as rigorous on buckets as on
    // the floats themselves, and 16-bit keys spread over their range need only two passes.
    float lf[kPerThread2], uf[kPerThread2];
    float lo_min = INFINITY, hi_max = -INFINITY;
#pragma unroll
    for (int x = 0; x < kPerThread2; x++) {
      const int j = slot_page(x);
      const float4 l4 = lv[x >> 2], u4 = uv[x >> 2];
      lf[x] = (x & 3) == 0 ? l4.x : (x & 3) == 1 ? l4.y : (x & 3) == 2 ? l4.z : l4.w;
      uf[x] = (x & 3) == 0 ? u4.x : (x & 3) == 1 ? u4.y : (x & 3) == 2 ? u4.z : u4.w;
      if ((x >> 2) < rounds && j < P && !is_forced(j, P, nS, nL)) {
        cand |= 1u << x;
        lo_min = fminf(lo_min, lf[x]);
        hi_max = fmaxf(hi_max, uf[x]);
      }
    }
    if constexpr (kMeanRescore) {
#pragma unroll
      for (int t = 0; t < kQRounds; t++)
        if (tid + kThreads * t < nq) qraw[tid + kThreads * t] = qv[t];
    } else if constexpr (kEnvRescore) {
      // the envelope scores' query layout: head r, channel c at (r 16 + u) E + e, c the RowMap
      // channel (u, cc, e)
#pragma unroll
      for (int t = 0; t < kQRounds; t++) {
        const int x = tid + kThreads * t;
        if (x < nq) {
          const uint32_t ws[4] = {qv[t].x, qv[t].y, qv[t].z, qv[t].w};
#pragma unroll
          for (int k = 0; k < 8; k++) {
            const int flat = 8 * x + k, rr = flat / D, c = flat - rr * D;
            const int chunk = c / ME::kElemsPerChunk, e_in = c - chunk * ME::kElemsPerChunk;
            qs[(rr * 16 + chunk % 16) * E + (chunk / 16) * ME::kElemsPerChunk + e_in] =
                (k & 1) ? bf16hi(ws[k >> 1]) : bf16lo(ws[k >> 1]);
          }
        }
      }
    }
    lo_min = wave_min_f32(lo_min);
    hi_max = wave_max_f32(hi_max);
    if (lane == 0) {
      mm[0][w] = __float_as_uint(lo_min);
      mm[1][w] = __float_as_uint(hi_max);
    }
    __syncthreads();
#pragma unroll
    for (int x = 0; x < kThreads / kWave; x++) {
      lo_min = fminf(lo_min, __uint_as_float(mm[0][x]));
      hi_max = fmaxf(hi_max, __uint_as_float(mm[1][x]));
    }
    const float span = hi_max - lo_min;
    const float scale = (span > 0.f && span < INFINITY) ? 65535.f / span : 0.f;
    uint32_t kl[kPerThread2], ku[kPerThread2];
#pragma unroll
    for (int x = 0; x < kPerThread2; x++) {
      kl[x] = (uint32_t)(int)fminf(fmaxf((lf[x] - lo_min) * scale, 0.f), 65535.f);
      ku[x] = (uint32_t)(int)fminf(fmaxf((uf[x] - lo_min) * scale, 0.f), 65535.f);
    }
    if constexpr (kMeanRescore) {
      // group-mean query: fp64 sums in head order, then finish_qbar's division (as one pass)
      const uint16_t* qh = reinterpret_cast<const uint16_t*>(qraw);
      for (int c = tid; c < D; c += kThreads) {
        double acc = 0.0;
        for (int r = 0; r < g; r++) acc += (double)bf16lo(qh[r * D + c]);
        qbar[c] = c < qdims ? finish_qbar_one(acc, g) : 0.0;
      }
    }
    RadixState sl = radix_init(0u, 0xffffu, Kfree), su = radix_init(0u, 0xffffu, Kfree + 1);
    dual_radix_select(kl, ku, cand, sl, su, hist, pick);
    const uint32_t t_lo = sl.prefix;                 // bucket of the K-th largest lower bound
    const uint32_t t_hi = su.prefix;                 // bucket of the (K+1)-th largest upper bound
    // each round's four consecutive pages in one 32-bit status store (forced pages stay chosen);
    // the chosen count and the undecided list grow by one atomic per wave
    int my_in = 0;
    uint32_t und_bits = 0;                           // bit x: slot_page(x) is undecided
    uint32_t word[kRounds2] = {};
#pragma unroll
    for (int x = 0; x < kPerThread2; x++) {
      const int j = slot_page(x);
      uint32_t st = (j < P && is_forced(j, P, nS, nL)) ? 1u : 0u;
      if ((cand >> x) & 1u) {
        if (kl[x] > t_hi) {
          st = 1u;
          my_in++;
        } else if (ku[x] >= t_lo) {
          st = 2u;
          und_bits |= 1u << x;
        }
      }
      word[x >> 2] |= st << (8 * (x & 3));
    }
#pragma unroll
    for (int y = 0; y < kRounds2; y++)
      if (y < rounds) *reinterpret_cast<uint32_t*>(&status[4 * tid + 4 * kThreads * y]) = word[y];
    my_in = (int)wave_last((uint32_t)wave_incl_sum(my_in));
    if (lane == 0 && my_in) atomicAdd(&counters[0], my_in);
    const int n_mine = __popc(und_bits);
    const int und_incl = wave_incl_sum(n_mine);
    const int und_wave = (int)wave_last((uint32_t)und_incl);
    int und_base = 0;
    if (lane == kWave - 1 && und_wave) und_base = atomicAdd(&counters[1], und_wave);
    int pos = __builtin_amdgcn_readlane(und_base, kWave - 1) + und_incl - n_mine;
    while (und_bits) {
      const int x = __builtin_ctz(und_bits);
      und_bits &= und_bits - 1u;
      const int j = slot_page(x);
      float lx = 0.f;
#pragma unroll
      for (int z = 0; z < kPerThread2; z++) lx = z == x ? lf[z] : lx;   // lf[x] without a dynamic index
      if constexpr (!kRescore) exact_keys[j] = float_key(lx);           // the exact score
      if (pos < kMaxUndecided) {
        und[pos] = j;
        if constexpr (!kRescore) und_key[pos] = float_key(lx);
      }
      pos++;
    }
    __syncthreads();
    need = Kfree - counters[0];
    n_und = counters[1];
    rescore_all = n_und > kMaxUndecided;
    if (rescore_all) {
      // pathological overlap of the bounds: re-score every candidate instead
#pragma unroll
      for (int x = 0; x < kPerThread2; x++) {
        if ((cand >> x) & 1u) {
          status[slot_page(x)] = 2;
          if constexpr (!kRescore) exact_keys[slot_page(x)] = float_key(lf[x]);
        }
      }
      need = Kfree;
      __syncthreads();
    }
  }

  // exact scores of the undecided pages: rows of 16 lanes, two pages per row at a time
  const int n_score = rescore_all ? P : n_und;
  if (need > 0) {
    if constexpr (kRescore) {
    const int row = tid >> 4, u = tid & 15;
    double qb[kMeanRescore ? E : 1];
    if constexpr (kMeanRescore) {
#pragma unroll
      for (int c = 0; c < M::kChunks; c++)
#pragma unroll
        for (int e = 0; e < 4; e++) qb[4 * c + e] = qbar[M::channel(u, c, e)];
    }
    for (int x0 = row; x0 < n_score; x0 += 2 * kRows) {
      const int x1 = x0 + kRows;
      const bool has1 = x1 < n_score;
      const int j0 = rescore_all ? x0 : und[x0];
      const int j1 = has1 ? (rescore_all ? x1 : und[x1]) : j0;
      const int64_t p0 = block_row(indices + base, j0, r, num_phys);
      const int64_t p1 = block_row(indices + base, j1, r, num_phys);
      float s0, s1;
      if constexpr (kMeanRescore) {
        uint32_t w0[RowWords<DD, false>::W], w1[RowWords<DD, false>::W];
        load_row_words<DD, false>(mean + (p0 * H + h) * D, u, w0);
        load_row_words<DD, false>(mean + (p1 * H + h) * D, u, w1);
        s0 = exact_row_score<DD, false>(qb, w0);
        s1 = exact_row_score<DD, false>(qb, w1);
      } else {
        constexpr int W = RowWords<DD, true>::W;
        uint32_t a0[W], a1[W], b0[needs_min(RK) ? W : 1], b1[needs_min(RK) ? W : 1];
        load_row_words<DD, true>(maxs + (p0 * H + h) * D, u, a0);
        load_row_words<DD, true>(maxs + (p1 * H + h) * D, u, a1);
        if constexpr (needs_min(RK)) {
          load_row_words<DD, true>(mins + (p0 * H + h) * D, u, b0);
          load_row_words<DD, true>(mins + (p1 * H + h) * D, u, b1);
          s0 = (float)env_exact<RK, DD>(qs, 0, g, u, a0, b0);
          s1 = (float)env_exact<RK, DD>(qs, 0, g, u, a1, b1);
        } else {
          s0 = (float)env_exact<RK, DD>(qs, 0, g, u, a0, a0);
          s1 = (float)env_exact<RK, DD>(qs, 0, g, u, a1, a1);
        }
      }
      if (u == 0) {
        if (rescore_all) {
          exact_keys[j0] = float_key(s0);               // forced pages' keys are never read
          if (has1) exact_keys[j1] = float_key(s1);
        } else {
          und_key[x0] = float_key(s0);
          exact_keys[j0] = float_key(s0);
          if (has1) {
            und_key[x1] = float_key(s1);
            exact_keys[j1] = float_key(s1);
          }
        }
      }
    }
    __syncthreads();
    }
    if (!rescore_all && n_und <= kWave) {
      // rank among the undecided by (key desc, page asc); the best `need` are chosen
      {
        if (w == 0) {
          // composite (key, ~page): larger is better; the others' composites come as LDS
          // broadcasts, four per step, so the loads of a step are in flight together
          const bool mine = lane < n_und;
          const int jx = mine ? und[lane] : 0;
          const uint64_t cx = mine ? ((uint64_t)und_key[lane] << 32) | (uint32_t)~jx : 0ull;
          auto comp = [&](int y) { return ((uint64_t)und_key[y] << 32) | (uint32_t)~und[y]; };
          int rank = 0;
          int y = 0;
          for (; y + 4 <= n_und; y += 4) {
            const uint64_t c0 = comp(y), c1 = comp(y + 1), c2 = comp(y + 2), c3 = comp(y + 3);
            rank += (c0 > cx) + (c1 > cx) + (c2 > cx) + (c3 > cx);
          }
          for (; y < n_und; y++) rank += comp(y) > cx;
          if (mine) status[jx] = rank < need ? 1 : 0;
        }
      }
    } else {
      // exact radix select over the exact keys of the undecided pages (status 2): every
      // candidate after a bound overflow (need = K_free), else the pages of the threshold
      // buckets when more than a wave of them is left (skewed scores, such as the NSA softmax,
      // put most candidates there); ranking them pairwise would cost n^2
      const int kk = rescore_all ? Kfree : need;
      uint32_t ke[kPerThread2];
      uint32_t sm = 0;                               // bit x: slot_page(x) is undecided
      uint32_t kmin = 0xffffffffu, kmax = 0u;
#pragma unroll
      for (int x = 0; x < kPerThread2; x++) {
        const int j = slot_page(x);
        const bool in = ((cand >> x) & 1u) && status[j] == 2;
        ke[x] = in ? exact_keys[j] : 0u;
        if (in) {
          sm |= 1u << x;
          kmin = min(kmin, ke[x]);
          kmax = max(kmax, ke[x]);
        }
      }
      kmin = wave_min_u32(kmin);
      kmax = wave_max_u32(kmax);
      if (lane == 0) {
        mm[0][w] = kmin;
        mm[1][w] = kmax;
      }
      __syncthreads();
#pragma unroll
      for (int x = 0; x < kThreads / kWave; x++) {
        kmin = min(kmin, mm[0][x]);
        kmax = max(kmax, mm[1][x]);
      }
      RadixState se = radix_init(kmin, kmax, kk), none;
      none.top = -1;
      dual_radix_select(ke, ke, sm, se, none, hist, pick);
      const uint32_t kth = se.prefix;
      // strictly better pages are in; equal keys go in by page order
      const int R = (P + kThreads - 1) / kThreads;
      const int j_lo = min(P, tid * R), j_hi = min(P, j_lo + R);
      int n_gt = 0, n_eq = 0;
      for (int j = j_lo; j < j_hi; j++) {
        if (status[j] != 2) continue;
        n_gt += exact_keys[j] > kth;
        n_eq += exact_keys[j] == kth;
      }
      int tot_gt, tot_eq;
      block_incl_scan(n_gt, wave_tot, &tot_gt);
      int eq_rank = block_incl_scan(n_eq, wave_tot, &tot_eq) - n_eq;
      for (int j = j_lo; j < j_hi; j++) {
        if (status[j] != 2) continue;
        const bool ch = exact_keys[j] > kth || (exact_keys[j] == kth && eq_rank++ < kk - tot_gt);
        status[j] = ch ? 1 : 0;
      }
    }
  } else if (n_und > 0) {
    for (int x = tid; x < n_und; x += kThreads) status[und[x]] = 0;   // need == 0
  }
  __syncthreads();

  // ascending compaction of the chosen pages: thread t reads the status bytes of pages
  // [16 t, 16 t + 16) in one 16-byte load (kThreads * 16 = kTwoPassKeys)
  static_assert(kThreads * 16 == kTwoPassKeys, "one 16-byte status load per thread");
  uint32_t chosen = 0;                             // bit e: page 16 tid + e
  {
    const uint4 w = *reinterpret_cast<const uint4*>(&status[16 * tid]);
    const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int e = 0; e < 16; e++)
      chosen |= (((ws[e >> 2] >> (8 * (e & 3))) & 0xffu) == 1u && 16 * tid + e < P) ? (1u << e) : 0u;
  }
  int tot_sel;
  int pos = block_incl_scan(__popc(chosen), wave_tot, &tot_sel) - __popc(chosen);
  while (chosen) {
    const int e = __builtin_ctz(chosen);
    chosen &= chosen - 1u;
    if (pos < max_sel) out[pos] = 16 * tid + e;
    pos++;
  }
  for (int m = tot_sel + tid; m < max_sel; m += kThreads) out[m] = -1;
  if (h == 0 && tid == 0) sel_count[i] = min(tot_sel, max_sel);
}

// The same exact one-pass selection for requests of at most kWaveMaxPages blocks, by one wave per
// (request, KV head) and without workgroup barriers: lane l holds the score keys of blocks
// 8l .. 8l + 7, an MSB-first radix select over 8-bit digits (a 256-bin LDS histogram per pass,
// starting below the bits that every candidate key shares) finds the K_free-th largest
// candidate key, and a prefix over the lanes, which hold the blocks in ascending order, places
// the equal keys by block index and compacts the chosen blocks.  With the decode step's append
// in the launch, either each selection workgroup appends its KV head (append_head), or, for
// blocks too large for that (AppendStep::wgs > 0), the workgroups past the batch's pairs append
// (append_spread) while the selection workgroups run.
constexpr int kWaveMaxPages = 512;
constexpr int kWaveKeys = kWaveMaxPages / kWave;   // keys per lane

__device__ __forceinline__ int wave_excl_scan(int x, int* total) {
  const int incl = wave_incl_sum(x);
  *total = (int)wave_last((uint32_t)incl);
  return incl - x;
}

__global__ __launch_bounds__(kWave) void topk_wave_kernel(
    const float* __restrict__ scores, int H, int ps, int r, int max_pages, int stride, int batch,
    const int32_t* __restrict__ indptr, const int32_t* __restrict__ indices, const int32_t* __restrict__ seq_lens,
    const int32_t* __restrict__ budget, int n_sink, int n_local, int max_sel, int32_t* __restrict__ sel_pages,
    int32_t* __restrict__ sel_count, const AppendStep ap) {
  __shared__ __align__(16) int hist[256];
  if ((int)blockIdx.x >= batch * H) {      // uniform: an append workgroup
    append_spread(ap, (int)blockIdx.x - batch * H, H, ps, r, indptr, indices, seq_lens);
    return;
  }
  const int lane = lane_id();
  const int i = blockIdx.x / H, h = blockIdx.x % H;
  // the score row loads with the request's geometry: lane l reads blocks 8l .. 8l + 7, clamped
  // into the row (stride >= 4 floats; entries past the request's blocks are never used)
  const float* row = scores + ((int64_t)h * batch + i) * stride;
  const float4 sa = *reinterpret_cast<const float4*>(row + min(kWaveKeys * lane, stride - 4));
  const float4 sb = *reinterpret_cast<const float4*>(row + min(kWaveKeys * lane + 4, stride - 4));
  const int base = indptr[i];
  const int P = num_pages(seq_lens[i], ps, (indptr[i + 1] - base) * r, min(max_pages, kWaveMaxPages));
  if (ap.app.knew && ap.wgs == 0) append_head<kWave>(ap, i, h, H, ps, r, base, seq_lens[i], P, indices);
  int Ktot = budget[i];
  Ktot = Ktot < max_sel ? Ktot : max_sel;
  Ktot = Ktot < 0 ? 0 : Ktot;
  int32_t* out = sel_pages + ((int64_t)i * H + h) * max_sel;
  const bool all = Ktot >= P;
  const int nS = min(n_sink, P), nL = min(n_local, P);
  const int nF = all ? P : nS + nL - max(0, nS - (P - nL));
  const int Kfree = all ? 0 : max(0, Ktot - nF);

  uint32_t key[kWaveKeys];
  uint32_t cand = 0;                       // bit x: block 8 lane + x is a candidate
  uint32_t kth = 0;                        // the K_free-th largest candidate key
  if (Kfree > 0) {                         // then P > Ktot >= 1
    const float f[kWaveKeys] = {sa.x, sa.y, sa.z, sa.w, sb.x, sb.y, sb.z, sb.w};
    uint32_t kmin = 0xffffffffu, kmax = 0u;
#pragma unroll
    for (int x = 0; x < kWaveKeys; x++) {
      const int j = kWaveKeys * lane + x;
      key[x] = float_key(f[x]);
      if (j < P && !is_forced(j, P, nS, nL)) {
        cand |= 1u << x;
        kmin = min(kmin, key[x]);
        kmax = max(kmax, key[x]);
      }
    }
    RadixState s = radix_init(wave_min_u32(kmin), wave_max_u32(kmax), Kfree);
    while (s.top >= 0) {                   // uniform over the wave
      const int sh = radix_shift(s);
      const uint32_t dm = radix_dmask(s);
      *reinterpret_cast<int4*>(&hist[4 * lane]) = make_int4(0, 0, 0, 0);
      __syncthreads();
#pragma unroll
      for (int x = 0; x < kWaveKeys; x++)
        if (((cand >> x) & 1u) && (key[x] & s.pmask) == s.prefix) atomicAdd(&hist[(key[x] >> sh) & dm], 1);
      __syncthreads();
      // the bin that holds the remaining-th largest key (lane l: bins 255-4l .. 252-4l), found by
      // exactly one lane and read from its registers
      int c[4], tot = 0;
#pragma unroll
      for (int e = 0; e < 4; e++) {
        c[e] = hist[255 - 4 * lane - e];
        tot += c[e];
      }
      int above = wave_incl_sum(tot) - tot, bin = -1, bin_above = 0;
#pragma unroll
      for (int e = 0; e < 4; e++) {
        if (above < s.remaining && above + c[e] >= s.remaining) {
          bin = 255 - 4 * lane - e;
          bin_above = above;
        }
        above += c[e];
      }
      const int src = __builtin_ctzll(__ballot(bin >= 0));
      const int pk[2] = {__builtin_amdgcn_readlane(bin, src), __builtin_amdgcn_readlane(bin_above, src)};
      radix_advance(s, pk);
      __syncthreads();                     // the histogram read before the next pass clears it
    }
    kth = s.prefix;
  }
  // candidates above the K_free-th key are in; equal keys go in by block order
  int n_gt = 0, n_eq = 0;
#pragma unroll
  for (int x = 0; x < kWaveKeys; x++) {
    if ((cand >> x) & 1u) {
      n_gt += key[x] > kth;
      n_eq += key[x] == kth;
    }
  }
  int tot_gt, tot_eq;
  wave_excl_scan(n_gt, &tot_gt);
  int eq_rank = wave_excl_scan(n_eq, &tot_eq);
  uint32_t chosen = 0;
#pragma unroll
  for (int x = 0; x < kWaveKeys; x++) {
    const int j = kWaveKeys * lane + x;
    bool c = false;
    if ((cand >> x) & 1u) c = key[x] > kth || (key[x] == kth && eq_rank++ < Kfree - tot_gt);
    else if (j < P) c = all || is_forced(j, P, nS, nL);
    chosen |= (uint32_t)c << x;
  }
  int tot_sel;
  int pos = wave_excl_scan(__popc(chosen), &tot_sel);
#pragma unroll
  for (int x = 0; x < kWaveKeys; x++) {
    if ((chosen >> x) & 1u) {
      if (pos < max_sel) out[pos] = kWaveKeys * lane + x;
      pos++;
    }
  }
  for (int m = tot_sel + lane; m < max_sel; m += kWave) out[m] = -1;
  if (h == 0 && lane == 0) sel_count[i] = min(tot_sel, max_sel);
}

// ------------------------------------------------------------------------------------
// Score flows over the operator table's Softmax, Conv1d and Sum, one workgroup per (request,
// KV head), in fp64 with one rounding to fp32:
//   NSA (its block top-k flow, Sec. 3.2: softmax, convolution, head sum, then top-K): for each query
//     head r of the group, p_rj = exp(z_rj - m_r) / l_r, the softmax over the request's pages of
//     the fp32 logits z_r (m_r their max, l_r = sum_j exp(z_rj - m_r); rows of up to
//     kFlowStaged pages multiply by the fp64 reciprocal of l_r); then the conv below; then the
//     sum over the group's heads, in head order.
//   positional smoothing (Appendix G): the conv of the block-mean scores.
// Conv1d along the pages with taps (1/4, 1/2, 1/4) and zero padding:
//   y_j = x_{j-1} / 4 + x_j / 2 + x_{j+1} / 4,  x_{-1} = x_P = 0.
// in: [rows][batch][stride] (NSA: a row per query head; smoothing: a row per KV head).
// out: [H][batch][stride].
// ------------------------------------------------------------------------------------
constexpr int kFlowStaged = 2048;    // NSA rows up to this many pages keep their exponentials in LDS

__device__ __forceinline__ double conv3(double left, double mid, double right) {
  return 0.25 * left + 0.5 * mid + 0.25 * right;
}

__device__ __forceinline__ double block_sum_f64(double x, double* red) {
  const int lane = lane_id(), w = threadIdx.x >> 6;
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) x += __shfl_xor(x, off, kWave);
  __syncthreads();                                   // red free from its previous use
  if (lane == 0) red[w] = x;
  __syncthreads();
  double t = 0.0;
#pragma unroll
  for (int k = 0; k < kThreads / kWave; k++) t += red[k];
  return t;
}

template <bool kNsa>
__global__ __launch_bounds__(kThreads) void flow_kernel(const float* __restrict__ in, float* __restrict__ out, int H,
                                                        int g, int ps, int r, int max_pages, int stride, int batch,
                                                        const int32_t* __restrict__ indptr,
                                                        const int32_t* __restrict__ seq_lens,
                                                        const int32_t* __restrict__ items) {
  __shared__ double red[kThreads / kWave];
  __shared__ float wave_fm[2][kThreads / kWave];
  __shared__ double m_of[16], l_of[16];
  __shared__ double e_lds[kNsa ? kFlowStaged : 1];  // exp(z_j - m) of one head's row
  const int tid = threadIdx.x;
  const int i = blockIdx.x / H, h = blockIdx.x % H;
  const int P = items ? max(0, min(items[i], stride))
                      : num_pages(seq_lens[i], ps, (indptr[i + 1] - indptr[i]) * r, max_pages);
  float* y = out + ((int64_t)h * batch + i) * stride;
  if constexpr (!kNsa) {
    const float* x = in + ((int64_t)h * batch + i) * stride;
    for (int j = tid; j < P; j += kThreads) {
      const double left = j > 0 ? (double)x[j - 1] : 0.0;
      const double right = j + 1 < P ? (double)x[j + 1] : 0.0;
      y[j] = (float)conv3(left, (double)x[j], right);
    }
    return;
  }
  if (P <= kFlowStaged) {
    // rows up to kFlowStaged pages: one exponential per page and head, staged in LDS for the
    // convolution's neighbours; thread t accumulates pages t, t + kThreads, ... in registers
    double acc[kFlowStaged / kThreads];
#pragma unroll
    for (int k = 0; k < kFlowStaged / kThreads; k++) acc[k] = 0.0;
    for (int r = 0; r < g; r++) {
      const float* z = in + ((int64_t)(h * g + r) * batch + i) * stride;
      float mx = -INFINITY, mn = INFINITY;
      for (int j = tid; j < P; j += kThreads) mx = fmaxf(mx, z[j]);
      __syncthreads();                               // wave_fm and e_lds free from their last use
      block_fminmax(mn, mx, wave_fm);
      double l = 0.0;
      for (int j = tid; j < P; j += kThreads) {
        const double e = exp((double)z[j] - (double)mx);
        e_lds[j] = e;
        l += e;
      }
      l = block_sum_f64(l, red);                     // its barriers also publish e_lds
      const double inv_l = 1.0 / l;
      for (int j = tid; j < P; j += kThreads) e_lds[j] *= inv_l;   // the softmax of the row
      __syncthreads();
#pragma unroll
      for (int k = 0; k < kFlowStaged / kThreads; k++) {
        const int j = tid + k * kThreads;
        if (j < P) acc[k] += conv3(j > 0 ? e_lds[j - 1] : 0.0, e_lds[j], j + 1 < P ? e_lds[j + 1] : 0.0);
      }
    }
#pragma unroll
    for (int k = 0; k < kFlowStaged / kThreads; k++) {
      const int j = tid + k * kThreads;
      if (j < P) y[j] = (float)acc[k];
    }
    return;
  }
  // longer rows: softmax statistics of each query head's row, then three exponentials per
  // page and head (the neighbours are recomputed rather than staged)
  for (int r = 0; r < g; r++) {
    const float* z = in + ((int64_t)(h * g + r) * batch + i) * stride;
    float mx = -INFINITY, mn = INFINITY;
    for (int j = tid; j < P; j += kThreads) mx = fmaxf(mx, z[j]);
    __syncthreads();                                 // wave_fm free from its previous use
    block_fminmax(mn, mx, wave_fm);
    double l = 0.0;
    for (int j = tid; j < P; j += kThreads) l += exp((double)z[j] - (double)mx);
    l = block_sum_f64(l, red);
    if (tid == 0) {
      m_of[r] = (double)mx;
      l_of[r] = l;
    }
  }
  __syncthreads();
  for (int j = tid; j < P; j += kThreads) {
    double acc = 0.0;
    for (int r = 0; r < g; r++) {
      const float* z = in + ((int64_t)(h * g + r) * batch + i) * stride;
      const double m = m_of[r], l = l_of[r];
      const double left = j > 0 ? exp((double)z[j - 1] - m) / l : 0.0;
      const double mid = exp((double)z[j] - m) / l;
      const double right = j + 1 < P ? exp((double)z[j + 1] - m) / l : 0.0;
      acc += conv3(left, mid, right);
    }
    y[j] = (float)acc;
  }
}

// Persistent grid: as many workgroups as can be resident at once, but no more than give each
// about kMinItemsPerWg (page, KV head) items (at least one per CU): a workgroup stages its
// request's query block (up to 18 KiB for the MLA geometry) before it streams, which only pays
// off over enough items.  The item count is bounded on the host by batch x max blocks x H.
// Measured on the MLA workload (16384 items; score + top-K): 30.0 us with every resident slot,
// 25.1 us at 32 items per workgroup, 27.1 us at 64 and 27.0 us at 128.
constexpr int kMinItemsPerWg = 32;
template <int KIND, int D>
void launch_score(const ScoreArgs& a, hipStream_t stream) {
  const size_t lds = (size_t)score_lds<KIND, D>(a.batch, a.Hq, a.H).total;
  // page_indptr in LDS up to kMaxLdsBatch requests, read from global memory beyond
  const bool lds_ind = a.batch <= kMaxLdsBatch;
  const void* fn = lds_ind ? reinterpret_cast<const void*>(score_kernel<KIND, D, true>)
                           : reinterpret_cast<const void*>(score_kernel<KIND, D, false>);
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kThreads, lds) != hipSuccess || per_cu < 1)
    per_cu = 1;
  // a persistent grid must be resident at once: also bound it by the CU's LDS
  hipFuncAttributes fa;
  if (hipFuncGetAttributes(&fa, fn) == hipSuccess) {
    const int by_lds = (int)(kLdsPerCu / (fa.sharedSizeBytes + lds));
    per_cu = std::max(1, std::min(per_cu, by_lds));
  }
  const int cus = device_cus();
  const long long items = (long long)a.batch * a.max_pages * a.H;
  const long long by_items = (items + kMinItemsPerWg - 1) / kMinItemsPerWg;
  const long long grid = std::max<long long>(cus, std::min<long long>((long long)per_cu * cus * kScoreGridFactor, by_items));
  if (lds_ind) hipLaunchKernelGGL((score_kernel<KIND, D, true>), dim3((unsigned)grid), dim3(kThreads), lds, stream, a);
  else hipLaunchKernelGGL((score_kernel<KIND, D, false>), dim3((unsigned)grid), dim3(kThreads), lds, stream, a);
}

}  // namespace

int device_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    cus = 0;
  return cus > 0 ? cus : 256;
}

size_t score_workspace_bytes(int batch, int num_kv_heads, int num_q_heads, int max_pages) {
  const size_t planes = std::max(2 * num_kv_heads, num_q_heads + num_kv_heads);
  size_t b = planes * (size_t)batch * (size_t)score_stride(max_pages) * sizeof(float);
  return (b + 255) & ~(size_t)255;
}

// One-pass scores of an ABI score kind (NSA: its per-head logits; smoothing: the block mean it
// smooths): the block mean for D in {64, 128, 576}, every other kind for D in {64, 128} (the
// host rejects the rest).
void launch_one_pass_score(int abi_kind, int Dqk, const ScoreArgs& a, hipStream_t stream) {
#define VX_ENV(K)                                   \
  do {                                              \
    if (Dqk == 64) launch_score<K, 64>(a, stream);  \
    else launch_score<K, 128>(a, stream);           \
  } while (0)
  switch (internal_kind(abi_kind)) {
    case kMeanDot:
      if (Dqk == 64) launch_score<kMeanDot, 64>(a, stream);
      else if (Dqk == 128) launch_score<kMeanDot, 128>(a, stream);
      else launch_score<kMeanDot, 576>(a, stream);
      break;
    case kQuest: VX_ENV(kQuest); break;
    case kQuestConsensus: VX_ENV(kQuestConsensus); break;
    case kEnvLower: VX_ENV(kEnvLower); break;
    case kQuestRectified: VX_ENV(kQuestRectified); break;
    case kHeadDot: VX_ENV(kHeadDot); break;
    default: VX_ENV(kMaxDot); break;
  }
#undef VX_ENV
}

hipError_t launch_score_topk(const Geometry& g, const uint16_t* q, int Hq, int kind, const float* mean,
                             const uint16_t* mean_bf, const uint16_t* maxs, const uint16_t* mins,
                             const int32_t* budget, int n_sink, int n_local, int max_sel, int32_t* sel_pages,
                             int32_t* sel_count, void* ws, int remap, int tau_q, uint32_t seed, hipStream_t stream,
                             const StepAppend& sa) {
  if (g.batch == 0) return hipSuccess;
  float* scores = reinterpret_cast<float*>(ws);
  const bool approx = remap != 0 || tau_q != 0;           // one-pass scores, then the radix select
  const int ik = internal_kind(kind);
  // the selection paths: the block mean's two passes, the envelope kinds' two passes, else one
  // pass of scores (through a flow for NSA and smoothing) selected by the one-wave kernel up to
  // kWaveMaxPages blocks per request, the bucketed kernel up to kTwoPassKeys, else the radix kernel
  const bool mean_two_pass = (kind == kMeanDot || kind == kAbiContent) && mean_bf && !approx;
  const bool env_two_pass =
      is_env(ik) && !approx && g.max_pages <= kTwoPassKeys && Hq <= 4 * g.H && (g.Dqk == 64 || g.Dqk == 128);
  const bool flow = kind == kAbiNsa || kind == kAbiSmooth;
  const bool wave = !approx && !mean_two_pass && !env_two_pass && g.max_pages <= kWaveMaxPages;
  // The step's append: inside the top-K launch, or first of all when the selection reads every
  // block's score (the flows couple the pages; the radix path is not fused).  A block too large
  // for one workgroup to refresh in the selection's shadow (a 64-token block of 576 channels)
  // gets workgroups of its own in the one-wave selection launch, or else a launch of its own
  // ahead of the selection.
  const bool spread = wave && !flow && g.bs * g.Dqk > kFusedAppendMaxElems;
  AppendStep ap{};
  if (sa.k_new) {
    if (approx || g.max_pages > kTwoPassKeys || flow || (g.bs * g.Dqk > kFusedAppendMaxElems && !spread)) {
      const hipError_t e =
          launch_kv_append_summarize(g, sa.k_new, sa.v_new, sa.mean, sa.mean_bf, sa.maxo, sa.mino, stream);
      if (e != hipSuccess) return e;
    } else {
      ap.app = summ::AppendArgs{sa.k_new, sa.v_new, const_cast<void*>(g.k), const_cast<void*>(g.v)};
      ap.k = g.k;
      ap.k_scale = g.k_scale;
      ap.kt = g.kv_dtype;
      ap.ps = g.ps;
      ap.D = g.Dqk;
      ap.num_phys = g.num_phys_pages;
      ap.mean = sa.mean;
      ap.mean_bf = sa.mean_bf;
      ap.maxo = sa.maxo;
      ap.mino = sa.mino;
      ap.max_pages = g.max_pages;
      ap.wgs = spread ? (g.H * (g.Dqk / 8) + kWave / 4 - 1) / (kWave / 4) : 0;
    }
  }
  ScoreArgs a;
  a.q = q;
  a.indptr = g.indptr;
  a.indices = g.indices;
  a.seq_lens = g.seq_lens;
  a.mean = mean;
  a.maxs = maxs;
  a.mins = mins;
  a.scores = scores;
  a.Hq = Hq;
  a.H = g.H;
  a.ps = g.bs;                               // scores are per block
  a.r = g.r;
  a.num_phys = g.num_phys_pages;
  a.max_pages = g.max_pages;
  a.batch = g.batch;
  a.stride = score_stride(g.max_pages);
  a.plane = (int64_t)g.H * g.batch * a.stride;
  a.qdims = kind == kAbiContent ? g.Dv : g.Dqk;
  if (mean_two_pass) {
    a.maxs = mean_bf;
    if (g.Dqk == 64) launch_score<kMeanBound, 64>(a, stream);
    else if (g.Dqk == 128) launch_score<kMeanBound, 128>(a, stream);
    else launch_score<kMeanBound, 576>(a, stream);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const float* upper = scores + a.plane;
#define VX_TWO_PASS(DD)                                                                                           \
  hipLaunchKernelGGL((topk_bucket_kernel<kMeanDot, DD>), dim3(g.batch * g.H), dim3(kThreads), 0, stream, scores,  \
                     upper, mean, nullptr, nullptr, q, Hq, g.H, a.qdims, g.bs, g.r, g.max_pages, a.stride, g.batch, \
                     g.num_phys_pages, g.indptr, g.indices, g.seq_lens, budget, n_sink, n_local, max_sel, sel_pages, \
                     sel_count, ap)
    if (g.Dqk == 64) VX_TWO_PASS(64);
    else if (g.Dqk == 128) VX_TWO_PASS(128);
    else VX_TWO_PASS(576);
#undef VX_TWO_PASS
    return hipGetLastError();
  }
  if (env_two_pass) {
    // the envelope kinds' exact two-pass selection: fp32 bound pass, then re-scoring of the
    // undecided pages in the bucketed select
    switch (ik) {
#define VX_ENV_TWO_PASS(K)                                                                                          \
  case K:                                                                                                          \
    if (g.Dqk == 64) {                                                                                             \
      launch_score<bound_of_env(K), 64>(a, stream);                                                                \
      hipLaunchKernelGGL((topk_bucket_kernel<K, 64>), dim3(g.batch * g.H), dim3(kThreads), 0, stream, scores,      \
                         scores + a.plane, nullptr, maxs, mins, q, Hq, g.H, a.qdims, g.bs, g.r, g.max_pages, a.stride, \
                         g.batch, g.num_phys_pages, g.indptr, g.indices, g.seq_lens, budget, n_sink, n_local,      \
                         max_sel, sel_pages, sel_count, ap);                                                       \
    } else {                                                                                                       \
      launch_score<bound_of_env(K), 128>(a, stream);                                                               \
      hipLaunchKernelGGL((topk_bucket_kernel<K, 128>), dim3(g.batch * g.H), dim3(kThreads), 0, stream, scores,     \
                         scores + a.plane, nullptr, maxs, mins, q, Hq, g.H, a.qdims, g.bs, g.r, g.max_pages, a.stride, \
                         g.batch, g.num_phys_pages, g.indptr, g.indices, g.seq_lens, budget, n_sink, n_local,      \
                         max_sel, sel_pages, sel_count, ap);                                                       \
    }                                                                                                              \
    break;
      VX_ENV_TWO_PASS(kQuest)
      VX_ENV_TWO_PASS(kQuestConsensus)
      VX_ENV_TWO_PASS(kEnvLower)
      VX_ENV_TWO_PASS(kQuestRectified)
#undef VX_ENV_TWO_PASS
      default: break;
    }
    return hipGetLastError();
  }
  if (kind == kAbiNsa || kind == kAbiSmooth) {
    // the flow's first step into the planes after the first H, its last step into plane 0
    float* first = scores + (int64_t)g.H * g.batch * a.stride;
    a.scores = first;
    a.plane = (int64_t)g.batch * a.stride;
    launch_one_pass_score(kind, g.Dqk, a, stream);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = launch_score_flow(kind, first, scores, a.stride, g.H, Hq, g.batch, nullptr, g.bs, g.r, g.max_pages,
                          g.indptr, g.seq_lens, stream);
    if (e != hipSuccess) return e;
  } else {
    launch_one_pass_score(kind, g.Dqk, a, stream);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (wave) {
    const int grid = g.batch * g.H + (ap.app.knew ? g.batch * ap.wgs : 0);
    hipLaunchKernelGGL(topk_wave_kernel, dim3(grid), dim3(kWave), 0, stream, scores, g.H, g.bs, g.r,
                       g.max_pages, a.stride, g.batch, g.indptr, g.indices, g.seq_lens, budget, n_sink, n_local,
                       max_sel, sel_pages, sel_count, ap);
    return hipGetLastError();
  }
  if (g.max_pages <= kTwoPassKeys && !approx) {
    hipLaunchKernelGGL((topk_bucket_kernel<kNoRescore, 0>), dim3(g.batch * g.H), dim3(kThreads), 0, stream, scores,
                       scores, nullptr, nullptr, nullptr, nullptr, Hq, g.H, g.Dqk, g.bs, g.r, g.max_pages, a.stride,
                       g.batch, g.num_phys_pages, g.indptr, g.indices, g.seq_lens, budget, n_sink, n_local, max_sel,
                       sel_pages, sel_count, ap);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(topk_kernel, dim3(g.batch * g.H), dim3(kThreads), 0, stream, scores, g.H, g.bs, g.r,
                     g.max_pages, a.stride, g.batch, g.indptr, g.seq_lens, nullptr, budget, n_sink, n_local, max_sel,
                     TopkOptions{remap, tau_q, seed}, sel_pages, sel_count);
  return hipGetLastError();
}

hipError_t launch_score(const Geometry& g, const uint16_t* q, int Hq, int kind, const float* mean,
                        const uint16_t* maxs, const uint16_t* mins, float* scores, int stride, hipStream_t stream) {
  if (g.batch == 0) return hipSuccess;
  ScoreArgs a;
  a.q = q;
  a.indptr = g.indptr;
  a.indices = g.indices;
  a.seq_lens = g.seq_lens;
  a.mean = mean;
  a.maxs = maxs;
  a.mins = mins;
  a.scores = scores;
  a.Hq = Hq;
  a.H = g.H;
  a.ps = g.bs;                               // scores are per block
  a.r = g.r;
  a.num_phys = g.num_phys_pages;
  a.max_pages = g.max_pages;
  a.batch = g.batch;
  a.stride = stride;
  a.plane = (int64_t)g.batch * stride;       // NSA logits: the rows of query head r start at r * plane
  a.qdims = kind == kAbiContent ? g.Dv : g.Dqk;
  launch_one_pass_score(kind, g.Dqk, a, stream);
  return hipGetLastError();
}

hipError_t launch_score_flow(int kind, const float* in, float* out, int stride, int H, int Hq, int batch,
                             const int32_t* items, int ps, int r, int max_pages, const int32_t* indptr,
                             const int32_t* seq_lens, hipStream_t stream) {
  if (batch == 0) return hipSuccess;
  if (kind == kAbiNsa)
    hipLaunchKernelGGL(flow_kernel<true>, dim3(batch * H), dim3(kThreads), 0, stream, in, out, H, Hq / H, ps, r,
                       max_pages, stride, batch, indptr, seq_lens, items);
  else
    hipLaunchKernelGGL(flow_kernel<false>, dim3(batch * H), dim3(kThreads), 0, stream, in, out, H, Hq / H, ps, r,
                       max_pages, stride, batch, indptr, seq_lens, items);
  return hipGetLastError();
}

hipError_t launch_topk_select(const float* scores, int stride, int H, int batch, const int32_t* items,
                              const int32_t* budget, int n_sink, int n_local, int max_sel, int remap, int tau_q,
                              uint32_t seed, int32_t* sel_pages, int32_t* sel_count, hipStream_t stream) {
  if (batch == 0) return hipSuccess;
  hipLaunchKernelGGL(topk_kernel, dim3(batch * H), dim3(kThreads), 0, stream, scores, H, 16, 1, stride, stride, batch,
                     nullptr, nullptr, items, budget, n_sink, n_local, max_sel, TopkOptions{remap, tau_q, seed},
                     sel_pages, sel_count);
  return hipGetLastError();
}

}  // namespace vx

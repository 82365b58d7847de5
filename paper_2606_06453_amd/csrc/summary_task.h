// One summary task of the cache stage (Sec. 3.1 Eq. 1; Sec. 3.2 Quest): 8 consecutive channels
// of one (block, KV head) slice, its Mean, Max and Min over the block's valid tokens, with TS
// adjacent lanes sharing the task (lane `slice` takes every TS-th token, quad DPP combines them).
// In append mode the step's new K/V rows are written at token L - 1 first, and the new key row
// enters its slice's running sums last, exactly where a pass over the page would add it.
// summarize_kernel and the top-K kernels (which run the decode step's append in their own
// launch) both call task(), so their summaries are bit-identical.
#pragma once
#include <type_traits>

#include "vx_device.h"
#include "vx_internal.h"

namespace vx {
namespace summ {

constexpr int kBatch = 8;        // token rows a lane loads per round trip (default)

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

// Task (block j of request i, KV head h, channel chunk c8); `active` false: the lane only joins
// the quad's DPP exchanges.  Block j is block j % r of the page at indices[base + j / r].
template <int TS, int KT, bool APPEND, int KB = kBatch>
__device__ __forceinline__ void task(const void* __restrict__ kv, float k_scale, int num_phys, int H, int ps, int bs,
                                     int r, int D, const int32_t* __restrict__ indices, int base, int L, int i, int j,
                                     int h, int c8, bool active, int slice, float* __restrict__ mean,
                                     uint16_t* __restrict__ mean_bf, uint16_t* __restrict__ maxo,
                                     uint16_t* __restrict__ mino, const AppendArgs& app) {
  // An fp8 cache value is the fp32 product scale * code, rounded; no product may be fused into
  // a sum (the compiler could fuse it in one launch's copy of this code and not in another's,
  // and the summaries of the append and of a pass over the page would then differ).
#pragma clang fp contract(off)
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
  // append: the step's K (and V) chunk load first; they are written to row n - 1 after the
  // block's other rows are in flight (nothing in this launch reads row n - 1)
  typename RC::Raw new_row{}, new_v{};
  const bool writer = APPEND && active && slice == 0;
  if constexpr (APPEND) {
    const int64_t in = (((int64_t)i * H + h) * D + c8 * 8) * (RC::kBytes / 8);
    new_row = *reinterpret_cast<const typename RC::Raw*>(static_cast<const char*>(app.knew) + in);
    if (writer && app.vnew)   // V rows have D channels too (GQA); an aliased V has no rows of its own
      new_v = *reinterpret_cast<const typename RC::Raw*>(static_cast<const char*>(app.vnew) + in);
  }

  float s[8], mx[8], mn[8];
#pragma unroll
  for (int e = 0; e < 8; e++) {
    s[e] = 0.f;
    mx[e] = -INFINITY;
    mn[e] = INFINITY;
  }
  // KB token rows per round trip: clamped, unconditional loads, then masked adds
  for (int t0 = slice; t0 < n_mem; t0 += TS * KB) {
    typename RC::Raw w[KB];
#pragma unroll
    for (int b = 0; b < KB; b++)
      w[b] = *reinterpret_cast<const typename RC::Raw*>(src + (int64_t)min(t0 + TS * b, n_mem - 1) * row_bytes);
    // The rows past the block's end are masked instead of skipped: a branch per row would let the
    // compiler sink each load into it, one round trip per row.  Adding +0 leaves s unchanged (s
    // starts at +0 and round-to-nearest never makes it -0), and -inf / +inf leave the max / min
    // unchanged, so the sums are those of the valid rows in the same order.
#pragma unroll
    for (int b = 0; b < KB; b++) {
      const bool ok = t0 + TS * b < n_mem;
      float x[8];
      RC::values(w[b], k_scale, x);
#pragma unroll
      for (int e = 0; e < 8; e++) {
        s[e] += ok ? x[e] : 0.f;
        mx[e] = fmaxf(mx[e], ok ? x[e] : -INFINITY);
        mn[e] = fminf(mn[e], ok ? x[e] : INFINITY);
      }
    }
  }
  if constexpr (APPEND) {
    if (writer) {
      const int64_t out = (row0 + (int64_t)(n - 1) * D) * (RC::kBytes / 8);
      *reinterpret_cast<typename RC::Raw*>(static_cast<char*>(app.kw) + out) = new_row;
      if (app.vnew) *reinterpret_cast<typename RC::Raw*>(static_cast<char*>(app.vw) + out) = new_v;
    }
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
  if (!active || slice != 0) return;
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

}  // namespace summ
}  // namespace vx

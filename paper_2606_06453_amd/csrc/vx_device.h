// Device-side helpers shared by the vx kernels (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vx {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(short)))) short s16x4_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;

constexpr int kWave = 64;

// ---- bfloat16 <-> float ------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }
__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  uint32_t r = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
  return (f != f) ? 0x7fc0u : r;
}

// ---- streaming loads ----------------------------------------------------------------
// Data read once per step (summaries, K/V tiles): the non-temporal hint keeps it from
// displacing reusable lines in L2 and the Infinity Cache.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
typedef float float2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint4 load_stream_u4(const void* p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint2 load_stream_u2(const void* p) {
  const u32x2_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(p));
  return make_uint2(v.x, v.y);
}

// ---- order-preserving key of a float (larger float -> larger key; -0.0 == +0.0) ------
__device__ __forceinline__ uint32_t float_key(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0;                     // -0.0 ranks as +0.0
  if (f != f) return 0;                            // NaN ranks below everything
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// ---- cross-lane ---------------------------------------------------------------------
// DPP controls (GFX9 encoding): row_ror:n = 0x120 + n rotates within a row of 16 lanes.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double x) {
  uint64_t u = (uint64_t)__double_as_longlong(x);
  int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)u, CTRL, 0xf, 0xf, false);
  int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(u >> 32), CTRL, 0xf, 0xf, false);
  return __longlong_as_double((long long)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo));
}

// Sum over the 16 lanes of a DPP row; every lane of the row receives the total (each lane adds
// in its own order).
__device__ __forceinline__ float row16_sum_f32(float x) {
  x += dpp_f32<0x128>(x);
  x += dpp_f32<0x124>(x);
  x += dpp_f32<0x122>(x);
  x += dpp_f32<0x121>(x);
  return x;
}

// Sum over the 16 lanes of a DPP row; every lane of the row receives the total.
__device__ __forceinline__ double row16_sum_f64(double x) {
  x += dpp_f64<0x128>(x);
  x += dpp_f64<0x124>(x);
  x += dpp_f64<0x122>(x);
  x += dpp_f64<0x121>(x);
  return x;
}

__device__ __forceinline__ float xor_shfl(float x, int mask) { return __shfl_xor(x, mask, kWave); }

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & (kWave - 1)); }

// Exclusive prefix count of `pred` over the wave's lanes, and the wave total.
__device__ __forceinline__ int wave_excl_count(bool pred, int* total) {
  uint64_t m = __ballot(pred);
  *total = __popcll(m);
  uint64_t below = (lane_id() == 0) ? 0ull : (~0ull >> (64 - lane_id()));
  return __popcll(m & below);
}

__device__ __forceinline__ int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Pages of request i that actually exist: ceil(L / ps), capped by the length of its page
// list (and by `cap`), so that broken contents can never index out of bounds.
__device__ __forceinline__ int num_pages(int L, int ps, int list_len, int cap) {
  int P = L > 0 ? ceil_div(L, ps) : 0;
  P = P < list_len ? P : list_len;
  P = P < cap ? P : cap;
  return P < 0 ? 0 : P;
}

// Physical page ids are the caller's contract; clamping keeps a broken id inside the cache.
__device__ __forceinline__ int64_t clamp_page(int p, int num_phys) {
  p = p < 0 ? 0 : p;
  return (int64_t)(p < num_phys ? p : num_phys - 1);
}

// Physical block of block reference jb (r blocks per page): block jb % r of the page at
// indices[jb / r].  Summaries of blocks are indexed by it.  r = 1: the physical page.
__device__ __forceinline__ int64_t block_row(const int32_t* indices, int jb, int r, int num_phys) {
  const int q = jb / r;
  return clamp_page(indices[q], num_phys) * r + (jb - q * r);
}

}  // namespace vx

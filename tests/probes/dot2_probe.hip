// Test-only probe: one v_dot2c_f32_bf16 per element, d[i] = a[i].lo * b[i].lo + a[i].hi * b[i].hi + c[i],
// so that a GPU test can check the rounding model that the envelope kinds' bound pass assumes of
// the instruction against exact sums on the host.  Not part of libvx.
#include <hip/hip_runtime.h>
#include <cstdint>

namespace {
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__global__ __launch_bounds__(256) void dot2_kernel(const uint32_t* __restrict__ a, const uint32_t* __restrict__ b,
                                                   const float* __restrict__ c, float* __restrict__ d, int n) {
  const int t = (int)(blockIdx.x * blockDim.x + threadIdx.x);
  if (t >= n) return;
  d[t] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a[t]), __builtin_bit_cast(bf16x2_t, b[t]), c[t],
                                         false);
}
}  // namespace

// a, b: n packed bf16 pairs; c, d: n floats; all device pointers.  Returns the hipError_t of the
// launch (n <= 0 launches nothing).
extern "C" int vxt_dot2_bf16(const uint32_t* a, const uint32_t* b, const float* c, float* d, int n,
                             hipStream_t stream) {
  if (n <= 0) return 0;
  hipLaunchKernelGGL(dot2_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, a, b, c, d, n);
  return (int)hipGetLastError();
}

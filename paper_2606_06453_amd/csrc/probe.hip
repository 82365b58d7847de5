// Measurement utility: the practical HBM read rate of this device for a plain stream of
// 16-byte loads with the non-temporal hint (the load form of the decode and score kernels).
// It sits beside the nameplate peak in the benchmark's roofline; it is not a step of the path.
#include "vx_device.h"
#include "vx_internal.h"

namespace vx {
namespace {

constexpr int kProbeThreads = 256;

// Grid-stride stream over n16 16-byte chunks, four loads in flight per lane.  The XOR of the
// words keeps every load live; a workgroup writes its value only in the (practically never
// taken) case that it equals an arbitrary constant, so the kernel writes nothing in practice.
__global__ __launch_bounds__(kProbeThreads) void stream_read_kernel(const uint4* __restrict__ p, int64_t n16,
                                                                     uint32_t* __restrict__ sink) {
  uint32_t acc = 0;
  const int64_t stride = (int64_t)gridDim.x * kProbeThreads;
  int64_t i = (int64_t)blockIdx.x * kProbeThreads + threadIdx.x;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const uint4 a = load_stream_u4(p + i);
    const uint4 b = load_stream_u4(p + i + stride);
    const uint4 c = load_stream_u4(p + i + 2 * stride);
    const uint4 d = load_stream_u4(p + i + 3 * stride);
    acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w;
  }
  for (; i < n16; i += stride) {
    const uint4 a = load_stream_u4(p + i);
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  if (acc == 0x9e3779b9u) sink[blockIdx.x] = acc;
}

}  // namespace

hipError_t launch_stream_read(const void* buf, int64_t bytes, uint32_t* sink, int workgroups, hipStream_t stream) {
  hipLaunchKernelGGL(stream_read_kernel, dim3(workgroups), dim3(kProbeThreads), 0, stream,
                     static_cast<const uint4*>(buf), bytes / 16, sink);
  return hipGetLastError();
}

}  // namespace vx

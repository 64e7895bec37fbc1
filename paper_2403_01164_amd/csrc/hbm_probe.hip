// Achievable HBM read bandwidth on this device: a streaming read of a device buffer
// with the same 16-byte non-temporal loads as the GEMV, many in flight per lane and
// no arithmetic to speak of.  The denominator the GEMV's measured bandwidth is
// compared with next to the nominal 8 TB/s (the rows of a GEMV cannot be read faster).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hbm_probe.h"

namespace hg {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kThreads = 256;
constexpr int kUnroll = 8;

__global__ __launch_bounds__(kThreads) void read_kernel(const u32x4* __restrict__ p, size_t n16, uint32_t* sink) {
  const __attribute__((address_space(1))) u32x4* g = (const __attribute__((address_space(1))) u32x4*)p;
  const size_t stride = (size_t)gridDim.x * kThreads * kUnroll;
  uint32_t acc = 0;
  size_t i = (size_t)blockIdx.x * kThreads * kUnroll + threadIdx.x;
  for (; i + (size_t)kThreads * (kUnroll - 1) < n16; i += stride) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) v[u] = __builtin_nontemporal_load(g + i + (size_t)kThreads * u);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc ^= v[u].x ^ v[u].w;
  }
  for (; i < n16; i += kThreads) acc ^= g[i].y;  // tail of a buffer that is not a whole number of steps
  if (acc == 0x9E3779B9u) sink[0] = acc;        // keeps the loads; practically never stores
}

__global__ void empty_kernel() {}

}  // namespace

hipError_t launch_empty(hipStream_t stream) {
  hipLaunchKernelGGL(empty_kernel, dim3(1), dim3(64), 0, stream);
  return hipGetLastError();
}

hipError_t launch_read(const void* buf, size_t bytes, uint32_t* sink, int grid, hipStream_t stream) {
  if (!buf || !sink || grid < 1 || (bytes & 15)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(read_kernel, dim3(grid), dim3(kThreads), 0, stream, (const u32x4*)buf, bytes / 16, sink);
  return hipGetLastError();
}

}  // namespace hg

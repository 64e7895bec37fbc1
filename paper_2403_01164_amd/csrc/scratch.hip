// Fixed split-K scratch of the matrix-core GEMV for callers that cannot allocate device
// memory (code under HIP graph capture, tight serving loops): one array per GPU, compiled
// into the library, whose device address is taken once per device.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "kernels.h"

namespace hg {

// ---- fixed split-K scratch for callers that cannot allocate ----
// One array per GPU, zero-initialised when the code object loads: kScratchCounterWords
// arrival counters, then kScratchFloats floats of partials (1.25 MiB).  Host code must not use the
// array's name as a device address (it is a host-side stand-in): the address is taken
// once per device with hipGetSymbolAddress and kept in g_scratch.
static __device__ __align__(256) uint32_t scratch[kScratchCounterWords + kScratchFloats];

namespace {
constexpr int kThreads = 256;
constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kScratchDevices] = {};

__global__ __launch_bounds__(kThreads) void zero_words_kernel(uint32_t* p, long long n) {
  for (long long i = (long long)blockIdx.x * kThreads + threadIdx.x; i < n; i += (long long)gridDim.x * kThreads)
    p[i] = 0u;
}
}  // namespace

hipError_t scratch_init(int device) {
  if (device < 0 || device >= kScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch[device]) return hipSuccess;
  void* ptr = nullptr;
  hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  // the counters must start at zero (every split launch returns the ones it used to zero)
  hipLaunchKernelGGL(zero_words_kernel, dim3(64), dim3(kThreads), 0, nullptr, (uint32_t*)ptr,
                     (long long)kScratchCounterWords);
  e = hipGetLastError();
  if (e == hipSuccess) e = hipStreamSynchronize(nullptr);
  if (e != hipSuccess) return e;
  g_scratch[device] = ptr;
  return hipSuccess;
}

void* scratch_ptr(int device) {
  if (device < 0 || device >= kScratchDevices) return nullptr;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  return g_scratch[device];
}

}  // namespace hg

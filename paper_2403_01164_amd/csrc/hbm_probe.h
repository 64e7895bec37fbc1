// Internal launch interface of the HBM read probe (not part of the C ABI).
#pragma once
#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace hg {

// Streams `bytes` (a multiple of 16) of device memory at buf with `grid` workgroups;
// sink is a device word the kernel writes only for one value of the data.
hipError_t launch_read(const void* buf, size_t bytes, uint32_t* sink, int grid, hipStream_t stream);

// One workgroup of one wavefront that does nothing (the launch round-trip probe).
hipError_t launch_empty(hipStream_t stream);

}  // namespace hg

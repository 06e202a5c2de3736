// Launch interface of the streaming-read ceiling kernels (a measurement aid).
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>

namespace spork {

// Read `bytes` of `src` with `grid` workgroups of 256 threads; mode 0:
// register loads, 1: direct-to-LDS loads in the attention kernel's ring
// shape, 2: non-temporal register loads. sink: grid * 256 words.
hipError_t launch_read_ceiling(const void* src, int64_t bytes, int32_t grid, int32_t mode, uint32_t* sink,
                               hipStream_t stream);

}  // namespace spork

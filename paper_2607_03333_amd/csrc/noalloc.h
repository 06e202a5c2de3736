// Interface of the library-owned scratch memory behind
// spork_verify_accept_noalloc.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstddef>

namespace spork {

// Size of the per-device scratch array (64 MiB): the partial results, list
// cursors and argmax keys of one call must fit.
constexpr size_t kScratchBytes = static_cast<size_t>(64) << 20;

// Device address of the current device's scratch array (looked up on the
// device's first call), with its first `control_bytes` bytes zero in stream
// order on `stream` (cleared by a small kernel when the previous call left
// fewer of them zero). Allocates no device memory.
hipError_t scratch_acquire(size_t control_bytes, hipStream_t stream, void** ptr);

}  // namespace spork

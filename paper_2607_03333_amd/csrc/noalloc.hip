// Library-owned scratch memory for spork_verify_accept_noalloc: a
// file-scope device array (each GPU the library runs on holds its own copy
// until the process ends) in place of the caller's workspace, for callers
// that cannot allocate device memory.
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <mutex>

#include "kernels.h"
#include "noalloc.h"

namespace spork {
namespace {

__device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};        // device address of `scratch`, per device
size_t g_clean[kMaxDevices] = {};      // leading scratch bytes known to be zero, per device

}  // namespace

hipError_t scratch_acquire(size_t control_bytes, hipStream_t stream, void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_ptr[dev] == nullptr) {
    // Once per device, with that device current: the host-side name of the
    // array is no device address; look the address up and use only it.
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_ptr[dev] = p;
    g_clean[dev] = 0;
  }
  // A call needs its control words zero. Every call leaves its own zero, and
  // the bytes after them hold its partial results: when a call needs more
  // control words than the previous one left zero, clear them first (a
  // kernel on the caller's stream, so it stays in stream order).
  if (control_bytes > g_clean[dev]) {
    e = launch_counter_reset(static_cast<int32_t*>(g_ptr[dev]), static_cast<int32_t>(control_bytes / 4), stream);
    if (e != hipSuccess) return e;
  }
  g_clean[dev] = control_bytes;
  *ptr = g_ptr[dev];
  return hipSuccess;
}

}  // namespace spork

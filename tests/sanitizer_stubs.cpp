// Kernel launchers for the host-sanitizer build of the library (tests only):
// the C ABI, block manager and planner are compiled with AddressSanitizer
// and UBSan by g++, and every launch fails loudly instead of reaching a GPU.
#include <hip/hip_runtime_api.h>

#include "ceiling_kernels.h"
#include "kernels.h"
#include "ngram_kernels.h"
#include "noalloc.h"
#include "vocab_kernels.h"

namespace spork {

hipError_t launch_attn_partial(const AttnArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_counter_reset(int32_t*, int32_t, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_merge(const AttnArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_argmax(const AcceptArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_accept_tail(const AcceptArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_image_patch(int32_t*, const ImagePatch&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_kv_write(int32_t, int32_t, int32_t, int32_t, int64_t, void*, void*, const int64_t*, const void*,
                           const void*, int32_t, int32_t*, hipStream_t) {
  return hipErrorNoDevice;
}
hipError_t launch_kv_copy(int32_t, int32_t, int32_t, int32_t, void*, void*, int32_t, int32_t, int32_t, hipStream_t) {
  return hipErrorNoDevice;
}
hipError_t launch_read_ceiling(const void*, int64_t, int32_t, int32_t, uint32_t*, hipStream_t) {
  return hipErrorNoDevice;
}
hipError_t launch_conf_chunks(const ConfArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_conf_final(const ConfArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_ngram_scan(const NgramArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_ngram_drafts(const NgramArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t scratch_acquire(size_t, hipStream_t, void**) { return hipErrorNoDevice; }

}  // namespace spork

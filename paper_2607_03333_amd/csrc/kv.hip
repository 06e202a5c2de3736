// gfx950 setup kernels: token scatter into the paged KV pools and the block
// copy of copy-on-write (Section 4.1). Not on the timed path.
#include "device_common.h"

namespace spork {
namespace {

// --------------------------------------------------------------------------
// Setup kernels.
// --------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256) kv_write_kernel(int hkv, int D, int BS, int64_t num_slots, T* kc,
                                                       T* vc, const int64_t* slots, const T* kn,
                                                       const T* vn, int n, int* bad) {
  constexpr int VEC = 16 / sizeof(T);
  const int per_tok = hkv * (D / VEC);
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= static_cast<int64_t>(n) * per_tok) return;
  const int i = static_cast<int>(idx / per_tok);
  const int rem = static_cast<int>(idx % per_tok);
  const int h = rem / (D / VEC), cchunk = rem % (D / VEC);
  const int64_t slot = slots[i];
  if (slot < 0 || slot >= num_slots) {
    if (rem == 0 && bad != nullptr) atomicAdd(bad, 1);
    return;
  }
  const int64_t b = slot / BS, off = slot % BS;
  const size_t src = (static_cast<size_t>(i) * hkv + h) * D + static_cast<size_t>(cchunk) * VEC;
  *reinterpret_cast<uint4*>(kc + ((static_cast<size_t>(b) * hkv + h) * BS + off) * D + cchunk * VEC) =
      *reinterpret_cast<const uint4*>(kn + src);
  const T* vs = vn + src;
  T* vd = vc + (static_cast<size_t>(b) * hkv + h) * static_cast<size_t>(D) * BS + off;
#pragma unroll
  for (int e = 0; e < VEC; ++e) vd[static_cast<size_t>(cchunk * VEC + e) * BS] = vs[e];
}

template <typename T>
__global__ void __launch_bounds__(256) kv_copy_kernel(int hkv, int D, int BS, T* kc, T* vc, int src, int dst,
                                                      int nv) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= static_cast<int64_t>(hkv) * nv * D) return;
  const int h = static_cast<int>(idx / (static_cast<int64_t>(nv) * D));
  const int rem = static_cast<int>(idx % (static_cast<int64_t>(nv) * D));
  const int off = rem / D, d = rem % D;
  const size_t ks = ((static_cast<size_t>(src) * hkv + h) * BS + off) * D + d;
  const size_t kd = ((static_cast<size_t>(dst) * hkv + h) * BS + off) * D + d;
  kc[kd] = kc[ks];
  const size_t vs = ((static_cast<size_t>(src) * hkv + h) * D + d) * BS + off;
  const size_t vd = ((static_cast<size_t>(dst) * hkv + h) * D + d) * BS + off;
  vc[vd] = vc[vs];
}

// Word writes into a plan's device image (spork_plan_advance): the patch
// travels as the kernel's argument, so nothing is copied from the host.
__global__ void __launch_bounds__(256) image_patch_kernel(int32_t* image, ImagePatch patch) {
  for (int i = threadIdx.x; i < patch.n; i += 256) image[patch.off[i]] = patch.val[i];
}

}  // namespace

hipError_t launch_image_patch(int32_t* image, const ImagePatch& patch, hipStream_t stream) {
  if (patch.n <= 0) return hipSuccess;
  hipLaunchKernelGGL(image_patch_kernel, dim3(1), dim3(256), 0, stream, image, patch);
  return hipGetLastError();
}

hipError_t launch_kv_write(int32_t dtype, int32_t hkv, int32_t head_dim, int32_t block_size,
                           int64_t num_slots, void* k_cache, void* v_cache, const int64_t* slots,
                           const void* k_new, const void* v_new, int32_t n, int32_t* bad_slots,
                           hipStream_t stream) {
  if (n == 0) return hipSuccess;
  const int vec = dtype == 1 ? 8 : 4;
  const int64_t total = static_cast<int64_t>(n) * hkv * (head_dim / vec);
  const dim3 grid(static_cast<unsigned>((total + 255) / 256));
  if (dtype == 1)
    hipLaunchKernelGGL(kv_write_kernel<uint16_t>, grid, dim3(256), 0, stream, hkv, head_dim, block_size, num_slots,
                       static_cast<uint16_t*>(k_cache), static_cast<uint16_t*>(v_cache), slots,
                       static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new), n, bad_slots);
  else
    hipLaunchKernelGGL(kv_write_kernel<float>, grid, dim3(256), 0, stream, hkv, head_dim, block_size, num_slots,
                       static_cast<float*>(k_cache), static_cast<float*>(v_cache), slots,
                       static_cast<const float*>(k_new), static_cast<const float*>(v_new), n, bad_slots);
  return hipGetLastError();
}

hipError_t launch_kv_copy(int32_t dtype, int32_t hkv, int32_t head_dim, int32_t block_size,
                          void* k_cache, void* v_cache, int32_t src, int32_t dst, int32_t n_valid,
                          hipStream_t stream) {
  if (n_valid == 0) return hipSuccess;
  const int64_t total = static_cast<int64_t>(hkv) * n_valid * head_dim;
  const dim3 grid(static_cast<unsigned>((total + 255) / 256));
  if (dtype == 1)
    hipLaunchKernelGGL(kv_copy_kernel<uint16_t>, grid, dim3(256), 0, stream, hkv, head_dim, block_size,
                       static_cast<uint16_t*>(k_cache), static_cast<uint16_t*>(v_cache), src, dst, n_valid);
  else
    hipLaunchKernelGGL(kv_copy_kernel<float>, grid, dim3(256), 0, stream, hkv, head_dim, block_size,
                       static_cast<float*>(k_cache), static_cast<float*>(v_cache), src, dst, n_valid);
  return hipGetLastError();
}

}  // namespace spork

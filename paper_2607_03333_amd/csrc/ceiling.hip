// Streaming-read ceiling of the HBM: plain kernels that only read a buffer,
// run beside the attention launch to state how much of the device's read
// bandwidth the attention stream reaches (a measurement aid, not part of the
// method).
//
//  * mode 0 / 2: register loads (2: non-temporal). Workgroup b reads its
//    contiguous share of the buffer with 16-byte vector loads, 8 in flight
//    per thread, and folds them with XOR into one word per thread (written
//    out, so no load is dead).
//  * mode 1: direct-to-LDS loads, the attention kernel's stream without its
//    arithmetic: 4 waves, a ring of 4 LDS slots of 16 KB, each wave issuing
//    4 global_load_lds_dwordx4 per slot, 3 slots in flight, one barrier per
//    slot. mode 3: the same with non-temporal loads.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "ceiling_kernels.h"

namespace spork {
namespace {

typedef __attribute__((address_space(3))) void* lds_void_ptr;
typedef __attribute__((address_space(1))) void* global_void_ptr;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <bool kNT>
__global__ void __launch_bounds__(256) read_regs(const uint4* __restrict__ src, int64_t n16, uint32_t* sink) {
  const int64_t lo = n16 * blockIdx.x / gridDim.x, hi = n16 * (blockIdx.x + 1) / gridDim.x;
  uint32_t acc = 0;
  int64_t i = lo + threadIdx.x;
  for (; i + 7 * 256 < hi; i += 8 * 256) {
    const u32x4* s4 = reinterpret_cast<const u32x4*>(src);
    u32x4 v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = kNT ? __builtin_nontemporal_load(s4 + i + k * 256) : s4[i + k * 256];
#pragma unroll
    for (int k = 0; k < 8; ++k) acc ^= v[k][0] ^ v[k][1] ^ v[k][2] ^ v[k][3];
  }
  for (; i < hi; i += 256) {
    const uint4 v = src[i];
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  sink[static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x] = acc;
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// 16 KB slots of 1024 16-byte chunks; wave w fills chunks (4w + k) * 64 + lane.
// kAux: the loads' cache-policy bits (2 = non-temporal).
template <int kAux>
__global__ void __launch_bounds__(256, 2) read_lds(const uint4* __restrict__ src, int64_t n16, uint32_t* sink) {
  constexpr int kRing = 4, kSlot = 1024;
  __shared__ uint4 ring[kRing][kSlot];
  const int64_t lo = n16 * blockIdx.x / gridDim.x / kSlot * kSlot;
  const int64_t hi = blockIdx.x + 1 == gridDim.x ? n16 / kSlot * kSlot : n16 * (blockIdx.x + 1) / gridDim.x / kSlot * kSlot;
  const int nst = static_cast<int>((hi - lo) / kSlot);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  auto issue = [&](int st) __attribute__((always_inline)) {
    const uint4* s = src + lo + static_cast<int64_t>(st) * kSlot;
    uint4* d = ring[st % kRing];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int c = (4 * wave + k) * 64;
      __builtin_amdgcn_global_load_lds((global_void_ptr)(s + c + lane), (lds_void_ptr)(d + c), 16, 0, kAux);
    }
  };
  for (int st = 0; st < kRing - 1 && st < nst; ++st) issue(st);
  for (int st = 0; st < nst; ++st) {
    const int after = nst - 1 - st < kRing - 2 ? nst - 1 - st : kRing - 2;
    if (after >= 2) wait_vmcnt<8>();
    else if (after == 1) wait_vmcnt<4>();
    else wait_vmcnt<0>();
    __syncthreads();
    if (st + kRing - 1 < nst) issue(st + kRing - 1);
  }
  wait_vmcnt<0>();
  __syncthreads();
  const uint4 v = ring[0][threadIdx.x];
  sink[static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x] = v.x ^ v.y ^ v.z ^ v.w;
}

}  // namespace

hipError_t launch_read_ceiling(const void* src, int64_t bytes, int32_t grid, int32_t mode, uint32_t* sink,
                               hipStream_t stream) {
  const int64_t n16 = bytes / 16;
  if (mode == 0)
    hipLaunchKernelGGL(read_regs<false>, dim3(grid), dim3(256), 0, stream, static_cast<const uint4*>(src), n16, sink);
  else if (mode == 2)
    hipLaunchKernelGGL(read_regs<true>, dim3(grid), dim3(256), 0, stream, static_cast<const uint4*>(src), n16, sink);
  else if (mode == 3)
    hipLaunchKernelGGL(read_lds<2>, dim3(grid), dim3(256), 0, stream, static_cast<const uint4*>(src), n16, sink);
  else
    hipLaunchKernelGGL(read_lds<0>, dim3(grid), dim3(256), 0, stream, static_cast<const uint4*>(src), n16, sink);
  return hipGetLastError();
}

}  // namespace spork

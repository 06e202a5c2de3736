// Device helpers shared by the gfx950 kernels: vector types, the fast
// base-2 exponential, DPP wave reductions, and the accept of a verify thread
// (run by the accept kernel and inside the merge launch).
#pragma once
#include <hip/hip_runtime.h>

#include <climits>
#include <cstdint>
#include <type_traits>

#include "kernels.h"

namespace spork {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kLn2 = 0.693147180559945309f;
constexpr float kLog2e = 1.442695040888963407f;

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// --------------------------------------------------------------------------
// Wave-wide reductions with DPP: butterflies inside each 16-lane row
// (quad permutes, half-row and row mirrors), then the row broadcasts 15 and
// 31 carry the partial results across rows; lane 63 ends with the total.
// --------------------------------------------------------------------------
template <int kCtrl, int kRowMask>
__device__ __forceinline__ float dpp_mov(float ident, float x) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, ident), __builtin_bit_cast(int, x),
                                         kCtrl, kRowMask, 0xF, false));
}

template <typename Op>
__device__ __forceinline__ float wave_reduce(float x, float ident, Op op) {
  x = op(x, dpp_mov<0xB1, 0xF>(ident, x));   // quad_perm [1,0,3,2]
  x = op(x, dpp_mov<0x4E, 0xF>(ident, x));   // quad_perm [2,3,0,1]
  x = op(x, dpp_mov<0x141, 0xF>(ident, x));  // row_half_mirror
  x = op(x, dpp_mov<0x140, 0xF>(ident, x));  // row_mirror
  x = op(x, dpp_mov<0x142, 0xA>(ident, x));  // row_bcast:15 into rows 1 and 3
  x = op(x, dpp_mov<0x143, 0xC>(ident, x));  // row_bcast:31 into rows 2 and 3
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 63));
}

__device__ __forceinline__ float wave_max(float x) {
  return wave_reduce(x, kNegInf, [](float a, float b) { return fmaxf(a, b); });
}
__device__ __forceinline__ float wave_sum(float x) {
  return wave_reduce(x, 0.0f, [](float a, float b) { return a + b; });
}

__device__ __forceinline__ int wave_min_int(int x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = min(x, __shfl_xor(x, o));
  return x;
}

// Accept for verify thread s, run by one wave: combine the chunk keys of its
// K+1 rows (lane r handles rows r, r+64, ...), then the first draft that
// differs from the greedy token ends the accepted prefix (a ballot per 64 rows).
__device__ __forceinline__ int greedy_of(const AcceptArgs& a, int row) {
  const uint64_t* kp = a.keys + static_cast<size_t>(row) * a.chunks;
  uint64_t best = 0;
  for (int c = 0; c < a.chunks; ++c) best = kp[c] > best ? kp[c] : best;
  return static_cast<int>(0xFFFFFFFFu - static_cast<uint32_t>(best));
}

__device__ __forceinline__ void accept_unit(const AcceptArgs& a, int s) {
  const int lane = threadIdx.x & 63, kd = a.k_drafts;
  int first = kd;
  for (int base = 0; base <= kd; base += 64) {
    const int r = base + lane;
    bool miss = false;
    if (r <= kd) {
      const int g = greedy_of(a, s * (kd + 1) + r);
      if (a.argmax_out != nullptr) a.argmax_out[s * (kd + 1) + r] = g;
      miss = r < kd && g != a.drafts[static_cast<size_t>(s) * kd + r];
    }
    const uint64_t bal = __ballot(miss);
    if (bal != 0 && first == kd) first = base + __builtin_ctzll(bal);
  }
  if (lane == 0) {
    a.accept_len[s] = first;
    a.next_token[s] = greedy_of(a, s * (kd + 1) + first);
  }
}

}  // namespace
}  // namespace spork

// Device helpers shared by the gfx950 kernels: vector types, the fast
// base-2 exponential, DPP reductions over eight lanes, the greedy argmax of a
// vocabulary chunk, and the accept of a verify thread (run by the accept
// kernel and inside the merge launch).
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
// Reductions over lanes 0-7 of a wave with DPP lane moves (no LDS round
// trip): the quad permutes [1,0,3,2] and [2,3,0,1] combine each group of four
// lanes, the half-row mirror (lane i <-> 7 - i inside each eight) combines
// the two groups; lane 0 then holds the result over lanes 0-7, read out as a
// wave-uniform value. Every lane of the wave must be active.
// --------------------------------------------------------------------------
template <int kCtrl>
__device__ __forceinline__ float dpp_mov(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), kCtrl, 0xF, 0xF, false));
}

template <typename Op>
__device__ __forceinline__ float lanes8_reduce(float x, Op op) {
  x = op(x, dpp_mov<0xB1>(x));   // quad_perm [1,0,3,2]
  x = op(x, dpp_mov<0x4E>(x));   // quad_perm [2,3,0,1]
  x = op(x, dpp_mov<0x141>(x));  // row_half_mirror
  return __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, x)));
}

__device__ __forceinline__ float lanes8_max(float x) {
  return lanes8_reduce(x, [](float a, float b) { return fmaxf(a, b); });
}
__device__ __forceinline__ float lanes8_sum(float x) {
  return lanes8_reduce(x, [](float a, float b) { return a + b; });
}

__device__ __forceinline__ int wave_min_int(int x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = min(x, __shfl_xor(x, o));
  return x;
}

// --------------------------------------------------------------------------
// Greedy argmax, first pass: the best (value, index) of one chunk of a row.
// Each thread scans its elements in increasing index order keeping the first
// strict maximum; chunks and threads combine through the 64-bit key
// (order-preserving value bits << 32) | (0xFFFFFFFF - index), whose maximum
// is the largest value at the lowest index. -0 is keyed as +0.
// --------------------------------------------------------------------------
__device__ __forceinline__ uint64_t argmax_key(float v, int idx) {
  if (idx == INT_MAX) return 0;
  uint32_t u = __float_as_uint(v == 0.0f ? 0.0f : v);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return (static_cast<uint64_t>(u) << 32) | (0xFFFFFFFFu - static_cast<uint32_t>(idx));
}

__device__ __forceinline__ float load_f(const float* p, int i) { return p[i]; }
__device__ __forceinline__ float load_f(const uint16_t* p, int i) {
  return __uint_as_float(static_cast<uint32_t>(p[i]) << 16);
}

// Online (max, sum of 2^((x - max) log2 e)) of a set of logits; an empty set
// or one holding only -inf is (-inf, 0).
struct MaxSum {
  float m = kNegInf, s = 0.0f;
  __device__ __forceinline__ void add_max(float nm, float terms_at_nm) {
    // fold in terms already scaled to a maximum nm >= this->m
    s = nm == kNegInf ? 0.0f : s * exp2_fast((m - nm) * kLog2e) + terms_at_nm;
    m = nm;
  }
  __device__ __forceinline__ void combine(float om, float os) {
    const float nm = fmaxf(m, om);
    s = nm == kNegInf ? 0.0f : s * exp2_fast((m - nm) * kLog2e) + os * exp2_fast((om - nm) * kLog2e);
    m = nm;
  }
};

// One (row, chunk) unit run by a workgroup of NT threads over the row's
// logits x: writes the chunk's argmax key to *key_out and, with kSum, the
// chunk's MaxSum to *ms_out.
template <typename T, int NT, bool kSum>
__device__ __forceinline__ void argmax_unit(const T* x, int vocab, int chunks, int c, uint64_t* key_out,
                                            float2* ms_out) {
  constexpr int VEC = 16 / sizeof(T);
  constexpr int NW = NT / 64;
  float best = kNegInf;
  int bidx = INT_MAX;
  MaxSum acc;
  const bool vec_ok = (vocab % VEC) == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0;
  if (vec_ok) {
    const int nv = vocab / VEC;
    const int lo = static_cast<int>(static_cast<int64_t>(nv) * c / chunks);
    const int hi = static_cast<int>(static_cast<int64_t>(nv) * (c + 1) / chunks);
    const uint4* xv = reinterpret_cast<const uint4*>(x);
    auto scan = [&](const uint4& u, int v) __attribute__((always_inline)) {
      const T* e = reinterpret_cast<const T*>(&u);
#pragma unroll
      for (int j = 0; j < VEC; ++j) {
        const float val = load_f(e, j);
        if (val > best || bidx == INT_MAX) {
          best = val;
          bidx = v * VEC + j;
        }
      }
      if constexpr (kSum) {
        float vm = load_f(e, 0);
#pragma unroll
        for (int j = 1; j < VEC; ++j) vm = fmaxf(vm, load_f(e, j));
        const float nm = fmaxf(acc.m, vm);
        float t = 0.0f;
#pragma unroll
        for (int j = 0; j < VEC; ++j) t += exp2_fast((load_f(e, j) - nm) * kLog2e);
        acc.add_max(nm, t);
      }
    };
    // four 16-byte loads in flight per thread, scanned in index order
    int v = lo + static_cast<int>(threadIdx.x);
    for (; v + 3 * NT < hi; v += 4 * NT) {
      const uint4 u0 = xv[v], u1 = xv[v + NT], u2 = xv[v + 2 * NT], u3 = xv[v + 3 * NT];
      scan(u0, v);
      scan(u1, v + NT);
      scan(u2, v + 2 * NT);
      scan(u3, v + 3 * NT);
    }
    for (; v < hi; v += NT) scan(xv[v], v);
  } else {
    const int lo = static_cast<int>(static_cast<int64_t>(vocab) * c / chunks);
    const int hi = static_cast<int>(static_cast<int64_t>(vocab) * (c + 1) / chunks);
    for (int i = lo + static_cast<int>(threadIdx.x); i < hi; i += NT) {
      const float val = load_f(x, i);
      if (val > best || bidx == INT_MAX) {
        best = val;
        bidx = i;
      }
      if constexpr (kSum) {
        const float nm = fmaxf(acc.m, val);
        acc.add_max(nm, exp2_fast((val - nm) * kLog2e));
      }
    }
  }
  uint64_t key = argmax_key(best, bidx);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const uint64_t other = __shfl_xor(key, o);
    key = other > key ? other : key;
    if constexpr (kSum) acc.combine(__shfl_xor(acc.m, o), __shfl_xor(acc.s, o));
  }
  if constexpr (NW > 1) {
    __shared__ uint64_t wk[NW];
    __shared__ float2 wms[NW];
    if ((threadIdx.x & 63) == 0) {
      wk[threadIdx.x >> 6] = key;
      if constexpr (kSum) wms[threadIdx.x >> 6] = make_float2(acc.m, acc.s);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      uint64_t k = wk[0];
      for (int i = 1; i < NW; ++i) k = wk[i] > k ? wk[i] : k;
      *key_out = k;
      if constexpr (kSum) {
        MaxSum t;
        t.m = wms[0].x;
        t.s = wms[0].y;
        for (int i = 1; i < NW; ++i) t.combine(wms[i].x, wms[i].y);
        *ms_out = make_float2(t.m, t.s);
      }
    }
  } else {
    if (threadIdx.x == 0) {
      *key_out = key;
      if constexpr (kSum) *ms_out = make_float2(acc.m, acc.s);
    }
  }
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

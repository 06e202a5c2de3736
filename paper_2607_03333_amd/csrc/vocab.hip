// gfx950 kernels over the vocabulary.
//
//  * argmax_chunks + accept: greedy token of every verify row (lowest index of
//    the row maximum) and the longest draft prefix equal to the greedy tokens
//    (Section 4.3, steps 2-3).
//  * conf_chunks + conf_final: top-1 log-probability of every probe position
//    and the D2 confidence gate over each tool-name span (Section 4.2).
#include "device_common.h"
#include "vocab_kernels.h"

namespace spork {
namespace {

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

template <typename T>
__global__ void __launch_bounds__(256) argmax_chunks(AcceptArgs a) {
  if (a.counters != nullptr)
    for (int i = blockIdx.x * 256 + threadIdx.x; i < a.n_counters; i += gridDim.x * 256) a.counters[i] = 0;
  const int row = blockIdx.x / a.chunks, c = blockIdx.x % a.chunks;
  argmax_unit<T, 256, false>(static_cast<const T*>(a.logits) + static_cast<size_t>(row) * a.vocab, a.vocab, a.chunks,
                             c, a.keys + static_cast<size_t>(row) * a.chunks + c, nullptr);
}

__global__ void __launch_bounds__(64) accept_kernel(AcceptArgs a) { accept_unit(a, blockIdx.x); }

// --------------------------------------------------------------------------
// D2 confidence. conf_chunks: per (row, chunk) the argmax key and the MaxSum.
// conf_final: the first ceil(n_rows / 64) single-wave blocks write each row's
// greedy token and top-1 log-probability l = -ln(sum over chunks of
// s_c 2^((m_c - M) log2 e)), M the row maximum (the greedy token's logit);
// the remaining n_probes blocks take, one wave per probe, the minimum l over
// the span's rows after its first, its exponential (1 for an empty set) and
// the gate. Span offsets are clamped to [0, n_rows]; a reversed span is empty.
// --------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256) conf_chunks(ConfArgs a) {
  const int row = blockIdx.x / a.chunks, c = blockIdx.x % a.chunks;
  const size_t u = static_cast<size_t>(row) * a.chunks + c;
  argmax_unit<T, 256, true>(static_cast<const T*>(a.logits) + static_cast<size_t>(row) * a.vocab, a.vocab, a.chunks,
                            c, a.keys + u, reinterpret_cast<float2*>(a.ms) + u);
}

__device__ __forceinline__ float row_logprob(const ConfArgs& a, int row, int* greedy) {
  const uint64_t* kp = a.keys + static_cast<size_t>(row) * a.chunks;
  const float2* mp = reinterpret_cast<const float2*>(a.ms) + static_cast<size_t>(row) * a.chunks;
  uint64_t best = 0;
  MaxSum t;
  for (int c = 0; c < a.chunks; ++c) {
    best = kp[c] > best ? kp[c] : best;
    const float2 ms = mp[c];
    t.combine(ms.x, ms.y);
  }
  *greedy = static_cast<int>(0xFFFFFFFFu - static_cast<uint32_t>(best));
  return -logf(t.s);
}

__global__ void __launch_bounds__(64) conf_final(ConfArgs a) {
  const int lane = threadIdx.x;
  const int row_blocks = (a.n_rows + 63) / 64;
  if (static_cast<int>(blockIdx.x) < row_blocks) {
    const int r = blockIdx.x * 64 + lane;
    if (r < a.n_rows) {
      int g;
      const float l = row_logprob(a, r, &g);
      if (a.argmax_out != nullptr) a.argmax_out[r] = g;
      if (a.logprob_out != nullptr) a.logprob_out[r] = l;
    }
    return;
  }
  const int p = blockIdx.x - row_blocks;
  const int lo = min(max(a.span_off[p], 0), a.n_rows);
  const int hi = min(max(a.span_off[p + 1], 0), a.n_rows);
  float lmin = 0.0f;  // l <= 0 for every row, so 0 stands for the empty set
  for (int r = lo + 1 + lane; r < hi; r += 64) {
    int g;
    lmin = fminf(lmin, row_logprob(a, r, &g));
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) lmin = fminf(lmin, __shfl_xor(lmin, o));
  if (lane == 0) {
    const float conf = expf(lmin);
    a.confidence_out[p] = conf;
    if (a.commit_out != nullptr) a.commit_out[p] = conf >= a.theta ? 1 : 0;
  }
}

}  // namespace

int32_t accept_chunks(int32_t rows, int32_t vocab) {
  const int32_t max_chunks = vocab / (256 * 8 * 4) > 1 ? vocab / (256 * 8 * 4) : 1;
  int32_t c = rows > 0 ? (2048 + rows - 1) / rows : 1;
  if (c > max_chunks) c = max_chunks;
  return c < 1 ? 1 : c;
}

hipError_t launch_argmax(const AcceptArgs& a, hipStream_t stream) {
  const int rows = a.n_verify * (a.k_drafts + 1);
  if (rows == 0) return hipSuccess;
  if (a.logits_dtype == 1)
    hipLaunchKernelGGL(argmax_chunks<uint16_t>, dim3(rows * a.chunks), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(argmax_chunks<float>, dim3(rows * a.chunks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_conf_chunks(const ConfArgs& a, hipStream_t stream) {
  if (a.n_rows == 0) return hipSuccess;
  if (a.logits_dtype == 1)
    hipLaunchKernelGGL(conf_chunks<uint16_t>, dim3(a.n_rows * a.chunks), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(conf_chunks<float>, dim3(a.n_rows * a.chunks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_conf_final(const ConfArgs& a, hipStream_t stream) {
  const int blocks = (a.n_rows + 63) / 64 + a.n_probes;
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(conf_final, dim3(blocks), dim3(64), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_accept_tail(const AcceptArgs& a, hipStream_t stream) {
  if (a.n_verify == 0) return hipSuccess;
  hipLaunchKernelGGL(accept_kernel, dim3(a.n_verify), dim3(64), (a.k_drafts + 1) * sizeof(int), stream, a);
  return hipGetLastError();
}

}  // namespace spork

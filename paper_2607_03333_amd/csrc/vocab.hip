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

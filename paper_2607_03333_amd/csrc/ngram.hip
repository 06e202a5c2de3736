// gfx950 kernels of the n-gram (prompt-lookup) draft proposer, the draft
// source of the engine's n-gram speculative decoding that D3's proposer
// wraps (Sections 4.3 and 6.1).
//
// The key is the last n tokens of a sequence of L tokens, n from n_max down
// to n_min; the latest earlier occurrence (with a token after it) of the
// longest key that occurs gives up to k drafts: the tokens that follow it.
// For a position p <= L - 2, m(p) is the length of the common suffix of
// tokens[0..p] and tokens[0..L-1]; an occurrence of the n-token key ends at p
// exactly when m(p) >= n. With m capped at n_max, the longest key that
// occurs is the largest capped m (if it reaches n_min), and its latest
// occurrence the largest p with that value, so one maximum over the 64-bit
// key (capped m << 32) | p decides both.
//
//  * ngram_scan: workgroup (sequence, chunk) computes m(p) over its chunk of
//    positions (one coalesced load per position; a further load per matched
//    token) and writes the chunk's largest key; the last chunk of a sequence
//    runs to its end, whatever its length.
//  * ngram_drafts: one wave per sequence takes the largest key over the
//    chunks and writes the drafts, -1 past the end of the sequence.
#include "device_common.h"
#include "ngram_kernels.h"

namespace spork {
namespace {

__global__ void __launch_bounds__(256) ngram_scan(NgramArgs a) {
  const int s = blockIdx.x / a.n_chunks, c = blockIdx.x % a.n_chunks;
  const int64_t base = a.seq_off[s];
  const int64_t L = a.seq_off[s + 1] - base;
  const int32_t* t = a.tokens + base;
  __shared__ int32_t tail[kNgramMaxN];
  const int tx = static_cast<int>(threadIdx.x);
  if (tx < a.n_max && tx < L) tail[tx] = t[L - 1 - tx];
  __syncthreads();
  uint64_t best = 0;
  const int64_t lo = static_cast<int64_t>(c) * kNgramChunk;
  const int64_t hi = c == a.n_chunks - 1 ? L - 1 : (lo + kNgramChunk < L - 1 ? lo + kNgramChunk : L - 1);
  for (int64_t p = lo + threadIdx.x; p < hi; p += 256) {
    int m = 0;
    while (m < a.n_max && m <= p && t[p - m] == tail[m]) ++m;
    if (m >= a.n_min) {
      const uint64_t key = (static_cast<uint64_t>(m) << 32) | static_cast<uint64_t>(p);
      best = key > best ? key : best;
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const uint64_t other = __shfl_xor(best, o);
    best = other > best ? other : best;
  }
  __shared__ uint64_t wk[4];
  if ((threadIdx.x & 63) == 0) wk[threadIdx.x >> 6] = best;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t k = wk[0];
    for (int i = 1; i < 4; ++i) k = wk[i] > k ? wk[i] : k;
    a.keys[static_cast<size_t>(s) * a.n_chunks + c] = k;
  }
}

__global__ void __launch_bounds__(64) ngram_drafts(NgramArgs a) {
  const int s = blockIdx.x, lane = threadIdx.x;
  uint64_t best = 0;
  for (int c = lane; c < a.n_chunks; c += 64) {
    const uint64_t k = a.keys[static_cast<size_t>(s) * a.n_chunks + c];
    best = k > best ? k : best;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const uint64_t other = __shfl_xor(best, o);
    best = other > best ? other : best;
  }
  const int64_t base = a.seq_off[s];
  const int64_t L = a.seq_off[s + 1] - base;
  const int64_t p = static_cast<int64_t>(best & 0xFFFFFFFFu);
  // drafts available after the occurrence: tokens p+1 .. L-1
  const int64_t avail = best == 0 ? 0 : L - 1 - p;
  const int cnt = static_cast<int>(avail < a.k ? avail : a.k);
  for (int i = lane; i < a.k; i += 64)
    a.drafts[static_cast<size_t>(s) * a.k + i] = i < cnt ? a.tokens[base + p + 1 + i] : -1;
  if (lane == 0) a.n_drafts[s] = cnt;
}

}  // namespace

hipError_t launch_ngram_scan(const NgramArgs& a, hipStream_t stream) {
  if (a.n_seqs == 0) return hipSuccess;
  hipLaunchKernelGGL(ngram_scan, dim3(a.n_seqs * a.n_chunks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_ngram_drafts(const NgramArgs& a, hipStream_t stream) {
  if (a.n_seqs == 0) return hipSuccess;
  hipLaunchKernelGGL(ngram_drafts, dim3(a.n_seqs), dim3(64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace spork

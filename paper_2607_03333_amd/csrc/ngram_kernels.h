// Launch interface of the n-gram (prompt-lookup) draft proposer.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>

namespace spork {

constexpr int32_t kNgramChunk = 2048;  // positions one workgroup scans
constexpr int32_t kNgramMaxN = 32;     // longest lookup key

struct NgramArgs {
  const int32_t* tokens;   // all sequences, concatenated
  const int64_t* seq_off;  // [n_seqs + 1] offsets into tokens
  int32_t n_seqs, n_chunks, n_min, n_max, k;
  uint64_t* keys;          // [n_seqs][n_chunks] workspace
  int32_t* drafts;         // [n_seqs][k]
  int32_t* n_drafts;       // [n_seqs]
};

// chunks per sequence for sequences of at most max_len tokens (longer ones
// are still scanned whole, by their last chunk's workgroup)
int32_t ngram_chunks(int64_t max_len);
hipError_t launch_ngram_scan(const NgramArgs& a, hipStream_t stream);
hipError_t launch_ngram_drafts(const NgramArgs& a, hipStream_t stream);

}  // namespace spork

// Launch interface of the vocabulary kernels that are not part of the
// attention and verify launches.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>

namespace spork {

// D2 confidence over a logits matrix [n_rows][vocab] and probe spans.
struct ConfArgs {
  const void* logits;
  int32_t logits_dtype, vocab, n_rows, chunks, n_probes;
  const int32_t* span_off;  // [n_probes + 1]
  float theta;
  int32_t* argmax_out;      // [n_rows], nullable
  float* logprob_out;       // [n_rows], nullable
  float* confidence_out;    // [n_probes]
  int32_t* commit_out;      // [n_probes], nullable
  uint64_t* keys;           // [n_rows][chunks] workspace
  float* ms;                // [n_rows][chunks][2] workspace: chunk max, sum of 2^((x - max) log2 e)
};

hipError_t launch_conf_chunks(const ConfArgs& a, hipStream_t stream);
hipError_t launch_conf_final(const ConfArgs& a, hipStream_t stream);

}  // namespace spork

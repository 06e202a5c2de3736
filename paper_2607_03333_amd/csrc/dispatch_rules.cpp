// Host-side sizing and dispatch rules shared by the C ABI and the kernel
// launchers: which attention shapes have a kernel, and how many chunks the
// vocabulary and n-gram passes split a row or sequence into.
#include <cstdint>

#include "kernels.h"
#include "ngram_kernels.h"

namespace spork {

// bf16: head_dim 128, 16- or 32-token blocks, workgroups of 4 or 8 waves with
// one or two row tiles per wave; fp32: head_dim 64 or 128, 16- or 32-token
// blocks, one wave with up to 4 row tiles. The kernel table in
// attention.hip instantiates exactly these.
bool attention_supported(int32_t dtype, int32_t head_dim, int32_t block_size, int32_t row_tiles, int32_t waves) {
  if (row_tiles < 1 || (block_size != 16 && block_size != 32)) return false;
  if (dtype == 1) {
    if (head_dim != 128 || (waves != 4 && waves != 8)) return false;
    const int32_t per_wave = (row_tiles + waves - 1) / waves;
    return per_wave >= 1 && per_wave <= 2;
  }
  if (dtype == 0) return (head_dim == 64 || head_dim == 128) && row_tiles <= 4;
  return false;
}

// Vocabulary chunks per logits row: enough (row, chunk) units for about
// 2048 workgroups, each chunk at least 8 16-byte loads per thread of a
// 256-thread workgroup.
int32_t accept_chunks(int32_t rows, int32_t vocab) {
  const int32_t max_chunks = vocab / (256 * 8 * 4) > 1 ? vocab / (256 * 8 * 4) : 1;
  int32_t c = rows > 0 ? (2048 + rows - 1) / rows : 1;
  if (c > max_chunks) c = max_chunks;
  return c < 1 ? 1 : c;
}

int32_t ngram_chunks(int64_t max_len) {
  const int64_t c = (max_len + kNgramChunk - 1) / kNgramChunk;
  return static_cast<int32_t>(c < 1 ? 1 : c);
}

}  // namespace spork

// Launch interface between the C ABI layer and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstddef>
#include <cstdint>

#include "plan_types.h"

namespace spork {

struct AcceptArgs {
  const void* logits;
  int32_t logits_dtype, vocab, n_verify, k_drafts, chunks;
  const int32_t* drafts;
  int32_t* accept_len;
  int32_t* next_token;
  int32_t* argmax_out;
  uint64_t* keys;  // [rows][chunks] workspace
  // nullable: int32 counters of the attention launch that follows, which the
  // argmax launch clears
  int32_t* counters;
  int32_t n_counters;
};

struct AttnArgs {
  const WaveDesc* waves;
  const ItemDesc* items;
  const RowDesc* rows;
  const int32_t* tables;
  const int32_t* merge_off;
  const int32_t* part_slot;  // merge position of each unit row's partial result
  // Unit lists (CSR over waves): the bf16 kernel's workgroup b takes the units
  // of list b % n_lists in order, through cursors[list] (zero before the launch).
  const int32_t* wg_off;
  int32_t* cursors;
  int32_t n_units, grid, n_lists, n_out, row_tiles;
  // waves of a bf16 workgroup: 4 (two persistent workgroups per compute unit,
  // up to 8 row tiles each) or 8 (one per compute unit, up to 16)
  int32_t wg_waves;
  int32_t hq, hkv, head_dim, block_size, dtype;
  float scale_log2;  // sm_scale * log2(e): scores are kept in base 2
  const void* q;
  const void* k_cache;
  const void* v_cache;
  void* out;
  float* lse;
  // [n_partials][head_dim] unnormalised partial outputs in the input dtype;
  // bf16 rows hold their channels in the bf16 writer's register order (see
  // the merge in attention.hip), fp32 rows in channel order.
  void* part_o;
  float* part_ml;  // [n_partials][2] running max (base 2) and sum
  // Verify step: accept units appended to the merge grid (acc.n_verify of them).
  AcceptArgs acc;
  // Argmax units (row x vocabulary chunk) the persistent bf16 launch works
  // through after its lists, through cursors[n_lists]; 0 when the argmax has
  // a launch of its own.
  int32_t tail_units;
  // Cursors the merge launch returns to zero for the next call (the
  // persistent launch's n_lists + 1; 0 otherwise).
  int32_t n_cursors;
};

// true if a kernel exists for this (dtype, head_dim, block_size, row_tiles)
bool attention_supported(int32_t dtype, int32_t head_dim, int32_t block_size, int32_t row_tiles, int32_t waves);
hipError_t launch_attn_partial(const AttnArgs& a, hipStream_t stream);
// zero n int32 words (a workspace's control words)
hipError_t launch_counter_reset(int32_t* counters, int32_t n, hipStream_t stream);
// log-sum-exp merge (+ accept of a.acc.n_verify verify threads)
hipError_t launch_merge(const AttnArgs& a, hipStream_t stream);


int32_t accept_chunks(int32_t rows, int32_t vocab);
hipError_t launch_argmax(const AcceptArgs& a, hipStream_t stream);
hipError_t launch_accept_tail(const AcceptArgs& a, hipStream_t stream);

// Up to kPatchMax word writes (word offset, value) into a plan's device
// image, carried in the kernel argument (under 4 KB).
constexpr int kPatchMax = 480;
struct ImagePatch {
  int32_t n;
  int32_t off[kPatchMax];
  int32_t val[kPatchMax];
};
hipError_t launch_image_patch(int32_t* image, const ImagePatch& patch, hipStream_t stream);

hipError_t launch_kv_write(int32_t dtype, int32_t hkv, int32_t head_dim, int32_t block_size,
                           int64_t num_slots, void* k_cache, void* v_cache, const int64_t* slots,
                           const void* k_new, const void* v_new, int32_t n, int32_t* bad_slots,
                           hipStream_t stream);
hipError_t launch_kv_copy(int32_t dtype, int32_t hkv, int32_t head_dim, int32_t block_size,
                          void* k_cache, void* v_cache, int32_t src, int32_t dst, int32_t n_valid,
                          hipStream_t stream);

}  // namespace spork

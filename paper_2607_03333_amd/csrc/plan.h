// Host planner: turns a batch of forked threads into the attention work list.
//
// Threads of one fork group share the longest common prefix of their block
// tables (capped so that every row may see all of it); that prefix is one
// work item per KV head whose rows are all members' rows, so its KV is read
// once per group. Each thread's remaining positions form its own item. Items
// are cut into work units (token range x row slice, split-K) on lists of
// near-equal cost, one per compute unit, and every output row lists the
// partial results the log-sum-exp merge combines.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "block_manager.h"
#include "plan_types.h"

namespace spork {

struct PlanShape {
  int32_t hq, hkv, head_dim, block_size, elem_bytes;
  int32_t unit_tiles_max;  // 16-row tiles one attention workgroup can hold
  int32_t units_per_cu;    // attention workgroups resident per compute unit
  int32_t units_per_cu_half;  // the same when every workgroup needs at most half the tiles
  bool persistent;         // resident workgroups each work through a list of units
  int32_t waves;           // waves per workgroup (bf16: 4 or 8; fp32: 1)
};

struct Plan {
  PlanShape shape{};
  int32_t n_threads = 0, n_rows = 0, n_groups = 0, n_items = 0;
  int32_t n_units = 0, grid = 0, n_partials = 0, row_tiles = 1, n_out = 0;
  int32_t n_lists = 0;  // unit lists (persistent launch: one per compute unit)
  int32_t max_range_tiles = 0;  // 16-row tiles of the largest range's row set, before slicing
  int64_t shared_tokens = 0, private_tokens = 0, flat_tokens = 0;
  // device image: sections at 256-byte aligned byte offsets
  std::vector<uint8_t> image;
  size_t off_waves = 0, off_items = 0, off_rows = 0, off_tables = 0, off_merge_off = 0,
         off_part_slot = 0, off_wg_off = 0;
  // Workspace: control words first (zero between calls: the list cursors of
  // a persistent launch), then the partial outputs (in the input dtype) and
  // their (m, l) pairs.
  size_t workspace_bytes = 0;
  size_t control_bytes = 0;
  int32_t n_cursors = 0;       // n_lists + 1 for a persistent launch, else 0
  size_t off_ws_cursors = 0;   // byte offsets inside the workspace
  size_t off_ws_o = 0;
  size_t off_ws_ml = 0;
  // What a later decode step needs to reuse the plan (spork_plan_advance):
  std::vector<int32_t> seqs, len;              // each thread's sequence and its length when planned
  std::vector<int32_t> grow;                   // tokens appended since, as last written into the image
  std::vector<std::vector<int32_t>> thread_items;  // the items of each thread's private range
  std::vector<std::vector<int32_t>> thread_table;  // each copied table as planned and patched since
  std::vector<int32_t> thread_table_off;       // its offset in the image's table area, -1 if not copied
  std::vector<int32_t> thread_table_cap;       // entries the image holds for it (planned + kTableReserve)
  std::vector<int32_t> open_units;             // units that end where their private range ends
};

// Block-table entries the bf16 kernel stages for a unit [tok_lo, tok_hi).
int32_t unit_table_span(int32_t tok_lo, int32_t tok_hi, int32_t block_size);

// Returns "" on success, else an error message (nothing is built).
std::string build_plan(const BlockManager& bm, const PlanShape& shape, const int32_t* seqs,
                       const int32_t* n_rows, const int32_t* groups, int32_t n_threads,
                       int32_t n_cu, Plan* out);

}  // namespace spork

// Work descriptors shared by the host planner and the device kernels.
#pragma once
#include <cstdint>

namespace spork {

// One attention work unit: a token range of one work item and a slice of the
// item's query rows. item < 0 marks padding that is skipped. (The bf16 kernel
// runs units on 4-wave workgroups, the fp32 kernel on 1-wave workgroups.)
struct WaveDesc {
  int32_t item;
  int32_t tok_lo;   // first context position of the range
  int32_t tok_hi;   // one past the last position
  int32_t row0;     // first row of the slice inside the item's row list
  int32_t nrows;    // rows in the slice (<= 16 * row tiles of the kernel)
  int32_t partial;  // first partial-result row this workgroup writes
};

// A (prefix or private) context range of one KV head and the rows reading it.
struct ItemDesc {
  int32_t kv_head;
  int32_t table_off;  // offset of the block table in the image's table area
  int32_t n_blocks;   // valid entries of that table when the plan was made
  int32_t row_off;    // offset of the item's rows in the row area
  int32_t n_rows;
  int32_t hi;         // end of the item's range when the plan was made
  // Tokens appended to the item's thread since the plan was made (a private
  // range reused by later decode steps; always 0 for shared ranges): the
  // range's last unit ends `grow` tokens later, its rows' horizons move by
  // `grow`, and its table holds the blocks of hi + grow tokens.
  int32_t grow;
  int32_t thread;     // the thread of a private range, -1 for a shared one
};

// One query row of an item: output index (query row * Hq + query head) and
// the last context position it may attend to.
struct RowDesc {
  int32_t qidx;
  int32_t horizon;
};

constexpr int kTileTokens = 32;   // tokens per inner-loop tile
// Longest token range of one work unit: its block-table slice (at most
// (kMaxUnitTokens + 3 * 32) / 16 + 1 entries for 16-token blocks) is staged
// in a 1040-entry LDS table by the bf16 kernel.
constexpr int kMaxUnitTokens = 16384;
// Upper bound of the shortest piece the planner cuts from a longer range, and
// the start-up cost of a unit in tokens of streaming (per-unit loads of the
// query rows and block table, and the refill of the load pipeline), used to
// balance the workgroups' lists. The start-up takes scalar descriptor loads
// and lets the query rows complete behind the first stage's loads, so 128
// balances better than 256 on small batches and costs nothing on large ones
// (measured).
constexpr int kMinPieceTokens = 512;
constexpr int kUnitOverheadTokens = 128;
// Ints between two unit-list cursors in the workspace: one 256-byte line
// each. Device-scope atomics on words that share a line serialize; with the
// cursors a line apart a contended take returns about 1.5 times sooner
// (measured with 512 workgroups).
constexpr int kCursorStride = 64;
constexpr int kXcds = 8;          // MI355X: 8 accelerator dies, workgroups dealt round-robin
// Block-table entries the image keeps free after each thread's table, for
// the blocks later decode steps append (see spork_plan_advance).
constexpr int kTableReserve = 64;
// Block-table entries of one unit's slice that the bf16 kernel stages in LDS.
constexpr int kUnitTableEntries = 1040;

}  // namespace spork

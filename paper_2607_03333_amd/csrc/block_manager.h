// Host block manager: reference-counted block tables with copy-on-write, the
// mechanism behind SPORK's prefix-cache fork (design D1, Section 4.1): a probe
// forked from the main thread reads the main thread's prefix KV in place.
//
// Allocation rule: a FIFO free queue seeded by the caller; a token that starts
// a block takes the queue front; the first token written into a partially
// filled block that another sequence references copies it first (the copy
// target is taken before any new block); freeing a sequence releases its
// entries in table order to the queue back. Failed appends change nothing.
#pragma once

#include <cstdint>
#include <deque>
#include <string>
#include <unordered_map>
#include <unordered_set>
#include <vector>

namespace spork {

struct CowCopy {
  int32_t src = -1, dst = -1, n_valid = 0;
};

enum class BmStatus { kOk, kUnknownSeq, kBadArg, kNoBlocks };

class BlockManager {
 public:
  BlockManager(int32_t num_blocks, int32_t block_size, const int32_t* free_order);

  int32_t num_blocks() const { return num_blocks_; }
  int32_t block_size() const { return block_size_; }

  int32_t seq_new();
  BmStatus append(int32_t seq, int32_t n, int64_t* slots, CowCopy* cow, int32_t* n_cow);
  // Appends to several distinct sequences, in order, exactly as the single
  // appends would run; all or nothing (the blocks needed are counted first,
  // copies that an earlier append of the batch makes unnecessary included).
  // slots: sum of n[i] entries in batch order; cows: up to k entries, *n_cows set.
  BmStatus append_batch(const int32_t* seqs, const int32_t* n, int32_t k, int64_t* slots, CowCopy* cows,
                        int32_t* n_cows);
  BmStatus fork(int32_t parent, int32_t* child);
  BmStatus free_seq(int32_t seq);

  bool has(int32_t seq) const { return seqs_.count(seq) != 0; }
  const std::vector<int32_t>& table(int32_t seq) const { return seqs_.at(seq).table; }
  int32_t length(int32_t seq) const { return seqs_.at(seq).length; }
  int32_t refcount(int32_t block) const { return ref_[block]; }
  const std::deque<int32_t>& free_queue() const { return free_; }

 private:
  struct Seq {
    std::vector<int32_t> table;
    int32_t length = 0;
  };
  int32_t take_block();

  int32_t num_blocks_, block_size_;
  std::deque<int32_t> free_;
  std::vector<int32_t> ref_;
  std::unordered_map<int32_t, Seq> seqs_;
  int32_t next_id_ = 0;
};

}  // namespace spork

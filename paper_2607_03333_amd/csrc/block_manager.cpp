#include "block_manager.h"

#include <unordered_map>
#include <unordered_set>

namespace spork {

BlockManager::BlockManager(int32_t num_blocks, int32_t block_size, const int32_t* free_order)
    : num_blocks_(num_blocks), block_size_(block_size), ref_(num_blocks, 0) {
  for (int32_t i = 0; i < num_blocks; ++i) free_.push_back(free_order ? free_order[i] : i);
}

int32_t BlockManager::seq_new() {
  const int32_t id = next_id_++;
  seqs_.emplace(id, Seq{});
  return id;
}

int32_t BlockManager::take_block() {
  const int32_t b = free_.front();
  free_.pop_front();
  ref_[b] = 1;
  return b;
}

BmStatus BlockManager::append(int32_t seq, int32_t n, int64_t* slots, CowCopy* cow, int32_t* n_cow) {
  auto it = seqs_.find(seq);
  if (it == seqs_.end()) return BmStatus::kUnknownSeq;
  if (n < 0) return BmStatus::kBadArg;
  Seq& s = it->second;
  const int32_t bs = block_size_;
  *n_cow = 0;
  if (n == 0) return BmStatus::kOk;
  // Blocks this append takes from the queue: one copy target when the tail
  // block is partially filled and shared, plus one per token that opens a block.
  const bool copy_tail = (s.length % bs) != 0 && ref_[s.table.back()] > 1;
  const int64_t first_new = (static_cast<int64_t>(s.length) + bs - 1) / bs;  // blocks in use
  const int64_t last_new = (static_cast<int64_t>(s.length) + n + bs - 1) / bs;
  const int64_t need = (last_new - first_new) + (copy_tail ? 1 : 0);
  if (need > static_cast<int64_t>(free_.size())) return BmStatus::kNoBlocks;
  if (copy_tail) {
    const int32_t src = s.table.back();
    const int32_t dst = take_block();
    ref_[src] -= 1;
    s.table.back() = dst;
    cow->src = src;
    cow->dst = dst;
    cow->n_valid = s.length % bs;
    *n_cow = 1;
  }
  for (int32_t i = 0; i < n; ++i) {
    const int32_t pos = s.length + i;
    if (pos % bs == 0) s.table.push_back(take_block());
    slots[i] = static_cast<int64_t>(s.table[pos / bs]) * bs + pos % bs;
  }
  s.length += n;
  return BmStatus::kOk;
}

BmStatus BlockManager::append_batch(const int32_t* seqs, const int32_t* n, int32_t k, int64_t* slots, CowCopy* cows,
                                    int32_t* n_cows) {
  *n_cows = 0;
  if (k < 0) return BmStatus::kBadArg;
  const int32_t bs = block_size_;
  std::unordered_set<int32_t> seen;
  std::unordered_map<int32_t, int32_t> dref;  // tail blocks released by earlier copies of this batch
  int64_t need = 0;
  for (int32_t i = 0; i < k; ++i) {
    auto it = seqs_.find(seqs[i]);
    if (it == seqs_.end()) return BmStatus::kUnknownSeq;
    if (n[i] < 0 || !seen.insert(seqs[i]).second) return BmStatus::kBadArg;
    if (n[i] == 0) continue;
    const Seq& s = it->second;
    if (s.length % bs != 0) {
      const int32_t tail = s.table.back();
      if (ref_[tail] + dref[tail] > 1) {
        need += 1;
        dref[tail] -= 1;
      }
    }
    need += (static_cast<int64_t>(s.length) + n[i] + bs - 1) / bs - (static_cast<int64_t>(s.length) + bs - 1) / bs;
  }
  if (need > static_cast<int64_t>(free_.size())) return BmStatus::kNoBlocks;
  int64_t at = 0;
  for (int32_t i = 0; i < k; ++i) {
    CowCopy cow;
    int32_t nc = 0;
    const BmStatus st = append(seqs[i], n[i], slots + at, &cow, &nc);
    if (st != BmStatus::kOk) return st;  // not reached: the batch was counted above
    if (nc) cows[(*n_cows)++] = cow;
    at += n[i];
  }
  return BmStatus::kOk;
}

BmStatus BlockManager::fork(int32_t parent, int32_t* child) {
  auto it = seqs_.find(parent);
  if (it == seqs_.end()) return BmStatus::kUnknownSeq;
  Seq copy = it->second;
  for (int32_t b : copy.table) ref_[b] += 1;
  const int32_t id = next_id_++;
  seqs_.emplace(id, std::move(copy));
  *child = id;
  return BmStatus::kOk;
}

BmStatus BlockManager::free_seq(int32_t seq) {
  auto it = seqs_.find(seq);
  if (it == seqs_.end()) return BmStatus::kUnknownSeq;
  for (int32_t b : it->second.table) {
    if (--ref_[b] == 0) free_.push_back(b);
  }
  seqs_.erase(it);
  return BmStatus::kOk;
}

}  // namespace spork

// Host-side bookkeeping of the streamed paged KV cache (the inference side of
// KV-streams, Section 2 "KV-streams" and Section 4 "Inference engine
// implementation"): cache blocks of block_size slots, a free list, and per
// sequence the list of its blocks in allocation order.  Tokens are appended
// at the tail of a sequence's last block; evicted entries are dropped for
// good (their slots are never refilled) and a block returns to the free list
// once none of its entries is live.  The device side (slot contents and the
// live marks read by the decode kernel) is updated by the caller with the
// slot lists these calls return.
#include "kvs_cache.h"

#include <algorithm>
#include <cstdio>
#include <unordered_set>

namespace kvs {

BlockManager::BlockManager(int num_blocks, int block_size, int num_seqs, int max_blocks)
    : nb_(num_blocks), bs_(block_size), ns_(num_seqs), mb_(max_blocks),
      blocks_(num_seqs), tail_fill_(num_seqs, block_size), live_(num_blocks, 0), slot_of_(num_seqs) {
  free_.reserve(num_blocks);
  for (int b = num_blocks - 1; b >= 0; --b) free_.push_back(b);   // block 0 is handed out first
}

static int fail_msg(std::string* err, int code, const char* msg, long long a = 0) {
  if (err) {
    char buf[256];
    snprintf(buf, sizeof(buf), msg, a);
    *err = buf;
  }
  return code;
}

int BlockManager::append(int seq, const int32_t* pos, int n, int32_t* slots, std::string* err) {
  if (seq < 0 || seq >= ns_) return fail_msg(err, kBadArg, "sequence index %lld out of range", seq);
  auto& map = slot_of_[seq];
  std::unordered_set<int> seen;
  for (int i = 0; i < n; ++i) {
    if (pos[i] < 0) return fail_msg(err, kBadArg, "negative trace position %lld", pos[i]);
    if (map.count(pos[i]) || !seen.insert(pos[i]).second)
      return fail_msg(err, kBadState, "trace position %lld is already in the cache", pos[i]);
  }
  // blocks this append needs, checked before anything changes
  const int room = bs_ - tail_fill_[seq];
  const long long need = n > room ? (n - room + bs_ - 1) / bs_ : 0;
  if (need > (long long)free_.size()) return fail_msg(err, kCapacity, "out of cache blocks (%lld more needed)", need);
  if ((long long)blocks_[seq].size() + need > mb_)
    return fail_msg(err, kCapacity, "sequence would hold more than max_blocks (%lld) blocks", mb_);
  for (int i = 0; i < n; ++i) {
    if (tail_fill_[seq] == bs_) {
      blocks_[seq].push_back(free_.back());
      free_.pop_back();
      tail_fill_[seq] = 0;
    }
    const int blk = blocks_[seq].back();
    const int slot = blk * bs_ + tail_fill_[seq]++;
    ++live_[blk];
    map[pos[i]] = slot;
    slots[i] = slot;
  }
  return kOk;
}

void BlockManager::drop_block(int seq, int blk) {
  auto& bl = blocks_[seq];
  const bool tail = !bl.empty() && bl.back() == blk;
  bl.erase(std::find(bl.begin(), bl.end(), blk));
  free_.push_back(blk);
  if (tail) tail_fill_[seq] = bs_;   // the next append opens a new block
}

int BlockManager::evict(int seq, const int32_t* pos, int n, int32_t* slots, std::string* err) {
  if (seq < 0 || seq >= ns_) return fail_msg(err, kBadArg, "sequence index %lld out of range", seq);
  auto& map = slot_of_[seq];
  std::unordered_set<int> seen;
  for (int i = 0; i < n; ++i) {
    if (!map.count(pos[i])) return fail_msg(err, kBadState, "trace position %lld is not in the cache", pos[i]);
    if (!seen.insert(pos[i]).second) return fail_msg(err, kBadState, "trace position %lld evicted twice", pos[i]);
  }
  for (int i = 0; i < n; ++i) {
    auto it = map.find(pos[i]);
    const int slot = it->second;
    map.erase(it);
    slots[i] = slot;
    const int blk = slot / bs_;
    if (--live_[blk] == 0) drop_block(seq, blk);
  }
  return kOk;
}

int BlockManager::release(int seq, int32_t* slots, int* n_slots, std::string* err) {
  if (seq < 0 || seq >= ns_) return fail_msg(err, kBadArg, "sequence index %lld out of range", seq);
  int k = 0;
  for (const auto& kv : slot_of_[seq]) slots[k++] = kv.second;
  std::sort(slots, slots + k);
  *n_slots = k;
  slot_of_[seq].clear();
  for (int blk : blocks_[seq]) {
    live_[blk] = 0;
    free_.push_back(blk);
  }
  blocks_[seq].clear();
  tail_fill_[seq] = bs_;
  return kOk;
}

void BlockManager::tables(int32_t* block_table, int32_t* seq_blocks) const {
  for (int s = 0; s < ns_; ++s) {
    const auto& bl = blocks_[s];
    seq_blocks[s] = (int32_t)bl.size();
    for (int i = 0; i < mb_; ++i) block_table[(size_t)s * mb_ + i] = i < (int)bl.size() ? bl[i] : 0;
  }
}

int BlockManager::live(int seq) const {
  return (seq >= 0 && seq < ns_) ? (int)slot_of_[seq].size() : -1;
}

}  // namespace kvs

// Internal interface of the host-side block manager of the streamed paged KV
// cache (kvs_cache.cpp).  Not part of the public ABI; the C entry points in
// kvs_api.cpp wrap it.
#pragma once

#include <stdint.h>

#include <string>
#include <unordered_map>
#include <vector>

namespace kvs {

class BlockManager {
 public:
  enum { kOk = 0, kBadArg = 1, kBadState = 2, kCapacity = 3 };

  BlockManager(int num_blocks, int block_size, int num_seqs, int max_blocks);

  // Slots for n new tokens of sequence seq at trace positions pos[0..n)
  // (all-or-nothing: on error nothing changes).
  int append(int seq, const int32_t* pos, int n, int32_t* slots, std::string* err);
  // Evict the entries at trace positions pos[0..n) (all-or-nothing); writes
  // their slots.  Blocks left with no live entry return to the free list.
  int evict(int seq, const int32_t* pos, int n, int32_t* slots, std::string* err);
  // Drop the whole sequence; writes its live slots (sorted) and their count.
  int release(int seq, int32_t* slots, int* n_slots, std::string* err);
  // block_table [num_seqs][max_blocks] (unused entries 0), seq_blocks [num_seqs].
  void tables(int32_t* block_table, int32_t* seq_blocks) const;
  int free_blocks() const { return (int)free_.size(); }
  int live(int seq) const;

  int num_blocks() const { return nb_; }
  int block_size() const { return bs_; }
  int num_seqs() const { return ns_; }
  int max_blocks() const { return mb_; }

 private:
  void drop_block(int seq, int blk);

  int nb_, bs_, ns_, mb_;
  std::vector<int> free_;                               // free block ids (LIFO)
  std::vector<std::vector<int>> blocks_;                // per sequence, allocation order
  std::vector<int> tail_fill_;                          // per sequence: used slots of its last block
  std::vector<int> live_;                               // per block: live entries
  std::vector<std::unordered_map<int, int>> slot_of_;   // per sequence: trace position -> slot
};

}  // namespace kvs

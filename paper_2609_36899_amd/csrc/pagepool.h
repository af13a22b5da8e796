// Host-side page pool, resident-set table and attention work planner.
//
// Pure C++ (no HIP): it compiles with g++ into a host-only test library as
// well as into the device library.  It owns the bookkeeping of the paged KV
// cache: which physical page holds which 16-token block of which sequence,
// the free list, reservations, and sequence ids with generation counters.
#pragma once

#include <stdint.h>

#include <string>
#include <vector>

#include "meta.h"

namespace pdec {

struct Status {
  int code = 0;
  std::string msg;
  static Status ok() { return {}; }
  static Status err(int c, std::string m) { return {c, std::move(m)}; }
  bool good() const { return code == 0; }
};

class PagePool {
 public:
  PagePool(int32_t n_pages, int32_t max_seqs, int32_t max_seq_len);

  int32_t n_pages() const { return n_pages_; }
  int32_t max_seqs() const { return max_seqs_; }
  int32_t max_seq_len() const { return max_seq_len_; }
  int32_t max_pages_per_seq() const { return max_pages_per_seq_; }
  int64_t free_pages() const { return (int64_t)free_.size(); }
  int64_t headroom_tokens() const { return free_pages() * kPage; }

  // Admit an empty sequence with ceil(reserve_tokens/16) reserved pages.
  Status alloc_seq(int32_t reserve_tokens, int32_t* id_out);
  // Departure: return every page of the sequence to the free list.
  Status free_seq(int32_t id);
  // Resolve an id to its slot; BAD_SEQ if unknown or stale.
  Status resolve(int32_t id, int32_t* slot) const;

  bool live(int32_t slot) const { return slot >= 0 && slot < max_seqs_ && seqs_[slot].live; }
  int32_t len(int32_t slot) const { return seqs_[slot].len; }
  const std::vector<int32_t>& pages(int32_t slot) const { return seqs_[slot].pages; }

  // Record of one grow() call, enough to take it back.
  struct GrowUndo {
    std::vector<int32_t> slots, old_len, old_npages;
    size_t old_pending = 0;
  };

  // Make room for `extra` more tokens on each listed slot and advance the
  // lengths.  All-or-nothing: on failure nothing changes.  The block-table
  // entries of newly attached pages are appended to the pending list.
  Status grow(const int32_t* slots, int32_t n, int32_t extra, GrowUndo* undo = nullptr);
  // The same with its own count per slot: slot slots[i] grows by extras[i].
  Status grow_each(const int32_t* slots, int32_t n, const int32_t* extras,
                   GrowUndo* undo = nullptr);
  // Take back a successful grow() (used when enqueueing device work fails,
  // before any other call changes the pool).
  void undo(const GrowUndo& u);

  // Block-table entries written on the host but not yet on the device, in
  // the order they were made.  No (slot, idx) appears twice: the device
  // writes them all in parallel.
  const std::vector<BtDelta>& pending() const { return pending_; }
  void clear_pending() { pending_.clear(); }

  // Pages needed to hold `tokens` tokens.
  static int32_t pages_for(int64_t tokens) { return (int32_t)((tokens + kPage - 1) / kPage); }

 private:
  struct Seq {
    bool live = false;
    int32_t gen = 0;
    int32_t len = 0;
    std::vector<int32_t> pages;  // logical order; may exceed pages_for(len) (reserve)
  };
  int32_t make_id(int32_t slot) const { return (seqs_[slot].gen << 16) | slot; }

  int32_t n_pages_, max_seqs_, max_seq_len_, max_pages_per_seq_;
  std::vector<int32_t> free_;        // stack of free page ids
  std::vector<int32_t> free_slots_;  // stack of free sequence slots
  std::vector<Seq> seqs_;
  std::vector<BtDelta> pending_;
};

// Query block description given to the planner.
struct QBlockSpec {
  int32_t q_row0, n_q, slot, pos0;
};

// Work groups the attention split pass aims for (four waves each).  Decode:
// six per CU, i.e. two rounds at the kernel's three resident groups per CU;
// measured against 1024..8192 on the 8B decode shapes (B = 8..256), fewer
// groups leave long-context batches unbalanced and more groups pay the
// per-item query load, partial write and combine.
constexpr int64_t kDecodeTargetGroups = 1536;
// Prefill: two per CU.  A prefill item's partial is 64-128 rows x (Dh + 2)
// floats, written and read back once per item, so fewer, longer items save
// that traffic while the MFMA-bound split pass still fills the GPU; measured
// against 1024..4096 on 8B-shaped re-prefill (4K-64K tokens) and tool-output
// appends (1-3% faster than 1024-2048, 8% faster than 4096).
constexpr int64_t kPrefillTargetGroups = 512;

// Items per KV head the planner aims for.
int64_t attn_target_items(int32_t n_kv_heads, int64_t target_groups = kDecodeTargetGroups);

// Split size (in pages, even, at least 8) for a key-axis workload of
// `total_pages` (summed over query blocks): the item count stays within
// attn_target_items(n_kv_heads, target_groups) plus one per query block.
int32_t choose_split_pages(int64_t total_pages, int32_t n_kv_heads,
                           int64_t target_groups = kDecodeTargetGroups);

// Cut every query block's key range [0, pos0 + n_q) into items of
// `split_pages` pages.  Fills qblocks (with item ranges) and items, and sets
// the dispatch order of the items (longest first, ties in item order).
void plan_attention(const std::vector<QBlockSpec>& specs, int32_t split_pages,
                    std::vector<AttnQBlock>* qblocks, std::vector<AttnItem>* items);

// Total pages touched by the query blocks (the key-axis workload).
int64_t total_key_pages(const std::vector<QBlockSpec>& specs);

// Bounds of one forward pass, checked on the host before any launch: every
// row's slot is a sequence slot and its position lies inside the sequence
// and the rotary table; every query block's rows lie inside the pass and its
// items inside the block's key range and the block-table row; every item
// belongs to its block; the dispatch order is a permutation; and each block
// covers its keys exactly once.  `pool` (nullable) adds: the slot is live,
// the block's keys are within the sequence length, and every page the block
// reads is one the sequence holds and below the pool size.
Status validate_pass(const std::vector<RowMeta>& rows, const std::vector<AttnQBlock>& qblocks,
                     const std::vector<AttnItem>& items, int32_t max_seqs, int32_t max_seq_len,
                     int32_t bt_stride, const PagePool* pool);

// Pending block-table entries: slots, indexes and pages in range, and no
// (slot, idx) twice.
Status validate_deltas(const std::vector<BtDelta>& d, int32_t max_seqs, int32_t bt_stride,
                       int32_t n_pages);

}  // namespace pdec

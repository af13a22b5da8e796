// Per-call metadata that the host planner builds and the kernels read.
//
// Plain structs with fixed sizes: the host packs them into one staging
// buffer and a single host-to-device copy moves them per call.
#pragma once

#include <stdint.h>

namespace pdec {

constexpr int kPage = 16;  // tokens per KV page

// One row of the activation matrix (one token being processed).
struct RowMeta {
  int32_t slot;  // sequence slot = row of the device block table
  int32_t pos;   // position of this token in its sequence
};

// A block of consecutive query rows (tokens) of one sequence that share
// attention work items: 1 token in decode; in prefill up to R / G tokens,
// G the GQA group and R the kernel's rows per item (128 or 256 with 128-dim
// heads, 64 with 64-dim heads), each token contributing G (token, head) rows.
struct AttnQBlock {
  int32_t q_row0;      // first activation row of the block
  int32_t n_q;         // rows in the block
  int32_t slot;        // sequence slot
  int32_t pos0;        // position of the first row; row j sits at pos0 + j
  int32_t item_begin;  // work items of this block: [item_begin, item_end)
  int32_t item_end;
  int32_t pad0, pad1;
};

// A contiguous range of logical pages of one query block (a split of the
// key axis).  Keys of the range are positions [16*page_begin, 16*(page_begin+n_pages)).
struct AttnItem {
  int32_t qblock;
  int32_t page_begin;
  int32_t n_pages;
  // Dispatch order: grid slot d processes item items[d].order.  The planner
  // orders items longest first so the short ones fill the tail of the grid.
  int32_t order;
};

// A block-table entry to write on the device: bt[slot][idx] = page.
struct BtDelta {
  int32_t slot;
  int32_t idx;
  int32_t page;
  int32_t pad;
};

}  // namespace pdec

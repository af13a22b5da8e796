#include "pagepool.h"

#include <algorithm>
#include <unordered_set>

#include "../../include/pdec.h"

namespace pdec {

PagePool::PagePool(int32_t n_pages, int32_t max_seqs, int32_t max_seq_len)
    : n_pages_(n_pages), max_seqs_(max_seqs), max_seq_len_(max_seq_len) {
  max_pages_per_seq_ = pages_for(max_seq_len);
  free_.resize(n_pages);
  // Stack top is the end: hand out page 0 first.
  for (int32_t i = 0; i < n_pages; ++i) free_[i] = n_pages - 1 - i;
  seqs_.resize(max_seqs);
  free_slots_.resize(max_seqs);
  for (int32_t i = 0; i < max_seqs; ++i) free_slots_[i] = max_seqs - 1 - i;
}

Status PagePool::resolve(int32_t id, int32_t* slot) const {
  if (id < 0) return Status::err(PDEC_BAD_SEQ, "negative sequence id");
  int32_t s = id & 0xFFFF;
  if (s >= max_seqs_ || !seqs_[s].live || make_id(s) != id)
    return Status::err(PDEC_BAD_SEQ, "unknown or stale sequence id " + std::to_string(id));
  *slot = s;
  return Status::ok();
}

Status PagePool::alloc_seq(int32_t reserve_tokens, int32_t* id_out) {
  if (reserve_tokens < 0 || reserve_tokens > max_seq_len_)
    return Status::err(PDEC_INVALID_ARG, "reserve_tokens outside [0, max_seq_len]");
  if (free_slots_.empty()) return Status::err(PDEC_INVALID_ARG, "no free sequence slot");
  int32_t need = pages_for(reserve_tokens);
  if ((int64_t)need > free_pages())
    return Status::err(PDEC_OUT_OF_PAGES, "reserve needs " + std::to_string(need) +
                                              " pages, " + std::to_string(free_pages()) +
                                              " free");
  int32_t s = free_slots_.back();
  free_slots_.pop_back();
  Seq& q = seqs_[s];
  q.live = true;
  q.len = 0;
  q.pages.clear();
  for (int32_t i = 0; i < need; ++i) {
    q.pages.push_back(free_.back());
    free_.pop_back();
    pending_.push_back({s, i, q.pages.back(), 0});
  }
  *id_out = make_id(s);
  return Status::ok();
}

Status PagePool::free_seq(int32_t id) {
  int32_t s;
  Status st = resolve(id, &s);
  if (!st.good()) return st;
  Seq& q = seqs_[s];
  for (auto it = q.pages.rbegin(); it != q.pages.rend(); ++it) free_.push_back(*it);
  // The slot's block-table entries that have not reached the device yet
  // describe pages it no longer holds.  They must go: the device applies all
  // pending entries at once and in no order, so an old entry (slot, idx)
  // left beside the next occupant's entry for the same (slot, idx) could win
  // and point that occupant at a page another sequence now owns.  Every
  // index the next occupant uses gets a fresh entry when it attaches a page.
  pending_.erase(std::remove_if(pending_.begin(), pending_.end(),
                                [s](const BtDelta& d) { return d.slot == s; }),
                 pending_.end());
  q.pages.clear();
  q.len = 0;
  q.live = false;
  q.gen = (q.gen + 1) & 0x7FFF;
  free_slots_.push_back(s);
  return Status::ok();
}

Status PagePool::grow(const int32_t* slots, int32_t n, int32_t extra, GrowUndo* undo) {
  std::vector<int32_t> extras((size_t)std::max(n, 0), extra);
  return grow_each(slots, n, extras.data(), undo);
}

Status PagePool::grow_each(const int32_t* slots, int32_t n, const int32_t* extras,
                           GrowUndo* undo) {
  int64_t need = 0;
  for (int32_t i = 0; i < n; ++i) {
    if (extras[i] < 0) return Status::err(PDEC_INVALID_ARG, "negative growth");
    const Seq& q = seqs_[slots[i]];
    int64_t new_len = (int64_t)q.len + extras[i];
    if (new_len > max_seq_len_)
      return Status::err(PDEC_SEQ_TOO_LONG, "sequence would reach " + std::to_string(new_len) +
                                                " tokens, max_seq_len " +
                                                std::to_string(max_seq_len_));
    need += std::max<int64_t>(0, pages_for(new_len) - (int64_t)q.pages.size());
  }
  if (need > free_pages())
    return Status::err(PDEC_OUT_OF_PAGES, "growth needs " + std::to_string(need) + " pages, " +
                                              std::to_string(free_pages()) + " free");
  if (undo) {
    undo->slots.assign(slots, slots + n);
    undo->old_len.resize(n);
    undo->old_npages.resize(n);
    undo->old_pending = pending_.size();
  }
  for (int32_t i = 0; i < n; ++i) {
    Seq& q = seqs_[slots[i]];
    if (undo) {
      undo->old_len[i] = q.len;
      undo->old_npages[i] = (int32_t)q.pages.size();
    }
    q.len += extras[i];
    int32_t want = pages_for(q.len);
    while ((int32_t)q.pages.size() < want) {
      int32_t p = free_.back();
      free_.pop_back();
      q.pages.push_back(p);
      pending_.push_back({slots[i], (int32_t)q.pages.size() - 1, p, 0});
    }
  }
  return Status::ok();
}

void PagePool::undo(const GrowUndo& u) {
  for (size_t i = u.slots.size(); i-- > 0;) {
    Seq& q = seqs_[u.slots[i]];
    while ((int32_t)q.pages.size() > u.old_npages[i]) {
      free_.push_back(q.pages.back());
      q.pages.pop_back();
    }
    q.len = u.old_len[i];
  }
  pending_.resize(std::min(pending_.size(), u.old_pending));
}

int64_t attn_target_items(int32_t n_kv_heads, int64_t target_groups) {
  return std::max<int64_t>(1, target_groups / std::max(1, n_kv_heads));
}

int32_t choose_split_pages(int64_t total_pages, int32_t n_kv_heads, int64_t target_groups) {
  // Enough work groups to keep 256 CUs busy through the tail of the grid,
  // while the per-item fixed cost (query load, partial write) stays small
  // next to the item's KV bytes.
  const int64_t target = attn_target_items(n_kv_heads, target_groups);
  int64_t s = (total_pages + target - 1) / target;
  s = std::max<int64_t>(8, s);
  s = (s + 1) & ~int64_t(1);
  return (int32_t)std::min<int64_t>(s, INT32_MAX - 1);
}

int64_t total_key_pages(const std::vector<QBlockSpec>& specs) {
  int64_t t = 0;
  for (const auto& q : specs) t += PagePool::pages_for((int64_t)q.pos0 + q.n_q);
  return t;
}

void plan_attention(const std::vector<QBlockSpec>& specs, int32_t split_pages,
                    std::vector<AttnQBlock>* qblocks, std::vector<AttnItem>* items) {
  qblocks->clear();
  items->clear();
  for (size_t i = 0; i < specs.size(); ++i) {
    const QBlockSpec& q = specs[i];
    AttnQBlock b{};
    b.q_row0 = q.q_row0;
    b.n_q = q.n_q;
    b.slot = q.slot;
    b.pos0 = q.pos0;
    b.item_begin = (int32_t)items->size();
    int32_t np = PagePool::pages_for((int64_t)q.pos0 + q.n_q);
    for (int32_t p = 0; p < np; p += split_pages)
      items->push_back({(int32_t)i, p, std::min(split_pages, np - p), 0});
    b.item_end = (int32_t)items->size();
    qblocks->push_back(b);
  }
  std::vector<int32_t> ord(items->size());
  for (size_t i = 0; i < ord.size(); ++i) ord[i] = (int32_t)i;
  std::stable_sort(ord.begin(), ord.end(), [&](int32_t a, int32_t b) {
    return (*items)[a].n_pages > (*items)[b].n_pages;
  });
  for (size_t i = 0; i < ord.size(); ++i) (*items)[i].order = ord[i];
}

Status validate_pass(const std::vector<RowMeta>& rows, const std::vector<AttnQBlock>& qblocks,
                     const std::vector<AttnItem>& items, int32_t max_seqs, int32_t max_seq_len,
                     int32_t bt_stride, const PagePool* pool) {
  auto bad = [](const std::string& m) { return Status::err(PDEC_INVALID_ARG, "validate: " + m); };
  const int64_t n_rows = (int64_t)rows.size(), n_items = (int64_t)items.size();
  for (int64_t r = 0; r < n_rows; ++r) {
    const RowMeta& m = rows[r];
    if (m.slot < 0 || m.slot >= max_seqs) return bad("row " + std::to_string(r) + " slot");
    if (m.pos < 0 || m.pos >= max_seq_len) return bad("row " + std::to_string(r) + " position");
    if (pool && (!pool->live(m.slot) || m.pos >= pool->len(m.slot)))
      return bad("row " + std::to_string(r) + " outside its sequence");
  }
  std::vector<char> seen((size_t)n_items, 0);
  for (const AttnItem& it : items) {
    if (it.order < 0 || it.order >= n_items || seen[it.order]) return bad("dispatch order");
    seen[it.order] = 1;
  }
  int64_t next_item = 0;
  for (size_t b = 0; b < qblocks.size(); ++b) {
    const AttnQBlock& q = qblocks[b];
    const std::string tag = "query block " + std::to_string(b);
    if (q.n_q < 1 || q.q_row0 < 0 || (int64_t)q.q_row0 + q.n_q > n_rows) return bad(tag + " rows");
    if (q.slot < 0 || q.slot >= max_seqs || q.pos0 < 0) return bad(tag + " slot or position");
    for (int j = 0; j < q.n_q; ++j) {
      const RowMeta& m = rows[q.q_row0 + j];
      if (m.slot != q.slot || m.pos != q.pos0 + j) return bad(tag + " disagrees with its rows");
    }
    const int64_t key_pages = PagePool::pages_for((int64_t)q.pos0 + q.n_q);
    if (key_pages > bt_stride) return bad(tag + " keys past the block-table row");
    if (q.item_begin != next_item || q.item_end < q.item_begin || q.item_end > n_items)
      return bad(tag + " item range");
    int64_t covered = 0;
    for (int32_t i = q.item_begin; i < q.item_end; ++i) {
      const AttnItem& it = items[i];
      if (it.qblock != (int32_t)b || it.n_pages < 1 || it.page_begin != covered)
        return bad("item " + std::to_string(i) + " of " + tag);
      covered += it.n_pages;
    }
    if (covered != key_pages) return bad(tag + " keys not covered exactly once");
    next_item = q.item_end;
    if (pool) {
      if (!pool->live(q.slot) || (int64_t)q.pos0 + q.n_q > pool->len(q.slot))
        return bad(tag + " reads past its sequence");
      const auto& pg = pool->pages(q.slot);
      if ((int64_t)pg.size() < key_pages) return bad(tag + " reads a page its sequence lacks");
      for (int64_t k = 0; k < key_pages; ++k)
        if (pg[k] < 0 || pg[k] >= pool->n_pages()) return bad(tag + " page id out of range");
    }
  }
  if (next_item != n_items) return bad("items not owned by a query block");
  return Status::ok();
}

Status validate_deltas(const std::vector<BtDelta>& d, int32_t max_seqs, int32_t bt_stride,
                       int32_t n_pages) {
  std::unordered_set<int64_t> keys;
  for (size_t i = 0; i < d.size(); ++i) {
    const BtDelta& e = d[i];
    if (e.slot < 0 || e.slot >= max_seqs || e.idx < 0 || e.idx >= bt_stride || e.page < 0 ||
        e.page >= n_pages)
      return Status::err(PDEC_INVALID_ARG,
                         "validate: block-table entry " + std::to_string(i) + " out of range");
    if (!keys.insert((int64_t)e.slot * bt_stride + e.idx).second)
      return Status::err(PDEC_INVALID_ARG, "validate: block-table entry (" +
                                               std::to_string(e.slot) + ", " +
                                               std::to_string(e.idx) + ") pending twice");
  }
  return Status::ok();
}

}  // namespace pdec

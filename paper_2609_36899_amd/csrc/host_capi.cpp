// Host-only C entry points over the page pool and the attention planner.
//
// Built with g++ into libpdec_host.so so that the bookkeeping half of the
// library (admission, reservation, growth, departure, stale ids, work-list
// planning) is testable on a machine without a GPU.  The device library
// compiles the same pagepool.cpp.
#include <cstring>
#include <string>
#include <vector>

#include "fp8_e4m3.h"
#include "pacing.h"
#include "pagepool.h"

using namespace pdec;

namespace {
thread_local std::string g_err;
int ret(const Status& s) {
  if (!s.good()) g_err = s.msg;
  return s.code;
}
}  // namespace

extern "C" {

const char* pp_last_error(void) { return g_err.c_str(); }

void* pp_create(int32_t n_pages, int32_t max_seqs, int32_t max_seq_len) {
  if (n_pages < 1 || max_seqs < 1 || max_seqs > 65535 || max_seq_len < 1) return nullptr;
  return new PagePool(n_pages, max_seqs, max_seq_len);
}

void pp_destroy(void* p) { delete (PagePool*)p; }

int pp_alloc(void* p, int32_t reserve, int32_t* id) {
  return ret(((PagePool*)p)->alloc_seq(reserve, id));
}

int pp_free(void* p, int32_t id) { return ret(((PagePool*)p)->free_seq(id)); }

int pp_len(void* p, int32_t id, int32_t* len) {
  int32_t slot;
  Status s = ((PagePool*)p)->resolve(id, &slot);
  if (s.good()) *len = ((PagePool*)p)->len(slot);
  return ret(s);
}

int64_t pp_headroom(void* p) { return ((PagePool*)p)->headroom_tokens(); }

// Resolve ids, then grow each by `extra` tokens, all or nothing.  With
// `undo_after` set the growth is taken back again (exercises undo()).
int pp_grow(void* p, const int32_t* ids, int32_t n, int32_t extra, int32_t undo_after) {
  PagePool* pool = (PagePool*)p;
  std::vector<int32_t> slots(n);
  for (int i = 0; i < n; ++i) {
    Status s = pool->resolve(ids[i], &slots[i]);
    if (!s.good()) return ret(s);
  }
  PagePool::GrowUndo u;
  Status s = pool->grow(slots.data(), n, extra, &u);
  if (s.good() && undo_after) pool->undo(u);
  return ret(s);
}

int32_t pp_pages(void* p, int32_t id, int32_t* out, int32_t cap) {
  int32_t slot;
  Status s = ((PagePool*)p)->resolve(id, &slot);
  if (!s.good()) return ret(s);
  const auto& pg = ((PagePool*)p)->pages(slot);
  for (int32_t i = 0; i < (int32_t)pg.size() && i < cap; ++i) out[i] = pg[i];
  return (int32_t)pg.size();
}

int32_t pp_slot(void* p, int32_t id) {
  int32_t slot = -1;
  Status s = ((PagePool*)p)->resolve(id, &slot);
  return s.good() ? slot : ret(s);
}

// Pending block-table entries as (slot, idx, page) triples; returns count.
int32_t pp_pending(void* p, int32_t* out3, int32_t cap) {
  const auto& d = ((PagePool*)p)->pending();
  for (int32_t i = 0; i < (int32_t)d.size() && i < cap; ++i) {
    out3[3 * i] = d[i].slot;
    out3[3 * i + 1] = d[i].idx;
    out3[3 * i + 2] = d[i].page;
  }
  return (int32_t)d.size();
}

void pp_clear_pending(void* p) { ((PagePool*)p)->clear_pending(); }

int32_t pp_choose_split(int64_t total_pages, int32_t n_kv_heads) {
  return choose_split_pages(total_pages, n_kv_heads);
}

int64_t pp_target_items(int32_t n_kv_heads) { return attn_target_items(n_kv_heads); }

// specs: n x (q_row0, n_q, slot, pos0).  Writes qblocks as 6 ints
// (q_row0, n_q, slot, pos0, item_begin, item_end) and items as 4 ints
// (qblock, page_begin, n_pages, order).  Returns the item count (or -1 if the
// item buffer is too small).
int32_t pp_plan(const int32_t* specs, int32_t n, int32_t split, int32_t* qb_out,
                int32_t* items_out, int32_t items_cap) {
  std::vector<QBlockSpec> sp(n);
  for (int i = 0; i < n; ++i)
    sp[i] = {specs[4 * i], specs[4 * i + 1], specs[4 * i + 2], specs[4 * i + 3]};
  std::vector<AttnQBlock> qb;
  std::vector<AttnItem> it;
  plan_attention(sp, split, &qb, &it);
  if ((int32_t)it.size() > items_cap) return -1;
  for (int i = 0; i < n; ++i) {
    const AttnQBlock& b = qb[i];
    const int32_t v[6] = {b.q_row0, b.n_q, b.slot, b.pos0, b.item_begin, b.item_end};
    std::memcpy(qb_out + 6 * i, v, sizeof(v));
  }
  for (size_t i = 0; i < it.size(); ++i) {
    items_out[4 * i] = it[i].qblock;
    items_out[4 * i + 1] = it[i].page_begin;
    items_out[4 * i + 2] = it[i].n_pages;
    items_out[4 * i + 3] = it[i].order;
  }
  return (int32_t)it.size();
}

int64_t pp_total_key_pages(const int32_t* specs, int32_t n) {
  std::vector<QBlockSpec> sp(n);
  for (int i = 0; i < n; ++i)
    sp[i] = {specs[4 * i], specs[4 * i + 1], specs[4 * i + 2], specs[4 * i + 3]};
  return total_key_pages(sp);
}

// Host bounds checks of a pass (validate_pass / validate_deltas), as the
// engine runs them under PDEC_VALIDATE.  rows: n_rows x (slot, pos);
// qblocks: n_qb x (q_row0, n_q, slot, pos0, item_begin, item_end); items:
// n_items x (qblock, page_begin, n_pages, order); pool (nullable) adds the
// checks against live sequences and their pages.  Returns 0 or an error code
// (pp_last_error names the failed check).
int pp_validate_pass(void* pool, const int32_t* rows, int32_t n_rows, const int32_t* qblocks,
                     int32_t n_qb, const int32_t* items, int32_t n_items, int32_t max_seqs,
                     int32_t max_seq_len, int32_t bt_stride) {
  std::vector<RowMeta> r(n_rows);
  for (int i = 0; i < n_rows; ++i) r[i] = {rows[2 * i], rows[2 * i + 1]};
  std::vector<AttnQBlock> q(n_qb);
  for (int i = 0; i < n_qb; ++i) {
    const int32_t* v = qblocks + 6 * i;
    q[i] = AttnQBlock{v[0], v[1], v[2], v[3], v[4], v[5], 0, 0};
  }
  std::vector<AttnItem> it(n_items);
  for (int i = 0; i < n_items; ++i)
    it[i] = {items[4 * i], items[4 * i + 1], items[4 * i + 2], items[4 * i + 3]};
  return ret(validate_pass(r, q, it, max_seqs, max_seq_len, bt_stride, (const PagePool*)pool));
}

// deltas: n x (slot, idx, page).
int pp_validate_deltas(const int32_t* deltas, int32_t n, int32_t max_seqs, int32_t bt_stride,
                       int32_t n_pages) {
  std::vector<BtDelta> d(n);
  for (int i = 0; i < n; ++i) d[i] = {deltas[3 * i], deltas[3 * i + 1], deltas[3 * i + 2], 0};
  return ret(validate_deltas(d, max_seqs, bt_stride, n_pages));
}

// E4M3 codes of n floats, as the fp8 KV page writes compute them.
void pp_e4m3_encode(const float* x, uint8_t* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = (uint8_t)e4m3_from_f32(x[i]);
}

// Pacing decision (the same code the device library exports as pacing_plan).
int32_t pp_pacing_plan(int64_t headroom, int64_t h_min, int64_t delta, int32_t n_active,
                       const int32_t* active_ids, const int32_t* active_len,
                       const int64_t* active_held, int32_t n_pending, const int32_t* pending_ids,
                       const int32_t* pending_len, int32_t* evict_out, int32_t* n_evict,
                       int32_t* place_out, int32_t* n_place) {
  std::vector<PacingResident> act(n_active);
  for (int i = 0; i < n_active; ++i) act[i] = {active_ids[i], active_len[i], active_held[i]};
  std::vector<PacingPending> pend(n_pending);
  for (int i = 0; i < n_pending; ++i) pend[i] = {pending_ids[i], pending_len[i]};
  std::vector<int32_t> ev, pl;
  pacing_plan(headroom, h_min, delta, act, pend, &ev, &pl);
  for (size_t i = 0; i < ev.size(); ++i) evict_out[i] = ev[i];
  for (size_t i = 0; i < pl.size(); ++i) place_out[i] = pl[i];
  *n_evict = (int32_t)ev.size();
  *n_place = (int32_t)pl.size();
  return 0;
}

}  // extern "C"

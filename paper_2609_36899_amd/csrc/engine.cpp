// C ABI of the decode library: engine state, workspace carving, per-call
// planning and the launch sequence of one decoder step.
//
// The engine is one rollout worker's decode backend (paper: Design,
// "Separating Departure from Placement"): it holds the resident set, its
// paged KV cache and the KV headroom, and runs iteration-level token batches
// over any subset of residents.  Host work per call is bookkeeping only
// (lengths, page growth, the attention work list); every step of the
// computation runs in the gfx950 kernels.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/pdec.h"
#include "kernels.h"
#include "pacing.h"
#include "pagepool.h"

using namespace pdec;

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

#define HIP_OR_FAIL(expr)                                                                \
  do {                                                                                   \
    hipError_t e_ = (expr);                                                              \
    if (e_ != hipSuccess)                                                                \
      return fail(PDEC_HIP_ERROR, std::string(#expr) + ": " + hipGetErrorString(e_));    \
  } while (0)

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

int64_t elem_bytes(int32_t dtype) { return dtype == PDEC_BF16 ? 2 : 4; }
int64_t kv_elem_bytes(const pdec_model_cfg* c) { return c->kv_fp8 ? 1 : elem_bytes(c->dtype); }

// ---------------------------------------------------------------------------
// Pinned staging ring for host-to-device metadata copies.
// ---------------------------------------------------------------------------
class Staging {
 public:
  ~Staging() { release(); }
  hipError_t init(size_t slot_bytes, int n_slots) {
    slot_bytes_ = slot_bytes;
    for (int i = 0; i < n_slots; ++i) {
      void* p = nullptr;
      hipError_t e = hipHostMalloc(&p, slot_bytes, hipHostMallocDefault);
      if (e != hipSuccess) return e;
      slots_.push_back(p);
      hipEvent_t ev;
      e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
      if (e != hipSuccess) return e;
      events_.push_back(ev);
      used_.push_back(false);
    }
    return hipSuccess;
  }
  void release() {
    for (size_t i = 0; i < slots_.size(); ++i) {
      if (used_[i]) (void)hipEventSynchronize(events_[i]);
      (void)hipEventDestroy(events_[i]);
      (void)hipHostFree(slots_[i]);
    }
    slots_.clear();
    events_.clear();
    used_.clear();
  }
  size_t slot_bytes() const { return slot_bytes_; }
  // Copies in pieces of at most one slot.
  hipError_t upload(void* dst, const void* src, size_t bytes, hipStream_t s) {
    size_t off = 0;
    while (off < bytes) {
      const size_t n = std::min(slot_bytes_, bytes - off);
      const int k = next_;
      next_ = (next_ + 1) % (int)slots_.size();
      if (used_[k]) {
        hipError_t e = hipEventSynchronize(events_[k]);
        if (e != hipSuccess) return e;
      }
      std::memcpy(slots_[k], (const char*)src + off, n);
      hipError_t e = hipMemcpyAsync((char*)dst + off, slots_[k], n, hipMemcpyHostToDevice, s);
      if (e != hipSuccess) return e;
      e = hipEventRecord(events_[k], s);
      if (e != hipSuccess) return e;
      used_[k] = true;
      off += n;
    }
    return hipSuccess;
  }

 private:
  std::vector<void*> slots_;
  std::vector<hipEvent_t> events_;
  std::vector<bool> used_;
  size_t slot_bytes_ = 0;
  int next_ = 0;
};

// ---------------------------------------------------------------------------
// Optional per-launch timing of chosen launch classes.  The launch records
// the kernel's own begin and end into the pair (see launch_timed), so timing
// adds no marker packets between kernels.
// ---------------------------------------------------------------------------
class LaunchTimer {
 public:
  ~LaunchTimer() { reset_pool(); }
  void enable(uint32_t mask) { mask_ = mask; }
  // Time one launch in every `every` of each selected class.
  void sample(int every) {
    every_ = every;
    for (int64_t& c : count_) c = 0;
  }
  bool on() const { return mask_ != 0; }
  // Events for one launch of class kind, or nulls when it is not timed.
  hipError_t pair(int kind, hipEvent_t* a, hipEvent_t* b) {
    *a = *b = nullptr;
    if (!(mask_ >> kind & 1u)) return hipSuccess;
    if (count_[kind]++ % every_ != 0) return hipSuccess;
    hipEvent_t ea, eb;
    hipError_t e = take(&ea);
    if (e != hipSuccess) return e;
    e = take(&eb);
    if (e != hipSuccess) {
      free_.push_back(ea);
      return e;
    }
    done_.push_back({kind, ea, eb});
    *a = ea;
    *b = eb;
    return hipSuccess;
  }
  // Sum of elapsed times (ms) and launch count of one kind; clears records.
  hipError_t read(int kind, double* ms, int64_t* count) {
    *ms = 0.0;
    *count = 0;
    std::vector<Rec> keep;
    for (const Rec& r : done_) {
      if (r.kind != kind) {
        keep.push_back(r);
        continue;
      }
      hipError_t e = hipEventSynchronize(r.b);
      if (e != hipSuccess) return e;
      float t = 0.f;
      e = hipEventElapsedTime(&t, r.a, r.b);
      if (e != hipSuccess) return e;
      *ms += t;
      *count += 1;
      free_.push_back(r.a);
      free_.push_back(r.b);
    }
    done_.swap(keep);
    return hipSuccess;
  }

 private:
  struct Rec {
    int kind;
    hipEvent_t a, b;
  };
  hipError_t take(hipEvent_t* ev) {
    if (!free_.empty()) {
      *ev = free_.back();
      free_.pop_back();
      return hipSuccess;
    }
    hipError_t e = hipEventCreate(ev);
    if (e == hipSuccess) all_.push_back(*ev);
    return e;
  }
  void reset_pool() {
    for (hipEvent_t e : all_) (void)hipEventDestroy(e);
    all_.clear();
    free_.clear();
    done_.clear();
  }
  uint32_t mask_ = 0;
  int every_ = 1;
  int64_t count_[3] = {0, 0, 0};
  std::vector<Rec> done_;
  std::vector<hipEvent_t> free_, all_;
};

// ---------------------------------------------------------------------------
// Workspace layout.
// ---------------------------------------------------------------------------
struct WsLayout {
  size_t rope, bt, meta, delta, x, h, o, u, q, lmg, part, att_ml, att_acc, total;
  size_t meta_bytes, part_elems, delta_cap;
  int64_t items_cap, qblocks_cap, rows_cap, part_row_slots;
  int32_t bt_stride;
};

constexpr size_t kDeltaCap = 65536;
// Sequence pieces one prefill pass may hold (kv_append_prefix_batch packs
// several sequences' tokens into one pass); also the most LM-head rows a
// prefill pass produces.
constexpr int kMaxPiecesPerPass = 64;
// Query rows per attention work item: decode (one wave) and prefill (four).
constexpr int kDecodeRows = 16;
// Query rows per prefill block: 128 for the LDS-staged prefill kernel (bf16
// activations, 128-dim heads; bf16 or E4M3 pages), 64 for the others.
int prefill_rows(const pdec_model_cfg& c) {
  return (c.dtype == PDEC_BF16 && c.head_dim == 128) ? 128 : 64;
}
// The LDS-staged kernel also takes 256-row blocks (eight waves share each
// stage, halving the load work per flop).  A pass switches to them when its
// 128-row blocks read at least this many key pages each on average (16K
// keys): measured on 4096-row re-prefill passes of the 8B shape, 256-row
// blocks were 2-9% slower at 0-2.5K cached keys, +1.8% at 12K, +3.8% at 28K
// and +10% at 61K.  PDEC_PREFILL_WIDE_PAGES at engine creation overrides it.
constexpr int64_t kWidePrefillPages = 1024;

int check_cfg(const pdec_model_cfg* c) {
  if (!c) return fail(PDEC_INVALID_ARG, "null cfg");
  if (c->n_layers < 1 || c->d_model < 1 || c->n_q_heads < 1 || c->n_kv_heads < 1 ||
      c->head_dim < 1 || c->ffn_dim < 1 || c->vocab < 1)
    return fail(PDEC_INVALID_ARG, "model dimensions must be positive");
  if (c->dtype != PDEC_F32 && c->dtype != PDEC_BF16)
    return fail(PDEC_INVALID_ARG, "dtype must be PDEC_F32 or PDEC_BF16");
  if (!(c->rms_eps >= 0.f) || !(c->rope_base > 0.f))
    return fail(PDEC_INVALID_ARG, "rms_eps must be >= 0 and rope_base > 0");
  if (c->n_q_heads % c->n_kv_heads != 0)
    return fail(PDEC_INVALID_ARG, "n_q_heads must be a multiple of n_kv_heads");
  const int G = c->n_q_heads / c->n_kv_heads;
  // A decode query block is the G query heads of one token: its rows fill
  // part of one 16-row MFMA tile, so groups of up to 16 heads (any size, rows
  // past G masked) are supported.
  if (G > 16) return fail(PDEC_UNSUPPORTED, "GQA group size must be at most 16");
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(PDEC_UNSUPPORTED, "head_dim must be 64 or 128");
  if (c->qk_norm != 0 && c->qk_norm != 1) return fail(PDEC_INVALID_ARG, "qk_norm must be 0 or 1");
  if (c->kv_fp8 != 0 && c->kv_fp8 != 1) return fail(PDEC_INVALID_ARG, "kv_fp8 must be 0 or 1");
  if (c->kv_fp8) {
    if (c->dtype != PDEC_BF16) return fail(PDEC_UNSUPPORTED, "fp8 KV pages need the bf16 path");
    if (!(c->kv_scale_k > 0.f) || !(c->kv_scale_v > 0.f) || !std::isfinite(c->kv_scale_k) ||
        !std::isfinite(c->kv_scale_v))
      return fail(PDEC_INVALID_ARG, "fp8 KV scales must be positive and finite");
  }
  if (c->dtype == PDEC_BF16 && (c->d_model % 64 || c->ffn_dim % 64))
    return fail(PDEC_UNSUPPORTED, "bf16 path needs d_model and ffn_dim multiples of 64");
  return PDEC_OK;
}

int64_t kv_token_bytes(const pdec_model_cfg* c) {
  return (int64_t)c->n_layers * 2 * c->n_kv_heads * c->head_dim * kv_elem_bytes(c);
}

size_t part_elems_for(const pdec_model_cfg* c, int64_t rows_cap) {
  const int qd = c->n_q_heads * c->head_dim, kvd = c->n_kv_heads * c->head_dim;
  const int shapes[4][2] = {{qd + 2 * kvd, c->d_model},
                            {c->d_model, qd},
                            {2 * c->ffn_dim, c->d_model},
                            {c->d_model, c->ffn_dim}};
  size_t best = 0;
  for (int64_t m = 1; m <= rows_cap; ++m) {
    for (auto& s : shapes) {
      int ks;
      const int S = gemm_plan_splits(c->dtype, (int)m, s[0], s[1], &ks);
      best = std::max(best, (size_t)S * (size_t)m * (size_t)s[0]);
    }
    if (c->dtype == PDEC_BF16)  // the split tail of a fused gate/up launch
      best = std::max(best, (size_t)swiglu_tail_part_elems((int)m, c->ffn_dim, c->d_model));
  }
  return best;
}

int make_layout(const pdec_model_cfg* c, int32_t max_seqs, int32_t max_seq_len,
                int32_t max_batch, int32_t max_chunk, WsLayout* L) {
  const int G = c->n_q_heads / c->n_kv_heads;
  const int64_t ab = elem_bytes(c->dtype);
  const int64_t qd = (int64_t)c->n_q_heads * c->head_dim;
  L->rows_cap = std::max(max_batch, max_chunk);
  // Decode: one query per block, 16-row items.  Prefill: prefill_rows / G
  // queries per block, prefill_rows-row items.
  const int pre_rows = prefill_rows(*c);
  // Each piece of a packed pass may leave one partly filled query block.
  auto blocks_for = [&](int rows) {
    return (max_chunk + (rows / G) - 1) / (rows / G) + std::min(kMaxPiecesPerPass, max_chunk);
  };
  auto items_for = [&](int rows) {
    return attn_target_items(c->n_kv_heads, kPrefillTargetGroups) + blocks_for(rows) + 16;
  };
  const int64_t pre_blocks = blocks_for(pre_rows);
  L->qblocks_cap = std::max<int64_t>(max_batch, pre_blocks);
  const int64_t items_dec = attn_target_items(c->n_kv_heads, kDecodeTargetGroups) + max_batch + 16;
  const int64_t items_pre = items_for(pre_rows);
  L->items_cap = std::max(items_dec, items_pre);
  L->part_row_slots = std::max(items_dec * kDecodeRows, items_pre * pre_rows);
  if (pre_rows == 128)  // passes with 256-row blocks: fewer blocks and items, more rows each
    L->part_row_slots = std::max(L->part_row_slots, items_for(256) * 256);
  L->bt_stride = PagePool::pages_for(max_seq_len);
  L->meta_bytes = align_up(L->rows_cap * sizeof(RowMeta)) +
                  align_up(L->qblocks_cap * sizeof(AttnQBlock)) +
                  align_up(L->items_cap * sizeof(AttnItem)) + align_up(L->rows_cap * 4) +
                  align_up(kMaxPiecesPerPass * 4);
  L->delta_cap = kDeltaCap;
  L->part_elems = part_elems_for(c, L->rows_cap);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  L->rope = take((size_t)max_seq_len * (c->head_dim / 2) * sizeof(float2));
  L->bt = take((size_t)max_seqs * L->bt_stride * 4);
  L->meta = take(L->meta_bytes);
  L->delta = take(L->delta_cap * sizeof(BtDelta));
  L->x = take((size_t)L->rows_cap * c->d_model * 4);
  L->h = take((size_t)L->rows_cap * c->d_model * ab);
  L->o = take((size_t)L->rows_cap * qd * ab);
  L->u = take((size_t)L->rows_cap * c->ffn_dim * ab);
  L->q = take((size_t)L->rows_cap * qd * ab);
  L->lmg = take((size_t)kMaxPiecesPerPass * c->d_model * ab);
  L->part = take(L->part_elems * 4);
  L->att_ml = take((size_t)L->part_row_slots * c->n_kv_heads * 2 * 4);
  L->att_acc = take((size_t)L->part_row_slots * c->n_kv_heads * c->head_dim * 4);
  L->total = off;
  return PDEC_OK;
}

}  // namespace

struct pdec_engine {
  pdec_model_cfg cfg;
  const void* embed = nullptr;
  const void* lm_head = nullptr;
  const float* final_norm = nullptr;
  std::vector<const float*> attn_norm, ffn_norm, q_norm, k_norm;
  std::vector<WSegs> w_qkv, w_o, w_gu, w_down;

  char* kv_pool = nullptr;
  int64_t n_pages = 0;
  int64_t page_stride = 0;  // elements of one page in one layer-kind block
  PagePool* pool = nullptr;
  int32_t max_batch = 0, max_chunk = 0;

  WsLayout ws{};
  char* base = nullptr;
  float2* rope_cs = nullptr;
  int32_t* bt = nullptr;
  char* meta = nullptr;
  BtDelta* delta = nullptr;
  float* x = nullptr;
  char *h = nullptr, *o = nullptr, *u = nullptr, *q = nullptr, *lmg = nullptr;
  float* part = nullptr;
  float* att_ml = nullptr;
  float* att_acc = nullptr;

  hipStream_t stream = nullptr;
  Staging staging;
  LaunchTimer timer;
  std::vector<char> host_meta;
  std::vector<int32_t> mark;
  int32_t epoch = 0;
  // PDEC_VALIDATE=1 at engine creation: every pass's rows, query blocks,
  // items, pages and pending block-table entries are bounds-checked on the
  // host before anything is enqueued.
  bool validate = false;
  // Mean key pages per 128-row block from which a prefill pass takes
  // 256-row blocks (kWidePrefillPages unless PDEC_PREFILL_WIDE_PAGES is set).
  int64_t wide_prefill_pages = kWidePrefillPages;

  int64_t ab() const { return elem_bytes(cfg.dtype); }
  int64_t kvb() const { return kv_elem_bytes(&cfg); }
  char* k_layer(int l) const { return kv_pool + (int64_t)(2 * l) * n_pages * page_stride * kvb(); }
  char* v_layer(int l) const {
    return kv_pool + (int64_t)(2 * l + 1) * n_pages * page_stride * kvb();
  }
};

namespace {

int flush_deltas(pdec_engine* E) {
  const auto& pend = E->pool->pending();
  if (E->validate) {
    Status st = validate_deltas(pend, E->pool->max_seqs(), E->ws.bt_stride, E->pool->n_pages());
    if (!st.good()) return fail(st.code, st.msg);
  }
  size_t off = 0;
  while (off < pend.size()) {
    const size_t n = std::min(E->ws.delta_cap, pend.size() - off);
    HIP_OR_FAIL(E->staging.upload(E->delta, pend.data() + off, n * sizeof(BtDelta), E->stream));
    HIP_OR_FAIL(launch_bt_deltas((int)n, E->delta, E->bt, E->ws.bt_stride, E->stream));
    off += n;
  }
  E->pool->clear_pending();
  return PDEC_OK;
}

int max_items_per_qblock(const std::vector<AttnQBlock>& qblocks) {
  int m = 0;
  for (const AttnQBlock& q : qblocks) m = std::max(m, q.item_end - q.item_begin);
  return m;
}

// One forward pass of the decoder over M = rows.size() rows.
struct Pass {
  int32_t rows_per_item = 0;  // query rows per block and item: 16 (decode), 64, 128 or 256
  std::vector<RowMeta> rows;
  std::vector<AttnQBlock> qblocks;
  std::vector<AttnItem> items;
  std::vector<int32_t> tokens;   // host token ids (prefill); empty: ids on the device
  bool lm_all = false;           // logits of every row (decode)
  std::vector<int32_t> lm_rows;  // otherwise: the rows whose logits are wanted
  int32_t lm_out0 = 0;           // output row of the first of them
};

// Workspace bounds of one pass; checked for every pass of a call before the
// first launch, so that a call either enqueues all of its work or none.
int check_pass(const pdec_engine* E, const Pass& p) {
  const int rows_per_item = p.rows_per_item;
  if ((int64_t)p.items.size() > E->ws.items_cap ||
      (int64_t)p.qblocks.size() > E->ws.qblocks_cap ||
      (int64_t)p.rows.size() > E->ws.rows_cap ||
      (int64_t)p.items.size() * rows_per_item > E->ws.part_row_slots ||
      (int64_t)p.lm_rows.size() > kMaxPiecesPerPass)
    return fail(PDEC_INVALID_ARG, "attention work list exceeds the workspace bound");
  // The attention kernels compute rows_per_item rows of a block (its queries
  // times the GQA group); a larger block would lose rows silently.
  const int G = E->cfg.n_q_heads / E->cfg.n_kv_heads;
  for (const AttnQBlock& q : p.qblocks)
    if ((int64_t)q.n_q * G > rows_per_item)
      return fail(PDEC_INVALID_ARG, "query block larger than its work items' rows");
  if (E->validate) {
    Status st = validate_pass(p.rows, p.qblocks, p.items, E->pool->max_seqs(),
                              E->pool->max_seq_len(), E->ws.bt_stride, E->pool);
    if (!st.good()) return fail(st.code, st.msg);
    for (int32_t r : p.lm_rows)
      if (r < 0 || r >= (int32_t)p.rows.size()) return fail(PDEC_INVALID_ARG, "validate: LM row");
  }
  return PDEC_OK;
}

// Enqueues one pass (its bounds already checked).  Logits of the selected
// rows go to logits + lm_out0 * vocab (nullable logits: none).
int enqueue_forward(pdec_engine* E, const Pass& p, const int32_t* tokens_dev, float* logits) {
  const pdec_model_cfg& c = E->cfg;
  const int rows_per_item = p.rows_per_item;
  const int M = (int)p.rows.size();
  int rc = flush_deltas(E);
  if (rc != PDEC_OK) return rc;

  // Pack the metadata into one host buffer and copy it in one go.
  const bool gather = logits && !p.lm_all && p.lm_rows.size() > 1;
  const size_t o_rows = 0;
  const size_t o_qb = align_up(p.rows.size() * sizeof(RowMeta));
  const size_t o_it = o_qb + align_up(p.qblocks.size() * sizeof(AttnQBlock));
  const size_t o_tok = o_it + align_up(p.items.size() * sizeof(AttnItem));
  const size_t o_lm = o_tok + align_up(p.tokens.size() * 4);
  const size_t total = o_lm + (gather ? p.lm_rows.size() * 4 : 0);
  E->host_meta.resize(std::max<size_t>(total, 1));
  char* hm = E->host_meta.data();
  std::memcpy(hm + o_rows, p.rows.data(), p.rows.size() * sizeof(RowMeta));
  std::memcpy(hm + o_qb, p.qblocks.data(), p.qblocks.size() * sizeof(AttnQBlock));
  std::memcpy(hm + o_it, p.items.data(), p.items.size() * sizeof(AttnItem));
  if (!p.tokens.empty()) std::memcpy(hm + o_tok, p.tokens.data(), p.tokens.size() * 4);
  if (gather) std::memcpy(hm + o_lm, p.lm_rows.data(), p.lm_rows.size() * 4);
  HIP_OR_FAIL(E->staging.upload(E->meta, hm, total, E->stream));
  const RowMeta* d_rows = (const RowMeta*)(E->meta + o_rows);
  const AttnQBlock* d_qb = (const AttnQBlock*)(E->meta + o_qb);
  const AttnItem* d_it = (const AttnItem*)(E->meta + o_it);
  const int32_t* d_tok = p.tokens.empty() ? tokens_dev : (const int32_t*)(E->meta + o_tok);
  const int32_t* d_lm = (const int32_t*)(E->meta + o_lm);
  const int dt = c.dtype;
  const int d = c.d_model, F = c.ffn_dim, Dh = c.head_dim;
  const int qd = c.n_q_heads * Dh, nqkv = qd + 2 * c.n_kv_heads * Dh;
  hipStream_t s = E->stream;
  const int n_items = (int)p.items.size(), n_qb = (int)p.qblocks.size();
  const int max_items = max_items_per_qblock(p.qblocks);

  HIP_OR_FAIL(launch_embed_norm(dt, M, d, c.vocab, d_tok, E->embed, E->attn_norm[0], c.rms_eps, E->x,
                                E->h, s));
  for (int l = 0; l < c.n_layers; ++l) {
    int ks, S;
    hipEvent_t ea, eb;
    S = gemm_plan_splits(dt, M, nqkv, d, &ks);
    HIP_OR_FAIL(E->timer.pair(PDEC_TIMER_GEMM, &ea, &eb));
    HIP_OR_FAIL(launch_gemm(dt, M, nqkv, d, E->h, d, E->w_qkv[l], E->part, S, ks, s, ea, eb));
    HIP_OR_FAIL(launch_qkv_rope_kv(dt, c.kv_fp8, c.kv_scale_k, c.kv_scale_v, M, Dh, c.n_q_heads,
                                   c.n_kv_heads, E->part, S, d_rows,
                                   E->rope_cs, E->bt, E->ws.bt_stride, E->q, E->k_layer(l),
                                   E->v_layer(l), E->page_stride,
                                   c.qk_norm ? E->q_norm[l] : nullptr,
                                   c.qk_norm ? E->k_norm[l] : nullptr, c.rms_eps, s));
    HIP_OR_FAIL(E->timer.pair(PDEC_TIMER_ATTENTION, &ea, &eb));
    HIP_OR_FAIL(launch_attention_split(dt, c.kv_fp8, c.kv_scale_k, c.kv_scale_v, Dh, rows_per_item,
                                       n_items, c.n_q_heads, c.n_kv_heads,
                                       d_it, d_qb,
                                       E->q, E->k_layer(l), E->v_layer(l), E->page_stride, E->bt,
                                       E->ws.bt_stride, E->att_ml, E->att_acc, s, ea, eb));
    if (rows_per_item == kDecodeRows)
      HIP_OR_FAIL(launch_attention_combine(Dh, rows_per_item, n_qb, max_items, c.n_q_heads,
                                           c.n_kv_heads, d_qb, E->att_ml, E->att_acc, E->o,
                                           dt == PDEC_BF16, s));
    else  // prefill: up to 128 rows and few items per block
      HIP_OR_FAIL(launch_attention_combine_rows(Dh, rows_per_item, n_qb, c.n_q_heads,
                                                c.n_kv_heads, d_qb, E->att_ml, E->att_acc, E->o,
                                                dt == PDEC_BF16, s));
    S = gemm_plan_splits(dt, M, d, qd, &ks);
    HIP_OR_FAIL(E->timer.pair(PDEC_TIMER_GEMM, &ea, &eb));
    HIP_OR_FAIL(launch_gemm(dt, M, d, qd, E->o, qd, E->w_o[l], E->part, S, ks, s, ea, eb));
    HIP_OR_FAIL(launch_resid_norm(dt, M, d, E->part, S, E->x, E->ffn_norm[l], c.rms_eps, E->h, s));
    S = gemm_plan_splits(dt, M, 2 * F, d, &ks);
    HIP_OR_FAIL(E->timer.pair(PDEC_TIMER_GEMM, &ea, &eb));
    if (dt == PDEC_BF16 && S == 1) {  // one work group per column: SwiGLU in the epilogue
      HIP_OR_FAIL(launch_gemm_swiglu(M, F, d, E->h, d, E->w_gu[l].ptr[0], E->w_gu[l].ptr[1],
                                     E->u, E->part, s, ea, eb));
    } else {
      HIP_OR_FAIL(launch_gemm(dt, M, 2 * F, d, E->h, d, E->w_gu[l], E->part, S, ks, s, ea, eb));
      HIP_OR_FAIL(launch_swiglu(dt, M, F, E->part, S, E->u, s));
    }
    S = gemm_plan_splits(dt, M, d, F, &ks);
    HIP_OR_FAIL(E->timer.pair(PDEC_TIMER_GEMM, &ea, &eb));
    HIP_OR_FAIL(launch_gemm(dt, M, d, F, E->u, F, E->w_down[l], E->part, S, ks, s, ea, eb));
    const float* next_gain = (l + 1 < c.n_layers) ? E->attn_norm[l + 1] : E->final_norm;
    HIP_OR_FAIL(launch_resid_norm(dt, M, d, E->part, S, E->x, next_gain, c.rms_eps, E->h, s));
  }
  if (logits && (p.lm_all || !p.lm_rows.empty())) {
    WSegs lm{};
    lm.ptr[0] = E->lm_head;
    lm.row_end[0] = c.vocab;
    lm.n_seg = 1;
    const int m_lm = p.lm_all ? M : (int)p.lm_rows.size();
    const char* a = E->h;
    if (gather) {
      HIP_OR_FAIL(launch_gather_rows(m_lm, d_lm, E->h, (int64_t)d * E->ab(), E->lmg, s));
      a = E->lmg;
    } else if (!p.lm_all) {
      a = E->h + (int64_t)p.lm_rows[0] * d * E->ab();
    }
    hipEvent_t ea, eb;
    HIP_OR_FAIL(E->timer.pair(PDEC_TIMER_LM_HEAD, &ea, &eb));
    HIP_OR_FAIL(launch_gemm(dt, m_lm, c.vocab, d, a, d, lm, logits + (int64_t)p.lm_out0 * c.vocab,
                            1, d, s, ea, eb));
  }
  return PDEC_OK;
}

std::mutex g_attn_mu;
Staging* g_attn_staging = nullptr;

}  // namespace

extern "C" {

const char* last_error(void) { return g_err.c_str(); }

int64_t kv_bytes_per_token(const pdec_model_cfg* cfg) {
  int rc = check_cfg(cfg);
  if (rc != PDEC_OK) return rc;
  return kv_token_bytes(cfg);
}

int64_t engine_workspace_bytes(const pdec_model_cfg* cfg, int32_t max_seqs, int32_t max_seq_len,
                               int32_t max_batch, int32_t max_chunk, int64_t kv_pool_bytes) {
  int rc = check_cfg(cfg);
  if (rc != PDEC_OK) return rc;
  if (max_seqs < 1 || max_seqs > 65535 || max_seq_len < 1 || max_batch < 1 || max_chunk < 1 ||
      kv_pool_bytes < 0)
    return fail(PDEC_INVALID_ARG, "limits must be positive (max_seqs <= 65535)");
  WsLayout L;
  make_layout(cfg, max_seqs, max_seq_len, max_batch, max_chunk, &L);
  return (int64_t)L.total;
}

int engine_create(const pdec_model_cfg* cfg, const pdec_weights* w, void* kv_pool,
                  int64_t kv_pool_bytes, int32_t max_seqs, int32_t max_seq_len, int32_t max_batch,
                  int32_t max_chunk, void* workspace, int64_t workspace_bytes, void* stream,
                  pdec_engine** out) {
  int rc = check_cfg(cfg);
  if (rc != PDEC_OK) return rc;
  if (!w || !kv_pool || !workspace || !out) return fail(PDEC_INVALID_ARG, "null pointer argument");
  if (max_seqs < 1 || max_seqs > 65535 || max_seq_len < 1 || max_batch < 1 || max_chunk < 1)
    return fail(PDEC_INVALID_ARG, "limits must be positive (max_seqs <= 65535)");
  if (!w->embed || !w->lm_head || !w->final_norm || !w->attn_norm || !w->wq || !w->wk ||
      !w->wv || !w->wo || !w->ffn_norm || !w->w_gate || !w->w_up || !w->w_down)
    return fail(PDEC_INVALID_ARG, "null weight pointer");
  for (int l = 0; l < cfg->n_layers; ++l)
    if (!w->attn_norm[l] || !w->wq[l] || !w->wk[l] || !w->wv[l] || !w->wo[l] ||
        !w->ffn_norm[l] || !w->w_gate[l] || !w->w_up[l] || !w->w_down[l])
      return fail(PDEC_INVALID_ARG, "null weight pointer in layer " + std::to_string(l));
  if (cfg->qk_norm) {
    if (!w->q_norm || !w->k_norm) return fail(PDEC_INVALID_ARG, "qk_norm needs q_norm/k_norm");
    for (int l = 0; l < cfg->n_layers; ++l)
      if (!w->q_norm[l] || !w->k_norm[l])
        return fail(PDEC_INVALID_ARG, "null q/k norm gain in layer " + std::to_string(l));
  }
  const int64_t page_bytes = kv_token_bytes(cfg) * kPage;
  const int64_t n_pages = kv_pool_bytes / page_bytes;
  if (n_pages < 1 || n_pages > INT32_MAX)
    return fail(PDEC_INVALID_ARG, "kv_pool_bytes must hold between 1 and 2^31-1 pages");
  WsLayout L;
  make_layout(cfg, max_seqs, max_seq_len, max_batch, max_chunk, &L);
  if (workspace_bytes < (int64_t)L.total)
    return fail(PDEC_INVALID_ARG, "workspace too small: need " + std::to_string(L.total));

  auto* E = new pdec_engine();
  E->cfg = *cfg;
  E->embed = w->embed;
  E->lm_head = w->lm_head;
  E->final_norm = w->final_norm;
  const int qd = cfg->n_q_heads * cfg->head_dim, kvd = cfg->n_kv_heads * cfg->head_dim;
  for (int l = 0; l < cfg->n_layers; ++l) {
    E->attn_norm.push_back(w->attn_norm[l]);
    E->ffn_norm.push_back(w->ffn_norm[l]);
    E->q_norm.push_back(cfg->qk_norm ? w->q_norm[l] : nullptr);
    E->k_norm.push_back(cfg->qk_norm ? w->k_norm[l] : nullptr);
    WSegs a{};
    a.ptr[0] = w->wq[l];
    a.ptr[1] = w->wk[l];
    a.ptr[2] = w->wv[l];
    a.row_end[0] = qd;
    a.row_end[1] = qd + kvd;
    a.row_end[2] = qd + 2 * kvd;
    a.n_seg = 3;
    E->w_qkv.push_back(a);
    WSegs o{};
    o.ptr[0] = w->wo[l];
    o.row_end[0] = cfg->d_model;
    o.n_seg = 1;
    E->w_o.push_back(o);
    WSegs gu{};
    gu.ptr[0] = w->w_gate[l];
    gu.ptr[1] = w->w_up[l];
    gu.row_end[0] = cfg->ffn_dim;
    gu.row_end[1] = 2 * cfg->ffn_dim;
    gu.n_seg = 2;
    E->w_gu.push_back(gu);
    WSegs dn{};
    dn.ptr[0] = w->w_down[l];
    dn.row_end[0] = cfg->d_model;
    dn.n_seg = 1;
    E->w_down.push_back(dn);
  }
  E->kv_pool = (char*)kv_pool;
  E->n_pages = n_pages;
  E->page_stride = (int64_t)cfg->n_kv_heads * kPage * cfg->head_dim;
  E->pool = new PagePool((int32_t)n_pages, max_seqs, max_seq_len);
  E->max_batch = max_batch;
  E->max_chunk = max_chunk;
  E->ws = L;
  E->base = (char*)workspace;
  E->rope_cs = (float2*)(E->base + L.rope);
  E->bt = (int32_t*)(E->base + L.bt);
  E->meta = E->base + L.meta;
  E->delta = (BtDelta*)(E->base + L.delta);
  E->x = (float*)(E->base + L.x);
  E->h = E->base + L.h;
  E->o = E->base + L.o;
  E->u = E->base + L.u;
  E->q = E->base + L.q;
  E->lmg = E->base + L.lmg;
  E->part = (float*)(E->base + L.part);
  E->att_ml = (float*)(E->base + L.att_ml);
  E->att_acc = (float*)(E->base + L.att_acc);
  E->stream = (hipStream_t)stream;
  E->mark.assign(max_seqs, 0);
  {
    const char* v = std::getenv("PDEC_VALIDATE");
    E->validate = v && v[0] && std::strcmp(v, "0") != 0;
    // A plain non-negative decimal count; anything else keeps the default.
    // Values are capped at 2^40 pages so the comparison cannot overflow.
    const char* w = std::getenv("PDEC_PREFILL_WIDE_PAGES");
    if (w && w[0]) {
      char* end = nullptr;
      const long long n = std::strtoll(w, &end, 10);
      if (end && *end == '\0' && n >= 0)
        E->wide_prefill_pages = std::min<int64_t>(n, int64_t(1) << 40);
    }
  }

  auto cleanup = [&](int code, const std::string& msg) {
    delete E->pool;
    delete E;
    return fail(code, msg);
  };
  hipError_t e = E->staging.init(std::max<size_t>(L.meta_bytes, L.delta_cap * sizeof(BtDelta)), 4);
  if (e != hipSuccess) return cleanup(PDEC_HIP_ERROR, std::string("staging: ") + hipGetErrorString(e));
  // Unwritten block-table entries read as page 0 rather than as garbage.
  e = hipMemsetAsync(E->bt, 0, (size_t)max_seqs * L.bt_stride * 4, E->stream);
  if (e == hipSuccess)
    e = launch_rope_table(max_seq_len, cfg->head_dim, (double)cfg->rope_base, E->rope_cs,
                          E->stream);
  if (e != hipSuccess) return cleanup(PDEC_HIP_ERROR, std::string("init: ") + hipGetErrorString(e));
  *out = E;
  return PDEC_OK;
}

void engine_destroy(pdec_engine* E) {
  if (!E) return;
  (void)hipStreamSynchronize(E->stream);
  E->staging.release();
  delete E->pool;
  delete E;
}

int engine_profile(pdec_engine* E, int32_t classes) {
  if (!E) return fail(PDEC_INVALID_ARG, "null engine");
  E->timer.enable((uint32_t)classes & 7u);
  return PDEC_OK;
}

int engine_profile_every(pdec_engine* E, int32_t every) {
  if (!E) return fail(PDEC_INVALID_ARG, "null engine");
  if (every < 1) return fail(PDEC_INVALID_ARG, "every must be >= 1");
  E->timer.sample(every);
  return PDEC_OK;
}

int engine_profile_read(pdec_engine* E, int32_t kind, double* total_ms, int64_t* launches) {
  if (!E || !total_ms || !launches) return fail(PDEC_INVALID_ARG, "null argument");
  if (kind < PDEC_TIMER_ATTENTION || kind > PDEC_TIMER_LM_HEAD)
    return fail(PDEC_INVALID_ARG, "unknown timer kind");
  HIP_OR_FAIL(E->timer.read(kind, total_ms, launches));
  return PDEC_OK;
}

int engine_set_stream(pdec_engine* E, void* stream) {
  if (!E) return fail(PDEC_INVALID_ARG, "null engine");
  E->stream = (hipStream_t)stream;
  return PDEC_OK;
}

int kv_alloc(pdec_engine* E, int32_t reserve_tokens, int32_t* seq_out) {
  if (!E || !seq_out) return fail(PDEC_INVALID_ARG, "null argument");
  Status st = E->pool->alloc_seq(reserve_tokens, seq_out);
  return st.good() ? PDEC_OK : fail(st.code, st.msg);
}

int kv_free(pdec_engine* E, int32_t seq) {
  if (!E) return fail(PDEC_INVALID_ARG, "null engine");
  Status st = E->pool->free_seq(seq);
  return st.good() ? PDEC_OK : fail(st.code, st.msg);
}

int kv_len(pdec_engine* E, int32_t seq, int32_t* len_out) {
  if (!E || !len_out) return fail(PDEC_INVALID_ARG, "null argument");
  int32_t slot;
  Status st = E->pool->resolve(seq, &slot);
  if (!st.good()) return fail(st.code, st.msg);
  *len_out = E->pool->len(slot);
  return PDEC_OK;
}

int kv_headroom(pdec_engine* E, int64_t* free_tokens_out) {
  if (!E || !free_tokens_out) return fail(PDEC_INVALID_ARG, "null argument");
  *free_tokens_out = E->pool->headroom_tokens();
  return PDEC_OK;
}

int kv_block_table(pdec_engine* E, int32_t seq, int32_t* pages_out, int32_t capacity,
                   int32_t* n_out) {
  if (!E || !n_out) return fail(PDEC_INVALID_ARG, "null argument");
  int32_t slot;
  Status st = E->pool->resolve(seq, &slot);
  if (!st.good()) return fail(st.code, st.msg);
  const auto& pg = E->pool->pages(slot);
  *n_out = (int32_t)pg.size();
  if ((int64_t)pg.size() > capacity || (!pages_out && !pg.empty()))
    return fail(PDEC_INVALID_ARG, "capacity too small for the block table");
  if (!pg.empty()) std::memcpy(pages_out, pg.data(), pg.size() * 4);
  return PDEC_OK;
}

int kv_extend_uninit(pdec_engine* E, int32_t seq, int32_t n_tokens) {
  if (!E) return fail(PDEC_INVALID_ARG, "null engine");
  if (n_tokens < 0) return fail(PDEC_INVALID_ARG, "n_tokens must be >= 0");
  int32_t slot;
  Status st = E->pool->resolve(seq, &slot);
  if (!st.good()) return fail(st.code, st.msg);
  st = E->pool->grow(&slot, 1, n_tokens);
  return st.good() ? PDEC_OK : fail(st.code, st.msg);
}

int decode_step(pdec_engine* E, int32_t B, const int32_t* ids, const int32_t* tokens_dev,
                float* logits) {
  if (!E || !ids || !tokens_dev || !logits) return fail(PDEC_INVALID_ARG, "null argument");
  if (B < 1 || B > E->max_batch)
    return fail(PDEC_INVALID_ARG, "batch " + std::to_string(B) + " outside [1, max_batch]");
  std::vector<int32_t> slots(B);
  if (++E->epoch == INT32_MAX) {
    std::fill(E->mark.begin(), E->mark.end(), 0);
    E->epoch = 1;
  }
  for (int b = 0; b < B; ++b) {
    Status st = E->pool->resolve(ids[b], &slots[b]);
    if (!st.good()) return fail(st.code, st.msg);
    if (E->mark[slots[b]] == E->epoch)
      return fail(PDEC_INVALID_ARG, "sequence id repeated in the batch");
    E->mark[slots[b]] = E->epoch;
  }
  PagePool::GrowUndo undo;
  Status st = E->pool->grow(slots.data(), B, 1, &undo);
  if (!st.good()) return fail(st.code, st.msg);

  Pass p;
  p.rows.resize(B);
  std::vector<QBlockSpec> specs(B);
  for (int b = 0; b < B; ++b) {
    const int32_t pos = E->pool->len(slots[b]) - 1;
    p.rows[b] = {slots[b], pos};
    specs[b] = {b, 1, slots[b], pos};
  }
  p.lm_all = true;
  plan_attention(specs, choose_split_pages(total_key_pages(specs), E->cfg.n_kv_heads), &p.qblocks,
                 &p.items);
  p.rows_per_item = kDecodeRows;
  int rc = check_pass(E, p);
  if (rc == PDEC_OK) rc = enqueue_forward(E, p, tokens_dev, logits);
  if (rc != PDEC_OK) E->pool->undo(undo);
  return rc;
}

int kv_append_prefix_batch(pdec_engine* E, int32_t n_seqs, const int32_t* ids,
                           const int32_t* n_tokens, const int32_t* tokens_host,
                           int32_t chunk_tokens, float* last_logits_dev) {
  if (!E || !ids || !n_tokens || !tokens_host) return fail(PDEC_INVALID_ARG, "null argument");
  if (n_seqs < 1 || n_seqs > E->pool->max_seqs())
    return fail(PDEC_INVALID_ARG, "n_seqs outside [1, max_seqs]");
  if (chunk_tokens < 1 || chunk_tokens > E->max_chunk)
    return fail(PDEC_INVALID_ARG, "chunk_tokens outside [1, max_chunk]");
  int64_t total = 0;
  for (int i = 0; i < n_seqs; ++i) {
    if (n_tokens[i] < 1) return fail(PDEC_INVALID_ARG, "every n_tokens must be >= 1");
    total += n_tokens[i];
  }
  for (int64_t i = 0; i < total; ++i)
    if (tokens_host[i] < 0 || tokens_host[i] >= E->cfg.vocab)
      return fail(PDEC_INVALID_ARG, "token id outside [0, vocab)");
  std::vector<int32_t> slots(n_seqs), len0(n_seqs);
  if (++E->epoch == INT32_MAX) {
    std::fill(E->mark.begin(), E->mark.end(), 0);
    E->epoch = 1;
  }
  for (int i = 0; i < n_seqs; ++i) {
    Status st = E->pool->resolve(ids[i], &slots[i]);
    if (!st.good()) return fail(st.code, st.msg);
    if (E->mark[slots[i]] == E->epoch) return fail(PDEC_INVALID_ARG, "sequence id repeated");
    E->mark[slots[i]] = E->epoch;
    len0[i] = E->pool->len(slots[i]);
  }
  PagePool::GrowUndo undo;
  Status st = E->pool->grow_each(slots.data(), n_seqs, n_tokens, &undo);
  if (!st.good()) return fail(st.code, st.msg);

  // Token batching: the sequences' tokens, in order, are packed into passes
  // of at most chunk_tokens rows and kMaxPiecesPerPass pieces.  A piece is a
  // run of one sequence's consecutive tokens; its rows see the sequence's
  // earlier pages (written by earlier passes or pieces) and, causally, each
  // other.  Every pass is planned and checked before the first launch.
  const int pre_rows = prefill_rows(E->cfg);
  const int G = E->cfg.n_q_heads / E->cfg.n_kv_heads;
  std::vector<Pass> passes;
  struct Piece {
    int32_t row0, take, slot, pos;
  };
  std::vector<Piece> pass_pieces;
  std::vector<QBlockSpec> specs;
  // Query blocks of the current pass (rows / G queries each, per piece),
  // then its work items.  The pass takes 256-row blocks where its 128-row
  // blocks would read long key ranges (kWidePrefillPages).
  auto close = [&]() {
    Pass& p = passes.back();
    auto build = [&](int rows) {
      const int QB = rows / G;
      specs.clear();
      for (const Piece& pc : pass_pieces)
        for (int32_t k = 0; k * QB < pc.take; ++k)
          specs.push_back({pc.row0 + k * QB, std::min(QB, pc.take - k * QB), pc.slot,
                           pc.pos + k * QB});
    };
    p.rows_per_item = pre_rows;
    build(pre_rows);
    if (pre_rows == 128 &&
        total_key_pages(specs) >= E->wide_prefill_pages * (int64_t)specs.size()) {
      p.rows_per_item = 256;
      build(256);
    }
    plan_attention(specs,
                   choose_split_pages(total_key_pages(specs), E->cfg.n_kv_heads,
                                      kPrefillTargetGroups),
                   &p.qblocks, &p.items);
    pass_pieces.clear();
  };
  int pieces = 0;
  int64_t tok0 = 0;
  for (int i = 0; i < n_seqs; ++i) {
    for (int32_t off = 0; off < n_tokens[i];) {
      if (passes.empty() || (int64_t)passes.back().rows.size() == chunk_tokens ||
          pieces == kMaxPiecesPerPass) {
        if (!passes.empty()) close();
        passes.emplace_back();
        pieces = 0;
      }
      Pass& p = passes.back();
      const int32_t row0 = (int32_t)p.rows.size();
      const int32_t take = std::min<int32_t>(n_tokens[i] - off, chunk_tokens - row0);
      const int32_t pos = len0[i] + off;
      for (int32_t j = 0; j < take; ++j) {
        p.rows.push_back({slots[i], pos + j});
        p.tokens.push_back(tokens_host[tok0 + off + j]);
      }
      pass_pieces.push_back({row0, take, slots[i], pos});
      off += take;
      ++pieces;
      if (off == n_tokens[i] && last_logits_dev) {
        if (p.lm_rows.empty()) p.lm_out0 = i;
        p.lm_rows.push_back(row0 + take - 1);
      }
    }
    tok0 += n_tokens[i];
  }
  close();
  for (const Pass& p : passes) {
    int rc = check_pass(E, p);
    if (rc != PDEC_OK) {
      E->pool->undo(undo);
      return rc;
    }
  }
  for (const Pass& p : passes) {
    int rc = enqueue_forward(E, p, nullptr, last_logits_dev);
    if (rc != PDEC_OK) {  // a HIP error: earlier passes may already be enqueued
      E->pool->undo(undo);
      return rc;
    }
  }
  return PDEC_OK;
}

int kv_append_prefix(pdec_engine* E, int32_t seq, const int32_t* tokens_host, int32_t n,
                     int32_t chunk_tokens, float* last_logits_dev) {
  if (!E || !tokens_host) return fail(PDEC_INVALID_ARG, "null argument");
  if (n < 1) return fail(PDEC_INVALID_ARG, "n must be >= 1");
  return kv_append_prefix_batch(E, 1, &seq, &n, tokens_host, chunk_tokens, last_logits_dev);
}

namespace {

// Device-visible address of pinned host memory (fails for pageable memory).
int host_device_ptr(const void* host, void** dev) {
  hipError_t e = hipHostGetDevicePointer(dev, const_cast<void*>(host), 0);
  if (e != hipSuccess || !*dev)
    return fail(PDEC_INVALID_ARG, "host buffer must be pinned (hipHostMalloc) memory");
  return PDEC_OK;
}

int enqueue_page_copy(pdec_engine* E, const std::vector<int32_t>& pages, int n_pages,
                      void* host_dev, int to_host) {
  if ((size_t)n_pages * sizeof(int32_t) > E->ws.delta_cap * sizeof(BtDelta))
    return fail(PDEC_INVALID_ARG, "sequence too long for one snapshot call");
  int rc = flush_deltas(E);
  if (rc != PDEC_OK) return rc;
  HIP_OR_FAIL(E->staging.upload(E->delta, pages.data(), (size_t)n_pages * 4, E->stream));
  const int64_t block_bytes = E->page_stride * E->kvb();
  HIP_OR_FAIL(launch_kv_page_copy(n_pages, (const int32_t*)E->delta, E->cfg.n_layers, E->n_pages,
                                  block_bytes, E->kv_pool, host_dev, to_host, E->stream));
  return PDEC_OK;
}

}  // namespace

int kv_export(pdec_engine* E, int32_t seq, void* host_dst, int64_t dst_bytes,
              int32_t* n_tokens_out) {
  if (!E || !host_dst || !n_tokens_out) return fail(PDEC_INVALID_ARG, "null argument");
  int32_t slot;
  Status st = E->pool->resolve(seq, &slot);
  if (!st.good()) return fail(st.code, st.msg);
  const int32_t len = E->pool->len(slot);
  const int n_pages = PagePool::pages_for(len);
  const int64_t need = (int64_t)n_pages * kPage * kv_token_bytes(&E->cfg);
  if (dst_bytes < need)
    return fail(PDEC_INVALID_ARG, "host buffer too small: need " + std::to_string(need));
  void* dev = nullptr;
  int rc = host_device_ptr(host_dst, &dev);
  if (rc != PDEC_OK) return rc;
  rc = enqueue_page_copy(E, E->pool->pages(slot), n_pages, dev, 1);
  if (rc == PDEC_OK) *n_tokens_out = len;
  return rc;
}

int kv_import(pdec_engine* E, int32_t seq, const void* host_src, int64_t src_bytes,
              int32_t n_tokens) {
  if (!E || !host_src) return fail(PDEC_INVALID_ARG, "null argument");
  if (n_tokens < 1) return fail(PDEC_INVALID_ARG, "n_tokens must be >= 1");
  int32_t slot;
  Status st = E->pool->resolve(seq, &slot);
  if (!st.good()) return fail(st.code, st.msg);
  if (E->pool->len(slot) != 0) return fail(PDEC_INVALID_ARG, "kv_import needs an empty sequence");
  const int n_pages = PagePool::pages_for(n_tokens);
  const int64_t need = (int64_t)n_pages * kPage * kv_token_bytes(&E->cfg);
  if (src_bytes < need)
    return fail(PDEC_INVALID_ARG, "host buffer too small: need " + std::to_string(need));
  void* dev = nullptr;
  int rc = host_device_ptr(host_src, &dev);
  if (rc != PDEC_OK) return rc;
  PagePool::GrowUndo undo;
  st = E->pool->grow(&slot, 1, n_tokens, &undo);
  if (!st.good()) return fail(st.code, st.msg);
  rc = enqueue_page_copy(E, E->pool->pages(slot), n_pages, dev, 0);
  if (rc != PDEC_OK) E->pool->undo(undo);
  return rc;
}

int sample(pdec_engine* E, int32_t B, const float* logits_dev, int32_t* tokens_dev_out,
           int32_t mode) {
  if (!E || !logits_dev || !tokens_dev_out) return fail(PDEC_INVALID_ARG, "null argument");
  if (mode != 0) return fail(PDEC_UNSUPPORTED, "only greedy sampling (mode 0) is implemented");
  if (B < 1) return fail(PDEC_INVALID_ARG, "batch must be >= 1");
  HIP_OR_FAIL(launch_argmax(B, E->cfg.vocab, logits_dev, tokens_dev_out, E->stream));
  return PDEC_OK;
}

int pacing_plan(int64_t headroom_tokens, int64_t h_min_tokens, int64_t delta_tokens,
                int32_t n_active, const int32_t* active_ids, const int32_t* active_len,
                const int64_t* active_held_tokens, int32_t n_pending, const int32_t* pending_ids,
                const int32_t* pending_len, int32_t* evict_out, int32_t* n_evict_out,
                int32_t* place_out, int32_t* n_place_out) {
  if (n_active < 0 || n_pending < 0 || !n_evict_out || !n_place_out)
    return fail(PDEC_INVALID_ARG, "bad counts or null output");
  if ((n_active && (!active_ids || !active_len || !active_held_tokens || !evict_out)) ||
      (n_pending && (!pending_ids || !pending_len)) || (n_active + n_pending && !place_out))
    return fail(PDEC_INVALID_ARG, "null array argument");
  if (h_min_tokens < 0 || delta_tokens < 0)
    return fail(PDEC_INVALID_ARG, "h_min and delta must be >= 0");
  std::vector<PacingResident> act(n_active);
  for (int i = 0; i < n_active; ++i) {
    if (active_len[i] < 0 || active_held_tokens[i] < 0)
      return fail(PDEC_INVALID_ARG, "negative length or held tokens");
    act[i] = {active_ids[i], active_len[i], active_held_tokens[i]};
  }
  std::vector<PacingPending> pend(n_pending);
  for (int i = 0; i < n_pending; ++i) {
    if (pending_len[i] < 0) return fail(PDEC_INVALID_ARG, "negative pending length");
    pend[i] = {pending_ids[i], pending_len[i]};
  }
  std::vector<int32_t> ev, pl;
  pdec::pacing_plan(headroom_tokens, h_min_tokens, delta_tokens, act, pend, &ev, &pl);
  for (size_t i = 0; i < ev.size(); ++i) evict_out[i] = ev[i];
  for (size_t i = 0; i < pl.size(); ++i) place_out[i] = pl[i];
  *n_evict_out = (int32_t)ev.size();
  *n_place_out = (int32_t)pl.size();
  return PDEC_OK;
}

int64_t sample_top_p_workspace_bytes(int32_t batch) {
  if (batch < 1) return fail(PDEC_INVALID_ARG, "batch must be positive");
  return sample_workspace_bytes(batch);
}

int sample_top_p(int32_t batch, int32_t vocab, const float* logits_dev, float temperature,
                 float top_p, const float* uniforms_dev, int32_t* tokens_dev_out,
                 void* workspace, int64_t workspace_bytes, void* stream) {
  if (batch < 1 || vocab < 1) return fail(PDEC_INVALID_ARG, "batch and vocab must be positive");
  if (!logits_dev || !uniforms_dev || !tokens_dev_out)
    return fail(PDEC_INVALID_ARG, "null argument");
  if (!(temperature > 0.f) || !std::isfinite(temperature))
    return fail(PDEC_INVALID_ARG, "temperature must be positive and finite");
  if (!(top_p > 0.f && top_p <= 1.f)) return fail(PDEC_INVALID_ARG, "top_p must be in (0, 1]");
  if (workspace_bytes < 0 || (workspace && workspace_bytes == 0))
    return fail(PDEC_INVALID_ARG, "bad workspace size");
  if (workspace && workspace_bytes < sample_workspace_bytes(batch))
    return fail(PDEC_INVALID_ARG, "workspace smaller than sample_top_p_workspace_bytes");
  HIP_OR_FAIL(launch_sample_top_p(batch, vocab, logits_dev, temperature, top_p, uniforms_dev,
                                  tokens_dev_out, workspace, workspace_bytes,
                                  (hipStream_t)stream));
  return PDEC_OK;
}

int sample_top_p_noalloc(int32_t batch, int32_t vocab, const float* logits_dev,
                         float temperature, float top_p, const float* uniforms_dev,
                         int32_t* tokens_dev_out, void* stream) {
  if (batch < 1 || vocab < 1) return fail(PDEC_INVALID_ARG, "batch and vocab must be positive");
  if (!logits_dev || !uniforms_dev || !tokens_dev_out)
    return fail(PDEC_INVALID_ARG, "null argument");
  if (!(temperature > 0.f) || !std::isfinite(temperature))
    return fail(PDEC_INVALID_ARG, "temperature must be positive and finite");
  if (!(top_p > 0.f && top_p <= 1.f)) return fail(PDEC_INVALID_ARG, "top_p must be in (0, 1]");
  const int64_t need = sample_workspace_bytes(batch), have = sample_scratch_bytes();
  if (need > have)
    return fail(PDEC_INVALID_ARG, "batch " + std::to_string(batch) + " needs " +
                                      std::to_string(need) + " bytes of scratch; the static "
                                      "scratch holds " + std::to_string(have));
  void* scratch = nullptr;
  if (need > 0) HIP_OR_FAIL(sample_scratch_ptr(&scratch));
  HIP_OR_FAIL(launch_sample_top_p(batch, vocab, logits_dev, temperature, top_p, uniforms_dev,
                                  tokens_dev_out, scratch, need > 0 ? have : 0,
                                  (hipStream_t)stream));
  return PDEC_OK;
}

int64_t packed_weight_bytes(int32_t dtype, int32_t N, int32_t K) {
  if ((dtype != PDEC_F32 && dtype != PDEC_BF16) || N < 1 || K < 1)
    return fail(PDEC_INVALID_ARG, "bad weight shape");
  if (dtype == PDEC_BF16) {
    if (K % 64) return fail(PDEC_UNSUPPORTED, "bf16 weights need K % 64 == 0");
    return (int64_t)((N + 127) / 128) * 128 * K * 2;
  }
  return (int64_t)N * K * 4;
}

int pack_weight(int32_t dtype, int32_t N, int32_t K, const void* w, void* packed, void* stream) {
  const int64_t bytes = packed_weight_bytes(dtype, N, K);
  if (bytes < 0) return (int)bytes;
  if (!w || !packed) return fail(PDEC_INVALID_ARG, "null argument");
  HIP_OR_FAIL(launch_pack_weight(dtype, N, K, w, packed, (hipStream_t)stream));
  return PDEC_OK;
}

int64_t weight_projection_workspace_bytes(int32_t dtype, int32_t M, int32_t N, int32_t K) {
  if ((dtype != PDEC_F32 && dtype != PDEC_BF16) || M < 1 || N < 1 || K < 1)
    return fail(PDEC_INVALID_ARG, "bad projection arguments");
  int ks;
  const int S = gemm_plan_splits(dtype, M, N, K, &ks);
  return S > 1 ? (int64_t)S * M * N * 4 : 0;
}

int weight_projection(int32_t dtype, int32_t M, int32_t N, int32_t K, const void* x,
                      const void* w, float* out, void* workspace, int64_t ws_bytes,
                      void* stream) {
  if (!x || !w || !out) return fail(PDEC_INVALID_ARG, "null argument");
  const int64_t need = weight_projection_workspace_bytes(dtype, M, N, K);
  if (need < 0) return (int)need;
  if (dtype == PDEC_BF16 && K % 64)
    return fail(PDEC_UNSUPPORTED, "bf16 projections need K % 64 == 0");
  if (N % 4) return fail(PDEC_UNSUPPORTED, "projections need N % 4 == 0");
  if (ws_bytes < need || (need > 0 && !workspace))
    return fail(PDEC_INVALID_ARG, "workspace too small: need " + std::to_string(need));
  WSegs ws{};
  ws.ptr[0] = w;
  ws.row_end[0] = N;
  ws.n_seg = 1;
  int ks;
  const int S = gemm_plan_splits(dtype, M, N, K, &ks);
  hipStream_t s = (hipStream_t)stream;
  float* dst = S > 1 ? (float*)workspace : out;
  HIP_OR_FAIL(launch_gemm(dtype, M, N, K, x, K, ws, dst, S, ks, s));
  if (S > 1) HIP_OR_FAIL(launch_sum_splits((int64_t)M * N, dst, S, out, s));
  return PDEC_OK;
}

int64_t swiglu_projection_workspace_bytes(int32_t dtype, int32_t M, int32_t F, int32_t K) {
  if ((dtype != PDEC_F32 && dtype != PDEC_BF16) || M < 1 || F < 1 || K < 1 || F > INT32_MAX / 2)
    return fail(PDEC_INVALID_ARG, "bad projection arguments");
  int ks;
  const int S = gemm_plan_splits(dtype, M, 2 * F, K, &ks);
  return (dtype == PDEC_BF16 && S == 1) ? swiglu_tail_part_elems(M, F, K) * 4
                                         : (int64_t)S * M * 2 * F * 4;
}

int swiglu_projection(int32_t dtype, int32_t M, int32_t F, int32_t K, const void* x,
                      const void* w_gate, const void* w_up, void* u, void* workspace,
                      int64_t ws_bytes, void* stream) {
  if (!x || !w_gate || !w_up || !u) return fail(PDEC_INVALID_ARG, "null argument");
  const int64_t need = swiglu_projection_workspace_bytes(dtype, M, F, K);
  if (need < 0) return (int)need;
  if (dtype == PDEC_BF16 && K % 64)
    return fail(PDEC_UNSUPPORTED, "bf16 projections need K % 64 == 0");
  if (F % 4) return fail(PDEC_UNSUPPORTED, "SwiGLU needs F % 4 == 0");
  if (ws_bytes < need || (need > 0 && !workspace))
    return fail(PDEC_INVALID_ARG, "workspace too small: need " + std::to_string(need));
  int ks;
  const int S = gemm_plan_splits(dtype, M, 2 * F, K, &ks);
  hipStream_t s = (hipStream_t)stream;
  // The same choice as the decoder layer.
  if (dtype == PDEC_BF16 && S == 1) {
    HIP_OR_FAIL(launch_gemm_swiglu(M, F, K, x, K, w_gate, w_up, u,
                                   need > 0 ? (float*)workspace : nullptr, s));
    return PDEC_OK;
  }
  WSegs ws{};
  ws.ptr[0] = w_gate;
  ws.ptr[1] = w_up;
  ws.row_end[0] = F;
  ws.row_end[1] = 2 * F;
  ws.n_seg = 2;
  HIP_OR_FAIL(launch_gemm(dtype, M, 2 * F, K, x, K, ws, (float*)workspace, S, ks, s));
  HIP_OR_FAIL(launch_swiglu(dtype, M, F, (const float*)workspace, S, u, s));
  return PDEC_OK;
}

int64_t paged_attention_workspace_bytes(int32_t batch, int32_t n_q_heads, int32_t n_kv_heads,
                                        int32_t head_dim, int64_t max_total_tokens) {
  (void)max_total_tokens;
  if (batch < 1 || n_q_heads < 1 || n_kv_heads < 1 || head_dim < 1)
    return fail(PDEC_INVALID_ARG, "sizes must be positive");
  const int64_t items_cap = attn_target_items(n_kv_heads) + batch + 16;
  return (int64_t)(align_up(batch * sizeof(AttnQBlock)) + align_up(items_cap * sizeof(AttnItem)) +
                   align_up(items_cap * n_kv_heads * 16 * 2 * 4) +
                   align_up(items_cap * n_kv_heads * 16 * (int64_t)head_dim * 4));
}

// kv_dtype: PDEC_F32 (fp32 q and pages), PDEC_BF16 (bf16 q and pages) or
// PDEC_FP8_E4M3 (bf16 q, E4M3 pages with scales).
static int paged_attention_impl(int32_t kv_dtype, float k_scale, float v_scale, int32_t B,
                                int32_t Hq, int32_t Hkv, int32_t Dh, const void* q,
                                const void* k_pages, const void* v_pages, const int32_t* bt,
                                int32_t bt_stride, const int32_t* lens, float* out,
                                void* workspace, int64_t ws_bytes, void* stream) {
  if (!q || !k_pages || !v_pages || !bt || !lens || !out || !workspace)
    return fail(PDEC_INVALID_ARG, "null argument");
  if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv || bt_stride < 1)
    return fail(PDEC_INVALID_ARG, "bad sizes");
  if (Hq / Hkv > 16) return fail(PDEC_UNSUPPORTED, "GQA group size must be at most 16");
  if (Dh != 64 && Dh != 128) return fail(PDEC_UNSUPPORTED, "head_dim must be 64 or 128");
  const int64_t need = paged_attention_workspace_bytes(B, Hq, Hkv, Dh, 0);
  if (ws_bytes < need) return fail(PDEC_INVALID_ARG, "workspace too small: need " + std::to_string(need));
  std::vector<QBlockSpec> specs(B);
  for (int b = 0; b < B; ++b) {
    if (lens[b] < 1 || (int64_t)lens[b] > (int64_t)bt_stride * kPage)
      return fail(PDEC_INVALID_ARG, "lens[b] outside [1, bt_stride*16]");
    specs[b] = {b, 1, b, lens[b] - 1};
  }
  std::vector<AttnQBlock> qblocks;
  std::vector<AttnItem> items;
  plan_attention(specs, choose_split_pages(total_key_pages(specs), Hkv), &qblocks, &items);

  const int64_t items_cap = attn_target_items(Hkv) + B + 16;
  if ((int64_t)items.size() > items_cap) return fail(PDEC_INVALID_ARG, "work list too large");
  char* base = (char*)workspace;
  const size_t o_qb = 0;
  const size_t o_it = align_up(B * sizeof(AttnQBlock));
  const size_t o_ml = o_it + align_up(items_cap * sizeof(AttnItem));
  const size_t o_acc = o_ml + align_up(items_cap * Hkv * 16 * 2 * 4);
  std::vector<char> hm(o_ml);
  std::memcpy(hm.data() + o_qb, qblocks.data(), qblocks.size() * sizeof(AttnQBlock));
  std::memcpy(hm.data() + o_it, items.data(), items.size() * sizeof(AttnItem));
  hipStream_t s = (hipStream_t)stream;
  {
    std::lock_guard<std::mutex> lk(g_attn_mu);
    if (!g_attn_staging) {
      auto* st = new Staging();
      hipError_t e = st->init(1 << 20, 4);
      if (e != hipSuccess) {
        delete st;
        return fail(PDEC_HIP_ERROR, std::string("staging: ") + hipGetErrorString(e));
      }
      g_attn_staging = st;
    }
    HIP_OR_FAIL(g_attn_staging->upload(base, hm.data(), o_ml, s));
  }
  const int64_t page_stride = (int64_t)Hkv * kPage * Dh;
  HIP_OR_FAIL(launch_attention_split(kv_dtype == PDEC_F32 ? PDEC_F32 : PDEC_BF16,
                                     kv_dtype == PDEC_FP8_E4M3, k_scale, v_scale, Dh, kDecodeRows,
                                     (int)items.size(), Hq, Hkv,
                                     (const AttnItem*)(base + o_it),
                                     (const AttnQBlock*)(base + o_qb), q, k_pages, v_pages,
                                     page_stride, bt, bt_stride, (float*)(base + o_ml),
                                     (float*)(base + o_acc), s));
  HIP_OR_FAIL(launch_attention_combine(Dh, kDecodeRows, B, max_items_per_qblock(qblocks), Hq,
                                       Hkv, (const AttnQBlock*)(base + o_qb),
                                       (float*)(base + o_ml), (float*)(base + o_acc), out, 0, s));
  return PDEC_OK;
}

int paged_decode_attention(int32_t dtype, int32_t B, int32_t Hq, int32_t Hkv, int32_t Dh,
                           const void* q, const void* k_pages, const void* v_pages,
                           const int32_t* bt, int32_t bt_stride, const int32_t* lens,
                           float* out, void* workspace, int64_t ws_bytes, void* stream) {
  if (dtype != PDEC_F32 && dtype != PDEC_BF16) return fail(PDEC_INVALID_ARG, "bad dtype");
  return paged_attention_impl(dtype, 1.f, 1.f, B, Hq, Hkv, Dh, q, k_pages, v_pages, bt,
                              bt_stride, lens, out, workspace, ws_bytes, stream);
}

int paged_decode_attention_fp8(int32_t B, int32_t Hq, int32_t Hkv, int32_t Dh, const void* q,
                               const void* k_pages, const void* v_pages, float k_scale,
                               float v_scale, const int32_t* bt, int32_t bt_stride,
                               const int32_t* lens, float* out, void* workspace,
                               int64_t ws_bytes, void* stream) {
  if (!(k_scale > 0.f) || !(v_scale > 0.f) || !std::isfinite(k_scale) || !std::isfinite(v_scale))
    return fail(PDEC_INVALID_ARG, "scales must be positive and finite");
  return paged_attention_impl(PDEC_FP8_E4M3, k_scale, v_scale, B, Hq, Hkv, Dh, q, k_pages,
                              v_pages, bt, bt_stride, lens, out, workspace, ws_bytes, stream);
}

}  // extern "C"

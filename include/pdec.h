/*
 * pdec.h: C ABI of the MI355X (gfx950) batched paged-decode library.
 *
 * The library runs the batched autoregressive decode step of a rollout
 * worker: every step reads the model weights once for the whole active batch
 * and each trajectory's own KV history (paper: Introduction; Design
 * Principles, "Specialization in Heterogeneous Pools").  The worker hosts a
 * resident set of trajectories and decides locally about batching and memory
 * (Design, "Separating Departure from Placement").  KV state lives in
 * fixed-size pages addressed through per-trajectory block tables.
 *
 * Conventions shared by every call:
 *   - Every function returns an int status (PDEC_OK or a negative code) unless
 *     stated otherwise.  last_error() returns a per-thread message for the
 *     last failure.
 *   - On any error no device work has been enqueued and the host-side state
 *     (sequence lengths, block tables, free pages) is unchanged.  The one
 *     exception is PDEC_HIP_ERROR from the runtime in the middle of a call
 *     that enqueues several launches: the host state is still restored, but
 *     launches before the failing one may have run (e.g. KV writes of the
 *     first chunks of a prefill).  Every check that can fail on the
 *     arguments runs before the first launch.
 *   - Setting the environment variable PDEC_VALIDATE=1 before engine_create
 *     makes that engine bounds-check every forward pass on the host before
 *     enqueueing it: row slots and positions, query blocks and their work
 *     items against the block-table row and the sequence's pages, page ids
 *     against the pool, and pending block-table entries (range, and no entry
 *     written twice).  A failed check returns PDEC_INVALID_ARG ("validate:
 *     ...") with nothing enqueued.  Off by default (host cost per call).
 *   - Prefill with bf16 activations and 128-dim heads groups query rows in
 *     blocks of 128 (128 / G queries, G the GQA group, rounded down; work
 *     groups of four waves); a pass whose blocks read
 *     long key ranges (on average at least 1024 pages, 16K keys, per
 *     128-row block) takes 256-row blocks (eight waves sharing each staged
 *     page).  PDEC_PREFILL_WIDE_PAGES=<pages> before engine_create sets that
 *     threshold for the engine (0: always 256-row blocks; a value that is not
 *     a non-negative decimal integer is ignored).  Results agree to float32
 *     summation order either way.
 *   - Device memory (weights, KV pool, workspace, tokens, logits) is owned by
 *     the caller and must outlive the engine.  The library owns host metadata
 *     and a small pinned staging ring only.
 *   - All device work of one engine is enqueued, asynchronously, on the one
 *     HIP stream the engine holds (engine_create / engine_set_stream).  No
 *     call waits for the device, except where a pinned staging slot is reused
 *     and the copy that last used it has not yet run.
 *   - "host" pointers are ordinary CPU memory; "dev" pointers are device
 *     memory of the current HIP device.
 *   - Sequence ids are opaque int32 handles; an id becomes stale when its
 *     sequence is freed, and stale ids are rejected with PDEC_BAD_SEQ.
 */
#ifndef PDEC_H
#define PDEC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PDEC_OK 0
#define PDEC_INVALID_ARG (-1)
#define PDEC_OUT_OF_PAGES (-2)
#define PDEC_BAD_SEQ (-3)
#define PDEC_SEQ_TOO_LONG (-4)
#define PDEC_HIP_ERROR (-5)
#define PDEC_UNSUPPORTED (-6)

/* Tokens per KV page. */
#define PDEC_PAGE_TOKENS 16

/* Storage type of weights and KV pages.  Activations between kernels, the
 * residual stream, norms, softmax statistics and every accumulator are fp32
 * on both paths; the BF16 path feeds bf16-rounded activations to its matrix
 * cores. */
#define PDEC_F32 0
#define PDEC_BF16 1
/* KV page storage only (pdec_model_cfg.kv_fp8, paged_decode_attention_fp8):
 * OCP 8-bit E4M3FN codes (sign, 4 exponent bits with bias 7, 3 mantissa
 * bits; subnormals m * 2^-9; largest finite 448; no infinities), written with
 * round-to-nearest-even, saturation at +-448 and the sign kept, and read back
 * as value(code) * scale.  Halves the bytes each decode step streams per
 * cached token (Background, "Hardware-Workload Interaction": long-context
 * decode is bound by KV traffic). */
#define PDEC_FP8_E4M3 2

/* Llama-style pre-norm decoder: RMSNorm, rotary position embedding
 * (rotate-half pairing), grouped-query attention with contiguous groups
 * (query head h reads KV head h / (n_q_heads / n_kv_heads)), SwiGLU FFN,
 * final RMSNorm and an untied LM head.  No biases. */
typedef struct pdec_model_cfg {
  int32_t n_layers;
  int32_t d_model;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;  /* 64 or 128 */
  int32_t ffn_dim;
  int32_t vocab;
  float rms_eps;
  float rope_base;
  int32_t dtype;     /* PDEC_F32 or PDEC_BF16 */
  int32_t qk_norm;   /* 1: per-head RMSNorm of q and k over head_dim before RoPE,
                        with gains weights->q_norm / k_norm (the Qwen3 family's
                        attention; the paper's models are Qwen3); 0: none */
  int32_t kv_fp8;    /* 1: KV pages hold PDEC_FP8_E4M3 codes of k / kv_scale_k and
                        v / kv_scale_v (bf16 path only); 0: pages in dtype */
  float kv_scale_k;  /* > 0, used when kv_fp8 */
  float kv_scale_v;
} pdec_model_cfg;

/* Device pointers to the weights, stored in cfg->dtype except the norm gains
 * (always fp32).  The embedding table is row-major [vocab][d_model].  The
 * projection matrices (wq ... w_down, lm_head), listed below in their
 * nn.Linear [out][in] shape, are passed as produced by pack_weight: for bf16
 * that is the group-major layout the weight-streaming kernels read, for fp32
 * the row-major matrix itself.
 * The per-layer members are HOST arrays of n_layers DEVICE pointers; the
 * arrays are copied by engine_create and may be freed afterwards. */
typedef struct pdec_weights {
  const void* embed;             /* [vocab][d_model] */
  const void* lm_head;           /* [vocab][d_model] */
  const float* final_norm;       /* [d_model] */
  const float* const* attn_norm; /* n_layers x [d_model] */
  const void* const* wq;         /* n_layers x [n_q_heads*head_dim][d_model] */
  const void* const* wk;         /* n_layers x [n_kv_heads*head_dim][d_model] */
  const void* const* wv;         /* n_layers x [n_kv_heads*head_dim][d_model] */
  const void* const* wo;         /* n_layers x [d_model][n_q_heads*head_dim] */
  const float* const* ffn_norm;  /* n_layers x [d_model] */
  const void* const* w_gate;     /* n_layers x [ffn_dim][d_model] */
  const void* const* w_up;       /* n_layers x [ffn_dim][d_model] */
  const void* const* w_down;     /* n_layers x [d_model][ffn_dim] */
  const float* const* q_norm;    /* n_layers x [head_dim]; only with cfg->qk_norm */
  const float* const* k_norm;    /* n_layers x [head_dim]; only with cfg->qk_norm */
} pdec_weights;

typedef struct pdec_engine pdec_engine;

/* Message describing the last failure on this thread ("" if none). */
const char* last_error(void);

/* Bytes of KV state one token occupies across all layers:
 * n_layers * 2 * n_kv_heads * head_dim * sizeof(dtype).  This is the
 * per-token footprint the paper uses to convert its decode reserve, given in
 * tokens, into KV-cache space (Implementation, scheduling parameters).
 * Returns a negative status for an invalid cfg. */
int64_t kv_bytes_per_token(const pdec_model_cfg* cfg);

/* Bytes of workspace engine_create needs for these limits; negative status on
 * invalid arguments.  max_batch bounds decode_step's batch; max_chunk bounds
 * kv_append_prefix's chunk_tokens; kv_pool_bytes is the pool that will be
 * passed to engine_create (it bounds the attention work list). */
int64_t engine_workspace_bytes(const pdec_model_cfg* cfg, int32_t max_seqs, int32_t max_seq_len,
                               int32_t max_batch, int32_t max_chunk, int64_t kv_pool_bytes);

/* Create an engine (one rollout worker's decode backend).
 *
 * kv_pool: device buffer of kv_pool_bytes, carved into
 *   n_pages = kv_pool_bytes / (PDEC_PAGE_TOKENS * kv_bytes_per_token(cfg))
 * pages.  Layout, for layer l, page p, KV head g:
 *   K block at [l][0][p][g] : [16 slots][head_dim]   (row per token)
 *   V block at [l][1][p][g] : [head_dim][16 slots]   (transposed per page)
 * i.e. the pool is [n_layers][2][n_pages][n_kv_heads][16 * head_dim].
 * workspace: device buffer of at least engine_workspace_bytes(...) bytes.
 * stream: a hipStream_t (NULL = the null stream).
 * The engine starts with an empty resident set and every page free.
 * Errors: PDEC_INVALID_ARG (bad sizes, null pointers), PDEC_UNSUPPORTED
 * (shapes the kernels do not handle: head_dim other than 64/128, GQA group
 * size above 16, BF16 dims not multiples of 64), PDEC_HIP_ERROR. */
int engine_create(const pdec_model_cfg* cfg, const pdec_weights* weights, void* kv_pool,
                  int64_t kv_pool_bytes, int32_t max_seqs, int32_t max_seq_len, int32_t max_batch,
                  int32_t max_chunk, void* workspace, int64_t workspace_bytes, void* stream,
                  pdec_engine** out);

/* Release host resources.  Waits for the engine's stream first. */
void engine_destroy(pdec_engine* engine);

/* Change the stream later calls enqueue on (hipStream_t). */
int engine_set_stream(pdec_engine* engine, void* stream);

/* Launch timing for measurement.  engine_profile(engine, classes) takes a
 * bitmask of the classes below ((1 << PDEC_TIMER_ATTENTION) | ...; 0 turns
 * timing off).  A timed launch records its own begin and end in a pair of
 * HIP events (hipExtLaunchKernelGGL), which still leaves the GPU idle for a
 * few microseconds around that launch, so select only what is being
 * measured.  engine_profile_every(engine, every) times one launch in every
 * `every` of each selected class (launches counted per class from this call;
 * every >= 1, default 1 = all); with every = n_layers + 1 a decode step
 * carries about one timed launch and the timed layer rotates from step to
 * step.  engine_profile_read synchronises on the events and returns the
 * summed elapsed time (ms) and the count of timed launches of one class,
 * clearing those records. */
#define PDEC_TIMER_ATTENTION 0 /* paged split-K attention pass, one per layer */
#define PDEC_TIMER_GEMM 1      /* the four weight projections of each layer */
#define PDEC_TIMER_LM_HEAD 2   /* the LM-head projection */
int engine_profile(pdec_engine* engine, int32_t classes);
int engine_profile_every(pdec_engine* engine, int32_t every);
int engine_profile_read(pdec_engine* engine, int32_t kind, double* total_ms, int64_t* launches);

/* Admit an empty trajectory and reserve ceil(reserve_tokens / 16) pages for
 * its growth.  Placement is feasible only if the footprint fits in the
 * headroom (Design, "Separating Departure from Placement": KV headroom), and
 * the per-resident decode reserve is a token count (Design, "Sustaining
 * Specialization": pacing thresholds).  Reserved pages are held by the
 * sequence and consumed first as it grows.
 * Errors: PDEC_OUT_OF_PAGES (not enough free pages, nothing changes),
 * PDEC_INVALID_ARG (reserve_tokens < 0 or > max_seq_len, or no free sequence
 * slot). */
int kv_alloc(pdec_engine* engine, int32_t reserve_tokens, int32_t* seq_out);

/* Departure: free every page of the sequence, raising the headroom at once
 * (Design, "Separating Departure from Placement").  The id becomes stale.
 * Work already enqueued that reads these pages still runs before any later
 * reuse, since every call uses the engine's one stream. */
int kv_free(pdec_engine* engine, int32_t seq);

/* Number of cached tokens of a sequence. */
int kv_len(pdec_engine* engine, int32_t seq, int32_t* len_out);

/* KV headroom H_w in tokens: free pages x 16 (reserved pages excluded). */
int kv_headroom(pdec_engine* engine, int64_t* free_tokens_out);

/* Copy the sequence's page ids (logical order, reserved pages included) into
 * pages_out (host, capacity entries); *n_out receives the count.
 * PDEC_INVALID_ARG if capacity is too small. */
int kv_block_table(pdec_engine* engine, int32_t seq, int32_t* pages_out, int32_t capacity,
                   int32_t* n_out);

/* Extend a sequence by n_tokens positions WITHOUT computing their KV: the
 * caller owns the content of those slots (benchmarks stage synthetic
 * contexts this way instead of running a long prefill).  Pages are grown
 * atomically.  Errors: PDEC_OUT_OF_PAGES, PDEC_SEQ_TOO_LONG, PDEC_BAD_SEQ. */
int kv_extend_uninit(pdec_engine* engine, int32_t seq, int32_t n_tokens);

/* Chunked prefill of n tokens onto the sequence's existing KV: the
 * destination-side re-prefill the paper falls back to when prepared KV cannot
 * be used (Design, "KV Preparation for Late-Bound Placement"), and the
 * backend's chunked prefill ordering.  Token i is placed at position
 * kv_len + i.  tokens_host: host array of n token ids.  The work is done in
 * chunks of at most chunk_tokens rows (1 <= chunk_tokens <= max_chunk); the
 * result does not depend on the chunking beyond rounding.  last_logits_dev
 * (nullable): device fp32 [vocab] receiving the logits at the last new
 * position.  Pages for all n tokens are taken up front.
 * Errors: PDEC_OUT_OF_PAGES, PDEC_SEQ_TOO_LONG, PDEC_BAD_SEQ, PDEC_INVALID_ARG
 * (n < 1, token id outside [0, vocab)). */
int kv_append_prefix(pdec_engine* engine, int32_t seq, const int32_t* tokens_host, int32_t n,
                     int32_t chunk_tokens, float* last_logits_dev);

/* The same for several sequences in one call (the backend's token batching of
 * prefill work; Design, "Separating Departure from Placement").  Sequence
 * seq_ids_host[i] receives n_tokens_host[i] tokens, taken in order from the
 * concatenation tokens_host (sum of n_tokens_host ids).  The tokens of all
 * sequences, in this order, are packed into forward passes of at most
 * chunk_tokens rows (a pass holds pieces of up to 64 sequences); each
 * sequence's result is the one kv_append_prefix would give, up to rounding.
 * last_logits_dev (nullable): device fp32 [n_seqs][vocab]; row i receives
 * the logits at sequence i's last new position.  Pages for every sequence
 * are taken up front, all or nothing.
 * Errors: as kv_append_prefix, and PDEC_INVALID_ARG for n_seqs outside
 * [1, max_seqs], repeated ids or any n_tokens_host[i] < 1. */
int kv_append_prefix_batch(pdec_engine* engine, int32_t n_seqs, const int32_t* seq_ids_host,
                           const int32_t* n_tokens_host, const int32_t* tokens_host,
                           int32_t chunk_tokens, float* last_logits_dev);

/* One decode step for `batch` distinct resident sequences (iteration-level
 * token batching; Design, "Separating Departure from Placement").
 * seq_ids_host: host [batch] ids, any order; tokens_dev: device int32 [batch],
 * token i is the input of seq_ids_host[i] at position kv_len(seq);
 * logits_dev: device fp32 [batch][vocab] receives the next-token logits.
 * Each sequence's result does not depend on the order or on the other
 * members of the batch.  Page growth is atomic across the whole batch.
 * Errors: PDEC_INVALID_ARG (batch outside [1, max_batch], repeated ids),
 * PDEC_BAD_SEQ, PDEC_SEQ_TOO_LONG, PDEC_OUT_OF_PAGES. */
int decode_step(pdec_engine* engine, int32_t batch, const int32_t* seq_ids_host,
                const int32_t* tokens_dev, float* logits_dev);

/* KV snapshot of a resident trajectory into host memory: phase 1 of the
 * paper's late-bound KV preparation, where a departing trajectory's KV is
 * copied from device memory to host DRAM over PCIe so its pages can be freed
 * while the host copy keeps it available (Design, "KV Preparation for
 * Late-Bound Placement").  host_dst must be PINNED host memory (hipHostMalloc)
 * of at least ceil(len/16) * 16 * kv_bytes_per_token bytes.  Layout of the
 * snapshot, page-major so that a prefix range of pages is one contiguous
 * range: [page][layer][K|V][n_kv_heads][16 * head_dim] with the V block
 * transposed as in the pool.  The copy is enqueued on the engine's stream;
 * synchronise it before reading host_dst.  The sequence stays resident (call
 * kv_free to depart); later work on the stream cannot overwrite its pages
 * before the copy has run.  *n_tokens_out receives the sequence length.
 * Errors: PDEC_BAD_SEQ, PDEC_INVALID_ARG (buffer too small or not pinned). */
int kv_export(pdec_engine* engine, int32_t seq, void* host_dst, int64_t dst_bytes,
              int32_t* n_tokens_out);

/* Restore a snapshot written by kv_export into an EMPTY sequence (fresh from
 * kv_alloc): pages for n_tokens are taken atomically and filled from
 * host_src (pinned host memory, same layout), and the sequence length
 * becomes n_tokens.  The alternative to re-prefilling the prefix from its
 * tokens (kv_append_prefix).
 * Errors: PDEC_BAD_SEQ, PDEC_OUT_OF_PAGES, PDEC_SEQ_TOO_LONG,
 * PDEC_INVALID_ARG (non-empty sequence, buffer too small or not pinned). */
int kv_import(pdec_engine* engine, int32_t seq, const void* host_src, int64_t src_bytes,
              int32_t n_tokens);

/* Next tokens from logits: mode 0 = greedy argmax, ties to the lowest id
 * (the paper does not state its sampler).  logits_dev: device fp32
 * [batch][vocab]; tokens_dev_out: device int32 [batch].
 * Errors: PDEC_UNSUPPORTED for any other mode, PDEC_INVALID_ARG. */
int sample(pdec_engine* engine, int32_t batch, const float* logits_dev, int32_t* tokens_dev_out,
           int32_t mode);

/* ---------------------------------------------------------------------------
 * Headroom pacing on this worker (Design, "Separating Departure from
 * Placement": pacing thresholds; Alg. pacing restricted to one worker, the
 * only one a single GPU holds).  A host-only decision; the caller carries it
 * out with kv_export / kv_free (eviction) and kv_alloc / kv_import or
 * kv_append_prefix (placement).
 *   Phase 1: while headroom_tokens < h_min_tokens and residents remain, evict
 *     the longest resident (ties: lower id); the headroom rises by its
 *     active_held_tokens (its pages x 16, reserve included).
 *   Phase 2: the pending trajectories, evicted ones included, in ascending
 *     length (ties: lower id): r is placed when headroom - footprint(r) >=
 *     h_min_tokens + (residents + 1) * delta_tokens, footprint(r) =
 *     ceil(length / 16) * 16; the headroom then falls by footprint(r).
 *   active_*: n_active entries (ids are the caller's); pending_*: n_pending.
 *   evict_out: capacity n_active, in eviction order; place_out: capacity
 *     n_active + n_pending, in placement order; counts in *n_evict_out,
 *     *n_place_out.  Host memory throughout.
 * Errors: PDEC_INVALID_ARG (negative counts, lengths or thresholds, null
 * arrays).
 * ------------------------------------------------------------------------- */
int pacing_plan(int64_t headroom_tokens, int64_t h_min_tokens, int64_t delta_tokens,
                int32_t n_active, const int32_t* active_ids, const int32_t* active_len,
                const int64_t* active_held_tokens, int32_t n_pending, const int32_t* pending_ids,
                const int32_t* pending_len, int32_t* evict_out, int32_t* n_evict_out,
                int32_t* place_out, int32_t* n_place_out);

/* ---------------------------------------------------------------------------
 * Temperature / nucleus (top-p) sampling for RL rollouts, which sample their
 * actions (Background, "RL Post-Training Workflow"; the paper does not state
 * its sampler).  Random numbers are inputs: uniforms_dev holds one u in
 * [0, 1) per row (values outside are clamped).  Per row b, with z the
 * logits, every decision after one fp64 exponential is integer arithmetic:
 *   q_v = rint(exp((z_v - max z) * (1/T)) * 2^40), S = sum q_v,
 *   nucleus = shortest prefix of the tokens ordered by (q desc, index asc)
 *             with mass >= ceil(rint(top_p * 2^24) * S / 2^24),
 *   Z = nucleus mass, target = floor(floor(u * 2^24) * Z / 2^24),
 *   token = first nucleus token in index order whose running mass > target.
 * A given (logits, T, top_p, u) always yields the same token.
 *   logits_dev: device fp32 [batch][vocab]; uniforms_dev: device fp32
 *   [batch]; tokens_dev_out: device int32 [batch].
 *   workspace: device scratch of at least sample_top_p_workspace_bytes(batch)
 *   bytes, owned by the caller, contents ignored on entry; or null (0 bytes),
 *   in which case one work group handles each row.  With it, rows of small
 *   batches are split over several work groups per pass; the tokens are the
 *   same either way.  Calls that share a workspace must not overlap.
 *   Asynchronous on stream.
 * Errors: PDEC_INVALID_ARG (temperature <= 0 or not finite, top_p outside
 * (0, 1], batch or vocab < 1, null pointer, a non-null workspace smaller than
 * required).
 * ------------------------------------------------------------------------- */
int64_t sample_top_p_workspace_bytes(int32_t batch);
int sample_top_p(int32_t batch, int32_t vocab, const float* logits_dev, float temperature,
                 float top_p, const float* uniforms_dev, int32_t* tokens_dev_out,
                 void* workspace, int64_t workspace_bytes, void* stream);

/* sample_top_p for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same tokens as sample_top_p, with the split form's scratch (row states and
 * per-chunk partial results, no more than about 4 MiB) in a static device
 * array that the library holds instead of a caller workspace.  The call
 * itself allocates nothing: the array exists once per GPU, from the time
 * the library is loaded until the process ends, and its device address is
 * looked up on the first call on each device (hipGetSymbolAddress).  Every
 * call on one GPU shares that GPU's array, so calls that overlap on one GPU
 * (on different streams, or from different threads) race and must not be
 * made; calls in one stream's order are safe.  Batches above 32 rows use
 * the one-group form, which needs no scratch.
 * Errors: as sample_top_p (without the workspace cases), and
 * PDEC_INVALID_ARG if a batch would need more scratch than the array holds
 * (the message gives both sizes). */
int sample_top_p_noalloc(int32_t batch, int32_t vocab, const float* logits_dev,
                         float temperature, float top_p, const float* uniforms_dev,
                         int32_t* tokens_dev_out, void* stream);

/* ---------------------------------------------------------------------------
 * Weight packing.  Each decode step streams every projection matrix from HBM
 * once for the whole batch (Introduction; Design Principles, "Specialization
 * in Heterogeneous Pools"), so bf16 matrices are stored in a layout whose
 * stream is long contiguous runs.  Columns form groups of 128 (the last group
 * zero-padded), each group 8 strips of 16 columns; a 16 x 32 block (strip s,
 * k-block b) is 1 KiB in the lane order of the MFMA B operand, and the eight
 * blocks of one k-block of a group are adjacent, so one k-step of 64 of a
 * group is a single 16 KiB run.  Element (n, k) is at
 *   (((G * K/32 + b) * 8 + s) * 64 + q * 16 + c) * 8 + e,
 *   n = 128 G + 16 s + c,  k = 32 b + 8 q + e.
 * fp32 matrices keep the row-major layout (pack_weight copies them).
 *   packed_weight_bytes: size of the packed form of an [N][K] matrix
 *     (bf16: ceil(N/128)*128*K*2 bytes, fp32: N*K*4), or a negative status.
 *   pack_weight: w is a device row-major [N][K] matrix in dtype; packed is a
 *     caller-owned device buffer of packed_weight_bytes(...) bytes, not
 *     overlapping w.  Asynchronous on stream.
 * Errors: PDEC_UNSUPPORTED (bf16 with K % 64 != 0), PDEC_INVALID_ARG.
 * ------------------------------------------------------------------------- */
int64_t packed_weight_bytes(int32_t dtype, int32_t N, int32_t K);

int pack_weight(int32_t dtype, int32_t N, int32_t K, const void* w, void* packed, void* stream);

/* ---------------------------------------------------------------------------
 * Isolated weight projection: out = x W^T with the engine's own plan and
 * kernels (the weight-streaming MFMA kernel up to 32 rows, MFMA tiles beyond,
 * split-K summed in a fixed order).
 *   x: device [M][K] in dtype; w: the [N][K] weight as produced by
 *   pack_weight; out: device fp32 [M][N]; workspace: device, at least
 *   weight_projection_workspace_bytes(...) bytes (may be 0).
 * Errors: PDEC_UNSUPPORTED (bf16 with K % 64 != 0, N % 4 != 0),
 * PDEC_INVALID_ARG.
 * ------------------------------------------------------------------------- */
int64_t weight_projection_workspace_bytes(int32_t dtype, int32_t M, int32_t N, int32_t K);

int weight_projection(int32_t dtype, int32_t M, int32_t N, int32_t K, const void* x,
                      const void* w, float* out, void* workspace, int64_t workspace_bytes,
                      void* stream);

/* ---------------------------------------------------------------------------
 * Isolated gate/up projection with SwiGLU, the first half of the decoder
 * block's feed-forward layer as decode_step and kv_append_prefix run it:
 *   u[m][n] = silu(g) * up,  g = x[m] . w_gate[n],  up = x[m] . w_up[n],
 *   silu(z) = z / (1 + exp(-z)),  n < F.
 * When one work group per column group covers K (bf16 whenever the planner
 * chooses no K split, as for every 8B-shaped batch), the product and the
 * SwiGLU run in one kernel and the fp32 gate/up values never reach memory;
 * otherwise the split-K partials go to the workspace and a second kernel sums
 * them and applies SwiGLU with the same fp32 arithmetic.  Up to 256 rows, if
 * the fused kernel's work groups would fill whole rounds of the GPU's 256
 * compute units plus a last round at most half full (F = 17408, the 14B
 * shape's FFN), the columns of that last round take the split form instead
 * (its partials in the workspace), so the tail runs as one round of short
 * work groups.
 *   x: device [M][K] in dtype; w_gate, w_up: [F][K] weights as produced by
 *   pack_weight; u: device [M][F] in dtype (bf16 rounded to nearest even);
 *   workspace: device, at least swiglu_projection_workspace_bytes(...) bytes
 *   (may be 0).
 * Errors: PDEC_UNSUPPORTED (bf16 with K % 64 != 0, F % 4 != 0),
 * PDEC_INVALID_ARG.
 * ------------------------------------------------------------------------- */
int64_t swiglu_projection_workspace_bytes(int32_t dtype, int32_t M, int32_t F, int32_t K);

int swiglu_projection(int32_t dtype, int32_t M, int32_t F, int32_t K, const void* x,
                      const void* w_gate, const void* w_up, void* u, void* workspace,
                      int64_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Isolated paged decode attention (one layer, no engine).
 *
 * For each sequence b and query head h (KV head g = h / (n_q_heads /
 * n_kv_heads)): out[b][h] = softmax(q[b][h] . K_g^T / sqrt(head_dim)) V_g over
 * the lens[b] cached positions of b.  Long-context decode attention is the
 * memory-bandwidth-bound part of the step (Design Principles,
 * "Specialization in Heterogeneous Pools").
 *   q: device [batch][n_q_heads][head_dim] in dtype;
 *   k_pages: device [n_pages][n_kv_heads][16][head_dim];
 *   v_pages: device [n_pages][n_kv_heads][head_dim][16];
 *   block_table_dev: device int32 [batch][bt_stride], logical page order;
 *   lens_host: host int32 [batch], each in [1, bt_stride * 16];
 *   out: device fp32 [batch][n_q_heads][head_dim];
 *   workspace: device, at least paged_attention_workspace_bytes(...) bytes
 *     (max_total_tokens is accepted for compatibility and ignored: the work
 *     list is bounded by the batch alone), owned by the caller; it holds the
 *     work list and the per-item partial results.  Calls that share a
 *     workspace must not overlap.
 * The work list is planned on the host and copied through a small pinned
 * staging ring that the library allocates on the first call and keeps.
 * Slots past lens[b] in the last page are never read.  Asynchronous on
 * stream.
 * Errors: PDEC_INVALID_ARG (null pointers, sizes < 1, n_q_heads not a
 * multiple of n_kv_heads, lens[b] outside [1, bt_stride * 16], workspace too
 * small), PDEC_UNSUPPORTED (head_dim other than 64 / 128, GQA group size
 * above 16), PDEC_HIP_ERROR.
 * ------------------------------------------------------------------------- */
int64_t paged_attention_workspace_bytes(int32_t batch, int32_t n_q_heads, int32_t n_kv_heads,
                                        int32_t head_dim, int64_t max_total_tokens);

int paged_decode_attention(int32_t dtype, int32_t batch, int32_t n_q_heads, int32_t n_kv_heads,
                           int32_t head_dim, const void* q, const void* k_pages,
                           const void* v_pages, const int32_t* block_table_dev, int32_t bt_stride,
                           const int32_t* lens_host, float* out, void* workspace,
                           int64_t workspace_bytes, void* stream);

/* The same with PDEC_FP8_E4M3 pages: q is bf16 [batch][n_q_heads][head_dim];
 * k_pages / v_pages hold codes in the page layout above (one byte per
 * element) that read back as value(code) * k_scale and value(code) * v_scale.
 * Errors as paged_decode_attention, and PDEC_INVALID_ARG for scales that are
 * not positive and finite. */
int paged_decode_attention_fp8(int32_t batch, int32_t n_q_heads, int32_t n_kv_heads,
                               int32_t head_dim, const void* q, const void* k_pages,
                               const void* v_pages, float k_scale, float v_scale,
                               const int32_t* block_table_dev, int32_t bt_stride,
                               const int32_t* lens_host, float* out, void* workspace,
                               int64_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* PDEC_H */

// Host-callable launchers of the gfx950 kernels.  Every launcher only
// enqueues on the given stream; argument checks are the caller's job (the
// engine validates shapes before any launch).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "meta.h"

namespace pdec {

// Weight matrix made of up to 3 row segments stacked along N (e.g. q|k|v or
// gate|up).  Segment s covers output columns [row_end[s-1], row_end[s]).
// bf16 segments are packed separately, each padded to whole 128-column
// groups; grp_end[s] counts the groups of segments 0..s (launch_gemm fills
// it from row_end).
struct WSegs {
  const void* ptr[3];
  int32_t row_end[3];
  int32_t n_seg;
  int32_t grp_end[3];
};

// ---- attention --------------------------------------------------------------
// Split pass: one work group per (item, KV head).  rows_per_item = 16
// (decode), 64 (prefill, fp8 pages or 64-dim heads) or 128 (prefill, bf16
// pages and 128-dim heads: the LDS-staged prefill kernel).  Writes per-row partial softmax
// statistics part_ml [items][Hkv][rows_per_item][2] = (max in log2 units,
// sum) and unnormalised outputs part_acc [items][Hkv][rows_per_item][head_dim].
// kv_fp8: K/V pages hold E4M3 codes read back as code * k_scale / v_scale.
hipError_t launch_attention_split(int dtype, int kv_fp8, float k_scale, float v_scale,
                                  int head_dim, int rows_per_item, int n_items,
                                  int n_q_heads,
                                  int n_kv_heads, const AttnItem* items,
                                  const AttnQBlock* qblocks, const void* q, const void* k_pages,
                                  const void* v_pages, int64_t page_stride_elems,
                                  const int32_t* block_table, int32_t bt_stride, float* part_ml,
                                  float* part_acc, hipStream_t stream,
                                  hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr);

// The LDS-staged prefill kernel (attention_prefill.hip) behind
// launch_attention_split for 128- or 256-row items with 128-dim heads, bf16
// pages (kv_fp8 = 0) or E4M3 pages (kv_fp8 = 1; scale_log2 then includes the
// K scale, and v_scale multiplies the partial outputs); scale_log2 =
// log2(e) / sqrt(head_dim) [* k_scale].
hipError_t launch_attention_prefill_bf16(int n_items, int rows_per_item, int n_q_heads,
                                         int n_kv_heads, int kv_fp8, const AttnItem* items,
                                         const AttnQBlock* qblocks, const void* q,
                                         const void* k_pages, const void* v_pages,
                                         int64_t page_stride_elems, const int32_t* block_table,
                                         int32_t bt_stride, float scale_log2, float v_scale,
                                         float* part_ml, float* part_acc, hipStream_t stream,
                                         hipEvent_t ev_start = nullptr,
                                         hipEvent_t ev_stop = nullptr);

// Merge pass for prefill blocks (rows_per_item >= 64): one work group per
// (query block, KV head, 16 rows), each row merging its block's items in
// item order; same partial layout and output as launch_attention_combine.
hipError_t launch_attention_combine_rows(int head_dim, int rows_per_item, int n_qblocks,
                                         int n_q_heads, int n_kv_heads, const AttnQBlock* qblocks,
                                         const float* part_ml, const float* part_acc, void* out,
                                         int out_bf16, hipStream_t stream);

// Merge pass: one work group per (query block, KV head); writes
// out [rows][n_q_heads][head_dim] as fp32 (out_bf16 = 0) or bf16.
hipError_t launch_attention_combine(int head_dim, int rows_per_item, int n_qblocks,
                                    int max_items, int n_q_heads, int n_kv_heads,
                                    const AttnQBlock* qblocks, const float* part_ml,
                                    const float* part_acc, void* out, int out_bf16,
                                    hipStream_t stream);

// ---- projections ------------------------------------------------------------
// out[s][m][n] = sum_{k in split s} A[m][k] * W[n][k]  (fp32 partial sums).
// bf16: A and W bf16, K % 64 == 0, k_split % 64 == 0.  f32: any sizes.
// Launchers taking ev_start/ev_stop record the kernel's own begin and end in
// them when given (timing without marker packets between kernels).
hipError_t launch_gemm(int dtype, int M, int N, int K, const void* A, int64_t lda,
                       const WSegs& w, float* out, int splits, int k_split, hipStream_t stream,
                       hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr);
// bf16 gate/up projection with the SwiGLU epilogue, no K split:
// u[m][n] = bf16(silu(g) * up), g and up the products of row m of A with
// column n of the packed gate and up matrices ([F][K] each), n < F.  Equals
// launch_gemm over the two segments (splits = 1) followed by launch_swiglu.
// Where the fused grid would leave a second round of work groups at most
// half full (up to 256 rows), the columns of that tail take launch_gemm with
// a K split into tail_part (fp32, at least swiglu_tail_part_elems floats)
// and launch_swiglu; with tail_part null the whole product is fused.
hipError_t launch_gemm_swiglu(int M, int F, int K, const void* A, int64_t lda, const void* w_gate,
                              const void* w_up, void* u, float* tail_part, hipStream_t stream,
                              hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr);
// fp32 elements launch_gemm_swiglu needs in tail_part for this shape (0: fused only).
int64_t swiglu_tail_part_elems(int M, int F, int K);
// Temperature / top-p sampling (sample.hip).
// With a workspace of sample_workspace_bytes(B) (> 0 only for small batches)
// every pass is split over several work groups per row; same tokens.
int64_t sample_workspace_bytes(int B);
// The static scratch of sample_top_p_noalloc: its size (at least
// sample_workspace_bytes(B) for every B) and this GPU's device address of it
// (looked up on the first call per device).
int64_t sample_scratch_bytes();
hipError_t sample_scratch_ptr(void** out);
hipError_t launch_sample_top_p(int B, int V, const float* logits, float temperature, float top_p,
                               const float* uniforms, int32_t* tokens, void* workspace,
                               int64_t ws_bytes, hipStream_t stream);
// bf16: pack a row-major [N][K] weight into the group-major layout the GEMM
// kernels read (((N + 127) / 128) * 128 * K elements); fp32: plain copy.
hipError_t launch_pack_weight(int dtype, int N, int K, const void* w, void* packed,
                              hipStream_t stream);
// Number of K splits the launcher plans for this shape (and the split size).
int gemm_plan_splits(int dtype, int M, int N, int K, int* k_split);

// ---- per-row and elementwise steps -------------------------------------------
// x[m] = E[tok[m]];  h[m] = rmsnorm(x[m]) * gain.  Ids are clamped to [0, vocab).
hipError_t launch_embed_norm(int dtype, int M, int d, int vocab, const int32_t* tokens,
                             const void* embed,
                             const float* gain, float eps, float* x, void* h, hipStream_t stream);
// x[m] += sum_s part[s][m];  h[m] = rmsnorm(x[m]) * gain.
hipError_t launch_resid_norm(int dtype, int M, int d, const float* part, int splits, float* x,
                             const float* gain, float eps, void* h, hipStream_t stream);
// Sum the q|k|v partials, rotate q and k at each row's position (cos/sin
// table [pos][head_dim/2] of float2), write q to q_out [M][Hq][Dh] and k, v
// into the row's page slot of this layer's pool.
hipError_t launch_qkv_rope_kv(int dtype, int kv_fp8, float k_scale, float v_scale, int M,
                              int head_dim, int n_q_heads, int n_kv_heads, const float* part,
                              int splits, const RowMeta* rows, const float2* rope_cs,
                              const int32_t* block_table, int32_t bt_stride, void* q_out,
                              void* k_pages, void* v_pages, int64_t page_stride_elems,
                              const float* q_gain, const float* k_gain, float eps,
                              hipStream_t stream);
// u[m][n] = silu(g) * up with g, up the summed partials of columns n and F+n.
// Row m of u starts at u + m * ldu (ldu 0: F).
hipError_t launch_swiglu(int dtype, int M, int F, const float* part, int splits, void* u,
                         hipStream_t stream, int64_t ldu = 0);
// out[i] = sum_s part[s][i] over `splits` slabs of n floats (n % 4 == 0).
hipError_t launch_sum_splits(int64_t n, const float* part, int splits, float* out,
                             hipStream_t stream);
// dst[i] = src[idx[i]] for n rows of row_bytes bytes (row_bytes % 4 == 0).
hipError_t launch_gather_rows(int n, const int32_t* idx, const void* src, int64_t row_bytes,
                              void* dst, hipStream_t stream);
// tokens[b] = argmax_v logits[b][v] (lowest index on ties).
hipError_t launch_argmax(int B, int V, const float* logits, int32_t* tokens, hipStream_t stream);
// bt[d.slot * stride + d.idx] = d.page for each delta.
hipError_t launch_bt_deltas(int n, const BtDelta* deltas, int32_t* bt, int32_t stride,
                            hipStream_t stream);
// cs[p][i] = (cos, sin)(p * base^(-2i/Dh)) evaluated in double precision.
hipError_t launch_rope_table(int max_pos, int head_dim, double base, float2* cs,
                             hipStream_t stream);

// ---- KV snapshot / restore ---------------------------------------------------
// Copy whole pages between the pool and a host buffer mapped for the device.
// Page i of the list moves between pool block [layer][kind][pages[i]] and
// host bytes [(i * n_layers * 2 + layer * 2 + kind) * block_bytes, + block_bytes).
hipError_t launch_kv_page_copy(int n_pages, const int32_t* pages_dev, int n_layers,
                               int64_t n_pool_pages, int64_t block_bytes, void* pool,
                               void* host_dev_ptr, int to_host, hipStream_t stream);

}  // namespace pdec

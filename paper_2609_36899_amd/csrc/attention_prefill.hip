// LDS-staged prefill attention for gfx950 (bf16 pages, 128-dim heads).
//
// Chunked prefill (the re-prefill path that rebuilds a trajectory's KV from
// its tokens, paper: KV Preparation for Late-Bound Placement) presents 128-row query
// blocks: 128/G queries of one chunk times the G query heads of a GQA group.
// Such blocks are MFMA-bound rather than HBM-bound, so this kernel shares each
// page between four waves through LDS instead of letting every wave stream it.
// It writes the same partials as the decode split kernel; they are merged by
// the row-split merge pass below.
#include "hip_common.h"
#include "kernels.h"

namespace pdec {

namespace {
// ---------------------------------------------------------------------------
// Prefill, bf16 pages.  A work group of 4 waves takes one (item, KV head) of
// a 128-row query block (128/G queries x G heads); wave w owns rows
// 32w .. 32w+31 as two 16-row tiles.  All four waves need every key of the
// item, so the pages pass through LDS two at a time (a stage: K of both
// pages, then V^T of both), fetched by LDS-DMA into a ring of four stages and
// read from there by every wave: each page crosses L2 once per work group
// rather than once per wave, and two stages stay in flight while one is
// used.  Each K and V fragment a wave reads from LDS serves both of its row
// tiles, which halves LDS traffic per MFMA against one tile per wave.  The
// math per page pair and row tile is the split kernel's (S^T = K Q^T,
// online softmax, O^T = V^T P^T).
//
// K rows in LDS: the 16-byte chunk j of key k of page p sits in slot
// j ^ kswz(k, p), so that the lanes of one fragment read (8 or 16 keys of the
// same chunk column) hit distinct banks; the swizzle goes on the DMA's source
// address.  V^T blocks are copied as they are (a fragment read covers 16
// dims x 32 bytes, already conflict-free).
// ---------------------------------------------------------------------------
__device__ __forceinline__ int kswz(int k, int p) {
  return (k & 3) | (((k >> 3) & 1) << 2) | (p << 3);  // < 16 chunks per 128-dim key row
}

// Pages of E4M3 codes (KT = uint8_t) are staged through registers instead:
// after the barrier each thread loads the 8-byte code chunks of its four LDS
// chunks of the next stage, and after the stage's compute it converts them to
// bf16 (exact: every E4M3 value is a bf16 value) and writes them where the
// DMA would have put the bf16 chunks.  Each code is converted once per work
// group rather than once per wave, and the compute is the bf16 one.  The K
// scale is folded into scale_log2 by the caller; the V scale multiplies the
// partial output once.
//
// WAVES = 4 takes 128-row blocks (two work groups per CU).  WAVES = 8 takes
// 256-row blocks: the same stages then feed twice the MFMA work, which halves
// the load work (DMA issue and LDS writes) per flop; the engine picks it for
// passes whose blocks read long key ranges, where that work weighs most.
template <int DH, typename KT, int WAVES>  // DH = 128; KT = uint16_t (bf16) or uint8_t (E4M3)
__global__ __launch_bounds__(64 * WAVES) __attribute__((amdgpu_waves_per_eu(2))) void attn_prefill_bf16(
    const AttnItem* __restrict__ items, const AttnQBlock* __restrict__ qblocks,
    const uint16_t* __restrict__ q, const KT* __restrict__ kpool,
    const KT* __restrict__ vpool, int64_t page_stride, const int32_t* __restrict__ bt,
    int32_t bt_stride, int32_t n_q_heads, int32_t n_kv_heads, float scale_log2, float v_scale,
    float* __restrict__ part_ml, float* __restrict__ part_acc) {
  constexpr bool kFp8 = sizeof(KT) == 1;
  constexpr int KC = DH / 32;   // k-steps of QK^T
  constexpr int DT = DH / 16;   // 16-wide dim tiles of PV
  constexpr int RT = 2;         // 16-row tiles per wave
  constexpr int THREADS = 64 * WAVES;
  constexpr int R = 16 * RT * WAVES;  // query rows per item
  constexpr int BLK = kPage * DH;          // elements of one page's K (or V^T) block
  constexpr int STAGE = 4 * BLK;           // K0 K1 V0 V1
  constexpr int CPK = DH / 8;              // 16-byte chunks per K row
  constexpr int LPT = STAGE * 2 / 16 / THREADS;  // DMA loads per thread per stage
  constexpr int D = 4;
  static_assert(DH == 128, "the K swizzle spans 16 chunks per key row");
  static_assert(WAVES == 4 || WAVES == 8, "128- or 256-row blocks");
  static_assert(LPT * THREADS * 8 == STAGE, "stage is a whole number of loads");
  __shared__ __attribute__((aligned(16))) uint16_t st0[STAGE];
  __shared__ __attribute__((aligned(16))) uint16_t st1[STAGE];
  __shared__ __attribute__((aligned(16))) uint16_t st2[STAGE];
  __shared__ __attribute__((aligned(16))) uint16_t st3[STAGE];
  auto stage_ptr = [&](int b) -> uint16_t* { return b == 0 ? st0 : b == 1 ? st1 : b == 2 ? st2 : st3; };

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int c16 = lane & 15, q4 = lane >> 4;
  const int g = blockIdx.x, item_id = items[blockIdx.y].order;
  const AttnItem it = items[item_id];
  const AttnQBlock qb = qblocks[it.qblock];
  const int G = n_q_heads / n_kv_heads;

  const int key0 = it.page_begin * kPage;
  const int key_end = (it.page_begin + it.n_pages) * kPage;
  const int kv_lim = min(qb.pos0 + qb.n_q, key_end);  // keys at or past it hold no data

  // This lane's query row in tile r.  Waves without rows still take part in
  // the stage loads and barriers; their results are not written.
  int row[RT], row_lim[RT];
  bool row_valid[RT];
  bf16x8 qf[RT][KC];
#pragma unroll
  for (int r = 0; r < RT; ++r) {
    row[r] = wave * 16 * RT + 16 * r + c16;
    const int jq = row[r] / G, head = g * G + (row[r] % G);
    row_valid[r] = jq < qb.n_q;
    row_lim[r] = row_valid[r] ? min(qb.pos0 + jq + 1, key_end) : key0;
    if (row_valid[r]) {
      const uint16_t* qrow = q + ((int64_t)(qb.q_row0 + jq) * n_q_heads + head) * DH;
#pragma unroll
      for (int c = 0; c < KC; ++c) qf[r][c] = *(const bf16x8*)(qrow + c * 32 + q4 * 8);
    } else {
#pragma unroll
      for (int c = 0; c < KC; ++c) qf[r][c] = bf16x8{};
    }
  }

  const int32_t* btrow = bt + (int64_t)qb.slot * bt_stride + it.page_begin;
  const int64_t head_off = (int64_t)g * BLK;
  const int n_st = (it.n_pages + 1) >> 1;
  const int last = n_st - 1;

  // DMA: load j of a stage fills chunk id = j * THREADS + tid of the stage,
  // i.e. chunk id & 255 of block id >> 8 (K page 0, K page 1, V page 0,
  // V page 1).  With four waves load j fills block j; with eight, blocks 2j
  // and 2j + 1 (the block is uniform over a wave).
  int src_off[LPT], src_blk[LPT];
#pragma unroll
  for (int j = 0; j < LPT; ++j) {
    const int blk = j * (WAVES / 4) + (WAVES == 8 ? (tid >> 8) : 0), c = tid & 255;
    src_blk[j] = blk;
    if (blk < 2) {
      const int k = c / CPK, slot = c % CPK;
      src_off[j] = k * DH + ((slot ^ kswz(k, blk)) * 8);
    } else {
      src_off[j] = c * 8;
    }
  }
  // The stage's two page numbers are read with uniform indices (scalar
  // loads): a per-lane page-table read would be a vector load, and waiting
  // for it would also wait for every stage in flight (loads retire in order).
  // A missing second page reads a valid page whose keys are masked.
  auto page_a_of = [&](int st) { return btrow[2 * st]; };
  auto page_b_of = [&](int st) { return btrow[min(2 * st + 1, it.n_pages - 1)]; };
  auto issue = [&](int page_a, int page_b, int buf) {
    uint16_t* base = stage_ptr(buf) + wave * 64 * 8;
    const int64_t base_a = (int64_t)page_a * page_stride + head_off;
    const int64_t base_b = (int64_t)page_b * page_stride + head_off;
#pragma unroll
    for (int j = 0; j < LPT; ++j)
      dma16((src_blk[j] < 2 ? kpool : vpool) + ((src_blk[j] & 1) ? base_b : base_a) + src_off[j],
            base + j * THREADS * 8);
  };
  // E4M3 pages: the codes of chunk j of a stage (8 bytes), then their bf16
  // values into LDS chunk j * THREADS + tid, as the DMA would place them.
  u32x2 codes[LPT];
  auto load_codes = [&](int page_a, int page_b) {
    const int64_t base_a = (int64_t)page_a * page_stride + head_off;
    const int64_t base_b = (int64_t)page_b * page_stride + head_off;
#pragma unroll
    for (int j = 0; j < LPT; ++j)
      codes[j] = load_stream<u32x2>((src_blk[j] < 2 ? kpool : vpool) +
                                    ((src_blk[j] & 1) ? base_b : base_a) + src_off[j]);
  };
  auto store_codes = [&](int buf) {
    uint16_t* base = stage_ptr(buf) + tid * 8;
#pragma unroll
    for (int j = 0; j < LPT; ++j) *(bf16x8*)(base + j * THREADS * 8) = e4m3x8_to_bf16(codes[j]);
  };

  // Lane-constant fragment offsets (as in the split kernel).
  const int k_tok = 8 * ((c16 >> 2) & 1) + (c16 & 3);  // + 4u
  const int k_page_sel = c16 >> 3;
  const int v_page_sel = q4 >> 1;
  const int v_tok0 = 8 * (q4 & 1);

  float m[RT];  // running max of scaled scores (log2 units), row-uniform
  // The normaliser comes out of one more MFMA per tile: an all-ones A
  // operand times P^T sums each row's rounded weights (element 0 of every
  // lane is its row's sum; the other elements are not used).
  f32x4 lacc[RT];
  f32x4 acc[RT][DT];
#pragma unroll
  for (int r = 0; r < RT; ++r) {
    m[r] = -INFINITY;
    lacc[r] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < DT; ++t) acc[r][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const bf16x8 ones = __builtin_bit_cast(bf16x8, u16x8{0x3F80, 0x3F80, 0x3F80, 0x3F80, 0x3F80,
                                                       0x3F80, 0x3F80, 0x3F80});
  // Stages wholly below every row's causal limit need no mask (keys below
  // pos0 + 1 are visible to all rows of the block; rows past the block's
  // queries are computed too and never written).
  const int open_end = min(qb.pos0 + 1, key_end);

  auto compute = [&](int st, int buf) {
    const uint16_t* sb = stage_ptr(buf);
    bf16x8 kf[2][KC];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int k = k_tok + 4 * u;
      const uint16_t* kr = sb + k_page_sel * BLK + k * DH;
#pragma unroll
      for (int c = 0; c < KC; ++c)
        kf[u][c] = *(const bf16x8*)(kr + (((4 * c + q4) ^ kswz(k, k_page_sel)) * 8));
    }
    const int kbase = key0 + (2 * st + v_page_sel) * kPage + v_tok0;
    const bool open = key0 + (2 * st + 2) * kPage <= open_end;  // uniform
    bf16x8 pf[RT];
#pragma unroll
    for (int r = 0; r < RT; ++r) {
      f32x4 s[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        s[u] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < KC; ++c)
          s[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[u][c], qf[r][c], s[u], 0, 0, 0);
      }
      // Raw scores; the scale (> 0) is applied to the max and inside the
      // exponent's FMA.  Masked keys are -inf, whose weight is exactly 0.
      // The mask sits under a uniform branch: most stages need none, and a
      // select merged with the open test would cost three VALU ops a score.
      float sv[8];
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) sv[4 * u + rr] = s[u][rr];
      if (!open) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          sv[e] = (kbase + e < row_lim[r]) ? sv[e] : -INFINITY;
      }
      float mloc = max2(max2(max2(sv[0], sv[1]), sv[2]), max2(max2(sv[3], sv[4]), sv[5]));
      mloc = max_over_key_groups(max2(max2(mloc, sv[6]), sv[7]));
      const float m_new = max2(m[r], mloc * scale_log2);
      const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
      if (__any(m_new != m[r])) {
        const float alpha = __builtin_amdgcn_exp2f(m[r] - m_use);
        lacc[r][0] *= alpha;
#pragma unroll
        for (int t = 0; t < DT; ++t) acc[r][t] *= alpha;
      }
      m[r] = m_new;
      uint32_t pw4[4];
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const f32x2 pv = {__builtin_amdgcn_exp2f(__builtin_fmaf(sv[e], scale_log2, -m_use)),
                          __builtin_amdgcn_exp2f(__builtin_fmaf(sv[e + 1], scale_log2, -m_use))};
        pw4[e / 2] = __builtin_bit_cast(uint32_t, __builtin_convertvector(pv, bf16x2));
      }
      pf[r] = __builtin_bit_cast(bf16x8, u32x4{pw4[0], pw4[1], pw4[2], pw4[3]});
    }
    u16x8 vf[DT];
#pragma unroll
    for (int t = 0; t < DT; ++t)
      vf[t] = *(const u16x8*)(sb + (2 + v_page_sel) * BLK + (t * 16 + c16) * kPage + v_tok0);
    if (__builtin_expect(key0 + (2 * st + 2) * kPage > kv_lim, 0)) {  // the block's last keys
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (kbase + e >= kv_lim)
#pragma unroll
          for (int t = 0; t < DT; ++t) vf[t][e] = 0;
    }
#pragma unroll
    for (int r = 0; r < RT; ++r) {
#pragma unroll
      for (int t = 0; t < DT; ++t)
        acc[r][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vf[t]),
                                                            pf[r], acc[r][t], 0, 0, 0);
      lacc[r] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pf[r], lacc[r], 0, 0, 0);
    }
  };

  // Ring of D stages, two in flight while one is used (stage indices
  // clamped to the last, so every step issues one stage and the count of
  // loads in flight is fixed).  After the barrier of step st every wave has
  // finished step st-1, whose stage then takes step st+3.
#pragma unroll
  for (int b = 0; b < D - 1; ++b) {
    if constexpr (kFp8) {
      load_codes(page_a_of(min(b, last)), page_b_of(min(b, last)));
      store_codes(b);
    } else {
      issue(page_a_of(min(b, last)), page_b_of(min(b, last)), b);
    }
  }
  // Page numbers of the next stage to issue, read one step ahead so that the
  // wait for the scalar loads (which also waits for LDS reads) finds them
  // arrived.
  int next_a = page_a_of(min(D - 1, last)), next_b = page_b_of(min(D - 1, last));
  auto step = [&](int s, int b) {
    if constexpr (kFp8) {
      wait_lds();  // this wave's stage writes of the previous step
      wg_barrier();
      load_codes(next_a, next_b);  // stage min(s + D - 1, last)
    } else {
      wait_vmem<(D - 2) * LPT>();
      wg_barrier();
      issue(next_a, next_b, (b + D - 1) % D);  // stage min(s + D - 1, last)
    }
    next_a = page_a_of(min(s + D, last));
    next_b = page_b_of(min(s + D, last));
    __builtin_amdgcn_sched_barrier(0);
    compute(s, b);
    // The stage of step s - 1, free since this step's barrier.
    if constexpr (kFp8) store_codes((b + D - 1) % D);
  };
  int st = 0;
  for (; st + D <= n_st; st += D) {
#pragma unroll
    for (int b = 0; b < D; ++b) step(st + b, b);
  }
  const int tail = n_st - st;  // uniform over the work group
#pragma unroll
  for (int b = 0; b < D; ++b)
    if (b < tail) step(st + b, b);
  wait_vmem<0>();  // no LDS write may still be in flight when the group ends
  if constexpr (kFp8) {
    wait_lds();
#pragma unroll
    for (int r = 0; r < RT; ++r)
#pragma unroll
      for (int t = 0; t < DT; ++t) acc[r][t] *= v_scale;
  }

#pragma unroll
  for (int r = 0; r < RT; ++r) {
    if (!row_valid[r]) continue;
    const int64_t prow = ((int64_t)item_id * n_kv_heads + g) * R + row[r];
    if (q4 == 0) {
      part_ml[prow * 2] = m[r];
      part_ml[prow * 2 + 1] = lacc[r][0];
    }
    float* pa = part_acc + prow * DH;
#pragma unroll
    for (int t = 0; t < DT; ++t) *(f32x4*)(pa + t * 16 + 4 * q4) = acc[r][t];
  }
}

// ---------------------------------------------------------------------------
// Merge of prefill partials.  A prefill query block has up to 128 rows and a
// handful of items, so the work is split by rows, not by items: a work group
// of 4 waves takes 16 rows (4 per wave, 16 lanes x DH/16 dims per row) and
// each row merges all of its block's items in item order with the
// online-softmax rule (m = max(m, m_i); l = l 2^(m_old-m) + l_i 2^(m_i-m);
// o likewise; output o / l), four items' loads in flight at a time.  No
// LDS and no barriers; the result does not depend on which work group runs
// when.
// ---------------------------------------------------------------------------
template <int DPL>
__device__ __forceinline__ void merge_row(float& m, float& l, float* o, float mi, float li,
                                          const float* oi) {
  const float mn = fmaxf(m, mi);
  const float mu = (mn == -INFINITY) ? 0.f : mn;  // both empty: keep zeros
  const float so = exp2f(m - mu), si = exp2f(mi - mu);
  l = l * so + li * si;
#pragma unroll
  for (int e = 0; e < DPL; ++e) o[e] = o[e] * so + oi[e] * si;
  m = mn;
}

template <int DH, typename OutT>
__global__ __launch_bounds__(256) void attn_combine_rows(const AttnQBlock* __restrict__ qblocks,
                                                         const float* __restrict__ part_ml,
                                                         const float* __restrict__ part_acc,
                                                         int32_t n_q_heads, int32_t n_kv_heads,
                                                         int32_t R, OutT* __restrict__ out) {
  constexpr int DPL = DH / 16;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int d0 = (lane & 15) * DPL;
  const AttnQBlock qb = qblocks[blockIdx.x];
  const int g = blockIdx.y;
  const int G = n_q_heads / n_kv_heads;
  const int r = blockIdx.z * 16 + wave * 4 + (lane >> 4);
  if (r >= qb.n_q * G) return;  // no barriers in this kernel
  float m = -INFINITY, l = 0.f, o[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) o[e] = 0.f;
  for (int i0 = qb.item_begin; i0 < qb.item_end; i0 += 4) {
    float2 ml[4];
    float a[4][DPL];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = min(i0 + u, qb.item_end - 1);
      const int64_t prow = ((int64_t)i * n_kv_heads + g) * R + r;
      ml[u] = *(const float2*)(part_ml + prow * 2);
#pragma unroll
      for (int e = 0; e < DPL; e += 4) {
        const float4 v = *(const float4*)(part_acc + prow * DH + d0 + e);
        a[u][e] = v.x;
        a[u][e + 1] = v.y;
        a[u][e + 2] = v.z;
        a[u][e + 3] = v.w;
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (i0 + u >= qb.item_end) break;
      merge_row<DPL>(m, l, o, ml[u].x, ml[u].y, a[u]);
    }
  }
  const float inv = 1.f / l;
  const int jq = r / G, head = g * G + r % G;
  OutT* orow = out + ((int64_t)(qb.q_row0 + jq) * n_q_heads + head) * DH + d0;
#pragma unroll
  for (int e = 0; e < DPL; ++e) orow[e] = Store<OutT>::from(o[e] * inv);
}

}  // namespace

hipError_t launch_attention_combine_rows(int head_dim, int rows_per_item, int n_qblocks,
                                         int n_q_heads, int n_kv_heads, const AttnQBlock* qblocks,
                                         const float* part_ml, const float* part_acc, void* out,
                                         int out_bf16, hipStream_t stream) {
  if (n_qblocks == 0) return hipSuccess;
  const dim3 grid(n_qblocks, n_kv_heads, (rows_per_item + 15) / 16);
  if (head_dim == 128) {
    if (out_bf16)
      attn_combine_rows<128, uint16_t><<<grid, 256, 0, stream>>>(
          qblocks, part_ml, part_acc, n_q_heads, n_kv_heads, rows_per_item, (uint16_t*)out);
    else
      attn_combine_rows<128, float><<<grid, 256, 0, stream>>>(
          qblocks, part_ml, part_acc, n_q_heads, n_kv_heads, rows_per_item, (float*)out);
  } else {
    if (out_bf16)
      attn_combine_rows<64, uint16_t><<<grid, 256, 0, stream>>>(
          qblocks, part_ml, part_acc, n_q_heads, n_kv_heads, rows_per_item, (uint16_t*)out);
    else
      attn_combine_rows<64, float><<<grid, 256, 0, stream>>>(
          qblocks, part_ml, part_acc, n_q_heads, n_kv_heads, rows_per_item, (float*)out);
  }
  return hipGetLastError();
}

hipError_t launch_attention_prefill_bf16(int n_items, int rows_per_item, int n_q_heads,
                                         int n_kv_heads, int kv_fp8, const AttnItem* items,
                                         const AttnQBlock* qblocks, const void* q,
                                         const void* k_pages, const void* v_pages,
                                         int64_t page_stride_elems, const int32_t* block_table,
                                         int32_t bt_stride, float scale_log2, float v_scale,
                                         float* part_ml, float* part_acc, hipStream_t stream,
                                         hipEvent_t ev_start, hipEvent_t ev_stop) {
  if (n_items == 0) return hipSuccess;
  if (rows_per_item != 128 && rows_per_item != 256) return hipErrorInvalidValue;
  // 32 rows per wave: 4 waves (256 threads) for 128 rows, 8 (512) for 256.
  const dim3 grid(n_kv_heads, n_items), block(2 * rows_per_item);
  const uint16_t* qq = (const uint16_t*)q;
#define PDEC_PREFILL(KT_, WAVES_, VS_)                                                          \
  return launch_timed(attn_prefill_bf16<128, KT_, WAVES_>, grid, block, stream, ev_start,     \
                      ev_stop, items, qblocks, qq, (const KT_*)k_pages, (const KT_*)v_pages,  \
                      page_stride_elems, block_table, bt_stride, n_q_heads, n_kv_heads,       \
                      scale_log2, VS_, part_ml, part_acc)
  if (kv_fp8) {
    if (rows_per_item == 256) PDEC_PREFILL(uint8_t, 8, v_scale);
    PDEC_PREFILL(uint8_t, 4, v_scale);
  }
  if (rows_per_item == 256) PDEC_PREFILL(uint16_t, 8, 1.f);
  PDEC_PREFILL(uint16_t, 4, 1.f);
#undef PDEC_PREFILL
}

}  // namespace pdec

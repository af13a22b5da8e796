// Paged split-K decode/prefill attention for gfx950.
//
// Long-context decode attention is bound by HBM bandwidth (paper: Design
// Principles, "Specialization in Heterogeneous Pools"): every cached K/V byte
// of a trajectory is read once per step.  The key axis of each query block
// is cut into work items of whole pages; each (item, KV head) work group
// streams its pages once, applies them to every query head of the GQA group,
// and leaves an online-softmax partial (max, sum, unnormalised output) that
// the combine pass merges.  Query rows of a block = (query, head-in-group)
// pairs: one query (G rows) per decode block; 128/G or 256/G queries per
// prefill block for the LDS-staged prefill kernel (128-dim heads, bf16 or
// E4M3 pages: attention_prefill.hip) and 64/G for the row-wave form of the
// split kernel here (64-dim heads).
//
// bf16 path: both products run on MFMA (v_mfma_f32_16x16x32_bf16).  Scores are
// computed transposed, S^T = K Q^T, so that each lane's output column is one
// query row; that keeps every softmax statistic lane-private and lets the
// score registers feed the P operand of O^T = V^T P^T without any shuffle.
// V pages are stored transposed ([Dh][16]) so each lane's V^T operand is one
// contiguous 16-byte load (8 bytes with fp8 pages).
#include "hip_common.h"
#include "kernels.h"

namespace pdec {

namespace {

constexpr float kLog2e = 1.4426950408889634f;

// Eight consecutive K or V elements as a bf16 MFMA fragment.  fp8 pages are
// read as 8 bytes (half the traffic) and decoded in registers; the decode is
// exact, so both products still run on bf16 MFMAs.
template <typename KT>
__device__ __forceinline__ bf16x8 load_kv8(const KT* p) {
  if constexpr (sizeof(KT) == 2) return load_stream<bf16x8>(p);
  else return e4m3x8_to_bf16(load_stream<u32x2>(p));
}

// ---------------------------------------------------------------------------
// bf16, MFMA.  One wave per work group.  Lane l: c16 = l % 16, q4 = l / 16.
//
// Per iteration two pages (32 keys).  S tile u (u = 0, 1) has A-row i (lanes
// with c16 = i) holding the key of page i/8, in-page token
// 8*((i/4)%2) + 4u + i%4.  The MFMA result puts rows 4*q4 + rr in lane
// (q4, c16), so a lane ends up with the 8 consecutive tokens
// 8*(q4%2) + (4u + rr) of page q4/2 for its query row c16: exactly the k-group
// the PV MFMA expects from that lane, matching a single 16-byte V^T load.
// ---------------------------------------------------------------------------
// RW x PW waves per work group.  RW > 1 (prefill): the waves take different
// 16-row slices of the query block over the same keys; their repeated page
// reads hit in L1/L2, so HBM sees each page once.  PW > 1 (decode): the waves
// take interleaved page pairs of the item for the same 16 rows and are merged
// through LDS at the end, so one item (and one partial) covers PW times the
// pages a single wave streams.
//
// KT is the KV page element: uint16_t (bf16) or uint8_t (fp8 E4M3 codes,
// load_kv8).  The K scale is folded into scale_log2 by the host and the V
// scale multiplies the partial output.
template <int DH, int RW, int PW, typename KT>
__global__ __launch_bounds__(64 * RW * PW)
__attribute__((amdgpu_waves_per_eu(sizeof(KT) == 1 ? 2 : 3))) void attn_split_bf16(
    const AttnItem* __restrict__ items, const AttnQBlock* __restrict__ qblocks,
    const uint16_t* __restrict__ q, const KT* __restrict__ kpool,
    const KT* __restrict__ vpool, int64_t page_stride, const int32_t* __restrict__ bt,
    int32_t bt_stride, int32_t n_q_heads, int32_t n_kv_heads, float scale_log2, float v_scale,
    float* __restrict__ part_ml, float* __restrict__ part_acc) {
  constexpr int KC = DH / 32;  // k-steps of QK^T
  constexpr int DT = DH / 16;  // 16-wide dim tiles of PV
  constexpr int R = 16 * RW;  // query rows per item
  // Head dims of k-step c for lane group q4 in the Q K^T product (any
  // permutation works if Q and K share it).  bf16: chunk q4 of 32-dim block c,
  // so a load instruction covers 64 contiguous bytes of each key row.  fp8:
  // lane group q4 owns the contiguous span [q4 * DH/4, (q4 + 1) * DH/4), so a
  // 16-byte load covers two k-steps and again 64 bytes per key row.
  auto qk_dim = [](int c, int q4) {
    return sizeof(KT) == 1 ? q4 * (DH / 4) + c * 8 : c * 32 + q4 * 8;
  };
  static_assert(RW == 1 || PW == 1, "waves split either rows or pages");
  // fp8: the wave index lives in a scalar register, so page-table reads
  // indexed by it are scalar loads that never wait behind the prefetched page
  // loads (vector loads complete in order).  The bf16 loop has no prefetch
  // and measured 1.5% faster with the vector form.
  const int wave = sizeof(KT) == 1 ? __builtin_amdgcn_readfirstlane(threadIdx.x >> 6)
                                   : (int)(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int rw = wave % RW, pw = wave / RW;
  const int c16 = lane & 15, q4 = lane >> 4;
  // The KV heads of one item are adjacent in the grid, so the work groups in
  // flight together read whole contiguous page regions ([page][Hkv][...]).
  const int g = blockIdx.x, item_id = items[blockIdx.y].order;
  const AttnItem it = items[item_id];
  const AttnQBlock qb = qblocks[it.qblock];
  const int G = n_q_heads / n_kv_heads;

  // This lane's query row (the B column of S^T and O^T).
  const int row = rw * 16 + c16;
  if (PW == 1 && rw * 16 >= qb.n_q * G) return;  // no rows; no barriers when PW == 1
  const int jq = row / G;
  const int head = g * G + (row % G);
  const bool row_valid = jq < qb.n_q;

  bf16x8 qf[KC];
  if (row_valid) {
    const uint16_t* qrow = q + ((int64_t)(qb.q_row0 + jq) * n_q_heads + head) * DH;
#pragma unroll
    for (int c = 0; c < KC; ++c) qf[c] = *(const bf16x8*)(qrow + qk_dim(c, q4));
  } else {
#pragma unroll
    for (int c = 0; c < KC; ++c) qf[c] = bf16x8{};
  }

  const int key0 = it.page_begin * kPage;
  const int key_end = (it.page_begin + it.n_pages) * kPage;
  // Keys at or past kv_lim hold no data for any row of this block: their V is
  // zeroed so that stale or poisoned slots cannot reach the output.
  const int kv_lim = min(qb.pos0 + qb.n_q, key_end);
  // Causal limit of this lane's row (exclusive).
  const int row_lim = row_valid ? min(qb.pos0 + jq + 1, key_end) : key0;

  const int32_t* btrow = bt + (int64_t)qb.slot * bt_stride + it.page_begin;
  const int64_t head_off = (int64_t)g * (kPage * DH);

  // Lane-constant offsets.
  const int k_tok = 8 * ((c16 >> 2) & 1) + (c16 & 3);  // + 4u
  const int k_page_sel = c16 >> 3;                     // 0: first page, 1: second
  const int v_page_sel = q4 >> 1;
  const int v_tok0 = 8 * (q4 & 1);

  float m = -INFINITY;  // running max of scaled scores (log2 units), row-uniform
  float l = 0.f;        // lane-partial sum of probabilities
  f32x4 acc[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int n_iter = (it.n_pages + 1) >> 1;
  constexpr bool kFp8 = sizeof(KT) == 1;
  // This lane's K and V fragment bases of page pair `iter`.
  auto pair_bases = [&](int iter, const KT*& kb, const KT*& vb) {
    const int pi = 2 * iter;
    const int page0 = btrow[pi];
    const int page1 = (pi + 1 < it.n_pages) ? btrow[pi + 1] : page0;
    const int64_t base0 = (int64_t)page0 * page_stride + head_off;
    const int64_t base1 = (int64_t)page1 * page_stride + head_off;
    kb = kpool + (k_page_sel ? base1 : base0);
    vb = vpool + (v_page_sel ? base1 : base0) + v_tok0;
  };
  // fp8 pages: the raw codes of the wave's next page pair are loaded one
  // iteration ahead (the index is clamped to the last pair: the final
  // prefetch re-reads it).  A lane's K dims are one contiguous span, so each
  // 16-byte load holds two k-steps.
  u32x4 kr[2][KC / 2];
  u32x2 vr[DT];
  auto load_raw = [&](int iter, u32x4(&k)[2][KC / 2], u32x2(&v)[DT]) {
    const KT *kb, *vb;
    pair_bases(iter, kb, vb);
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int j = 0; j < KC / 2; ++j)
        k[u][j] = load_stream<u32x4>(kb + (k_tok + 4 * u) * DH + qk_dim(2 * j, q4));
#pragma unroll
    for (int t = 0; t < DT; ++t) v[t] = load_stream<u32x2>(vb + (t * 16 + c16) * kPage);
  };
  // One page pair: scores, online softmax and the PV product.
  auto step = [&](int iter, const bf16x8(&kf)[2][KC], u16x8(&vf)[DT]) {
    const int pi = 2 * iter;
    f32x4 s[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      s[u] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < KC; ++c)
        s[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[u][c], qf[c], s[u], 0, 0, 0);
    }

    // Keys of this lane: e = 4u + rr  ->  position kbase + e.
    const int kbase = key0 + (pi + v_page_sel) * kPage + v_tok0;
    float sv[8];
    float mloc = -INFINITY;
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int e = 4 * u + rr;
        const float x = (kbase + e < row_lim) ? s[u][rr] * scale_log2 : -INFINITY;
        sv[e] = x;
        mloc = max2(mloc, x);
      }
    mloc = max_over_key_groups(mloc);
    const float m_new = max2(m, mloc);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    // Rescale only when some row's running max moved (wave-uniform test).
    if (__any(m_new != m)) {
      const float alpha = __builtin_amdgcn_exp2f(m - m_use);
      l *= alpha;
#pragma unroll
      for (int t = 0; t < DT; ++t) acc[t] *= alpha;
    }
    m = m_new;

    // P in bf16 (hardware round-to-nearest-even); the normaliser sums exactly
    // the rounded weights the MFMA consumes.
    uint32_t pw4[4];
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      const f32x2 pv = {__builtin_amdgcn_exp2f(sv[e] - m_use),
                        __builtin_amdgcn_exp2f(sv[e + 1] - m_use)};
      const uint32_t bits = __builtin_bit_cast(uint32_t, __builtin_convertvector(pv, bf16x2));
      pw4[e / 2] = bits;
      l += __uint_as_float(bits << 16) + __uint_as_float(bits & 0xFFFF0000u);
    }
    u16x8 pbits = __builtin_bit_cast(u16x8, u32x4{pw4[0], pw4[1], pw4[2], pw4[3]});

    if (__builtin_expect(key0 + (pi + 2) * kPage > kv_lim, 0)) {  // wave-uniform: the block's last keys
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (kbase + e >= kv_lim)
#pragma unroll
          for (int t = 0; t < DT; ++t) vf[t][e] = 0;
    }

    const bf16x8 pf = __builtin_bit_cast(bf16x8, pbits);
#pragma unroll
    for (int t = 0; t < DT; ++t)
      acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vf[t]), pf,
                                                       acc[t], 0, 0, 0);
  };
  if constexpr (kFp8) {
    // Two raw buffers in turn: while one pair is decoded and used, the
    // wave's next pair streams into the other (no register copies, which
    // would wait for the loads).
    u32x4 kr2[2][KC / 2];
    u32x2 vr2[DT];
    auto decode = [&](const u32x4(&k)[2][KC / 2], const u32x2(&v)[DT], bf16x8(&kf)[2][KC],
                      u16x8(&vf)[DT]) {
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int j = 0; j < KC / 2; ++j) {
          kf[u][2 * j] = e4m3x8_to_bf16(u32x2{k[u][j].x, k[u][j].y});
          kf[u][2 * j + 1] = e4m3x8_to_bf16(u32x2{k[u][j].z, k[u][j].w});
        }
#pragma unroll
      for (int t = 0; t < DT; ++t) vf[t] = __builtin_bit_cast(u16x8, e4m3x8_to_bf16(v[t]));
    };
    if (pw < n_iter) load_raw(pw, kr, vr);
    for (int iter = pw; iter < n_iter; iter += 2 * PW) {
      bf16x8 kf[2][KC];
      u16x8 vf[DT];
      load_raw(min(iter + PW, n_iter - 1), kr2, vr2);
      __builtin_amdgcn_sched_barrier(0);  // keep the prefetch ahead of the decode's waits
      decode(kr, vr, kf, vf);
      step(iter, kf, vf);
      if (iter + PW >= n_iter) break;  // wave-uniform
      load_raw(min(iter + 2 * PW, n_iter - 1), kr, vr);
      __builtin_amdgcn_sched_barrier(0);
      decode(kr2, vr2, kf, vf);
      step(iter + PW, kf, vf);
    }
  } else {
    for (int iter = pw; iter < n_iter; iter += PW) {
      // K: 2 tiles x KC fragments of 16 B; V: DT fragments of 16 B.
      const int pi = 2 * iter;
      const int page0 = btrow[pi];
      const int page1 = (pi + 1 < it.n_pages) ? btrow[pi + 1] : page0;
      const int64_t base0 = (int64_t)page0 * page_stride + head_off;
      const int64_t base1 = (int64_t)page1 * page_stride + head_off;
      const KT* kb = kpool + (k_page_sel ? base1 : base0);
      bf16x8 kf[2][KC];
      u16x8 vf[DT];
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int c = 0; c < KC; ++c)
          kf[u][c] = load_kv8(kb + (k_tok + 4 * u) * DH + qk_dim(c, q4));
      const KT* vb = vpool + (v_page_sel ? base1 : base0) + v_tok0;
#pragma unroll
      for (int t = 0; t < DT; ++t)
        vf[t] = __builtin_bit_cast(u16x8, load_kv8(vb + (t * 16 + c16) * kPage));
      step(iter, kf, vf);
    }
  }

  l = sum_over_key_groups(l);
  if constexpr (PW > 1) {
    // Page-split waves hand (m, l, acc) to wave 0, which merges them in wave
    // order with the online-softmax rule.
    __shared__ float sm[PW - 1][64][4 * DT + 2];
    if (pw > 0) {
      float* d = sm[pw - 1][lane];
      d[0] = m;
      d[1] = l;
#pragma unroll
      for (int t = 0; t < DT; ++t)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) d[2 + 4 * t + rr] = acc[t][rr];
    }
    __syncthreads();
    if (pw > 0) return;
#pragma unroll
    for (int w = 0; w < PW - 1; ++w) {
      const float* d = sm[w][lane];
      const float mn = fmaxf(m, d[0]);
      const float mu = (mn == -INFINITY) ? 0.f : mn;
      const float so = exp2f(m - mu), sw = exp2f(d[0] - mu);
      l = l * so + d[1] * sw;
#pragma unroll
      for (int t = 0; t < DT; ++t)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) acc[t][rr] = acc[t][rr] * so + d[2 + 4 * t + rr] * sw;
      m = mn;
    }
  }
  if (row_valid) {
    const int64_t prow = ((int64_t)item_id * n_kv_heads + g) * R + row;
    if (q4 == 0) {
      part_ml[prow * 2] = m;
      part_ml[prow * 2 + 1] = l;
    }
    float* pa = part_acc + prow * DH;
#pragma unroll
    for (int t = 0; t < DT; ++t) {
      if constexpr (sizeof(KT) == 1) acc[t] *= v_scale;
      *(f32x4*)(pa + t * 16 + 4 * q4) = acc[t];
    }
  }
}

// ---------------------------------------------------------------------------
// fp32, VALU.  One wave per work group; lane = head dimension (DH/64 per
// lane).  Rows and keys are walked one at a time: this path serves the small
// fp32 decoder, where launches, not bytes, set the step time.
// ---------------------------------------------------------------------------
template <int DH>
__global__ __launch_bounds__(64) void attn_split_f32(
    const AttnItem* __restrict__ items, const AttnQBlock* __restrict__ qblocks,
    const float* __restrict__ q, const float* __restrict__ kpool, const float* __restrict__ vpool,
    int64_t page_stride, const int32_t* __restrict__ bt, int32_t bt_stride, int32_t n_q_heads,
    int32_t n_kv_heads, int32_t R, float scale_log2, float* __restrict__ part_ml,
    float* __restrict__ part_acc) {
  constexpr int E = DH / 64;
  const int lane = threadIdx.x;
  const int g = blockIdx.x, item_id = items[blockIdx.y].order;
  const AttnItem it = items[item_id];
  const AttnQBlock qb = qblocks[it.qblock];
  const int G = n_q_heads / n_kv_heads;
  const int key0 = it.page_begin * kPage;
  const int key_end = (it.page_begin + it.n_pages) * kPage;
  const int32_t* btrow = bt + (int64_t)qb.slot * bt_stride;
  const int64_t head_off = (int64_t)g * (kPage * DH);

  for (int r = 0; r < qb.n_q * G; ++r) {
    const int jq = r / G, head = g * G + r % G;
    const float* qrow = q + ((int64_t)(qb.q_row0 + jq) * n_q_heads + head) * DH;
    float qv[E], acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      qv[e] = qrow[lane + 64 * e] * scale_log2;
      acc[e] = 0.f;
    }
    float m = -INFINITY, l = 0.f;
    const int lim = min(qb.pos0 + jq + 1, key_end);
    for (int kp = key0; kp < lim; ++kp) {
      const int64_t base = (int64_t)btrow[kp / kPage] * page_stride + head_off;
      const int t = kp % kPage;
      float part = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) part += qv[e] * kpool[base + t * DH + lane + 64 * e];
      const float s = wave_sum(part);
      const float m_new = fmaxf(m, s);
      const float alpha = exp2f(m - m_new);
      const float p = exp2f(s - m_new);
      l = l * alpha + p;
#pragma unroll
      for (int e = 0; e < E; ++e)
        acc[e] = acc[e] * alpha + p * vpool[base + (lane + 64 * e) * kPage + t];
      m = m_new;
    }
    const int64_t prow = ((int64_t)item_id * n_kv_heads + g) * R + r;
    if (lane == 0) {
      part_ml[prow * 2] = m;
      part_ml[prow * 2 + 1] = l;
    }
#pragma unroll
    for (int e = 0; e < E; ++e) part_acc[prow * DH + lane + 64 * e] = acc[e];
  }
}

// ---------------------------------------------------------------------------
// Merge the partials of each (query row, head) with the online-softmax rule:
// m = max(m, m_i); l = l e^(m_old-m) + l_i e^(m_i-m); o likewise; output o/l.
// One work group of 4 waves per (query block, KV head).  Wave w merges items
// w, w+4, w+8, ... (in order), then wave 0 merges the four results in wave
// order, so the result is deterministic.  A lane owns DH/16 consecutive dims
// of one of four rows at a time.
// ---------------------------------------------------------------------------
template <int DPL>
__device__ __forceinline__ void merge_into(float& m, float& l, float* o, float mi, float li,
                                           const float* oi) {
  const float mn = fmaxf(m, mi);
  const float mu = (mn == -INFINITY) ? 0.f : mn;  // both empty: keep zeros
  const float so = exp2f(m - mu), si = exp2f(mi - mu);
  l = l * so + li * si;
#pragma unroll
  for (int e = 0; e < DPL; ++e) o[e] = o[e] * so + oi[e] * si;
  m = mn;
}

template <int DH, typename OutT, int NW>
__global__ __launch_bounds__(64 * NW) void attn_combine(const AttnQBlock* __restrict__ qblocks,
                                                       const float* __restrict__ part_ml,
                                                       const float* __restrict__ part_acc,
                                                       int32_t n_q_heads, int32_t n_kv_heads,
                                                       int32_t R, OutT* __restrict__ out) {
  constexpr int DPL = DH / 16;
  __shared__ float sh[NW][64][DPL + 2];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int rsub = lane >> 4, d0 = (lane & 15) * DPL;
  const AttnQBlock qb = qblocks[blockIdx.x];
  const int g = blockIdx.y;
  const int G = n_q_heads / n_kv_heads;
  const int rows = qb.n_q * G;
  for (int r0 = 0; r0 < rows; r0 += 4) {
    const int r = min(r0 + rsub, rows - 1);
    float m = -INFINITY, l = 0.f, o[DPL];
#pragma unroll
    for (int e = 0; e < DPL; ++e) o[e] = 0.f;
    // Items i0 + 4u (u = 0..3) of this wave's stride, loads issued first.
    for (int i0 = qb.item_begin + wave; i0 < qb.item_end; i0 += 4 * NW) {
      float2 ml[4];
      float a[4][DPL];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = min(i0 + NW * u, qb.item_end - 1);
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
        if (i0 + NW * u >= qb.item_end) break;
        merge_into<DPL>(m, l, o, ml[u].x, ml[u].y, a[u]);
      }
    }
    sh[wave][lane][0] = m;
    sh[wave][lane][1] = l;
#pragma unroll
    for (int e = 0; e < DPL; ++e) sh[wave][lane][2 + e] = o[e];
    __syncthreads();
    if (wave == 0 && r0 + rsub < rows) {
      for (int w = 1; w < NW; ++w)
        merge_into<DPL>(m, l, o, sh[w][lane][0], sh[w][lane][1], &sh[w][lane][2]);
      const float inv = 1.f / l;
      const int jq = r / G, head = g * G + r % G;
      OutT* orow = out + ((int64_t)(qb.q_row0 + jq) * n_q_heads + head) * DH + d0;
#pragma unroll
      for (int e = 0; e < DPL; ++e) orow[e] = Store<OutT>::from(o[e] * inv);
    }
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_attention_split(int dtype, int kv_fp8, float k_scale, float v_scale,
                                  int head_dim, int rows_per_item, int n_items,
                                  int n_q_heads, int n_kv_heads, const AttnItem* items,
                                  const AttnQBlock* qblocks, const void* q, const void* k_pages,
                                  const void* v_pages, int64_t page_stride_elems,
                                  const int32_t* block_table, int32_t bt_stride, float* part_ml,
                                  float* part_acc, hipStream_t stream, hipEvent_t ev_start,
                                  hipEvent_t ev_stop) {
  if (n_items == 0) return hipSuccess;
  const dim3 grid(n_kv_heads, n_items);
  const float scale_log2 = kLog2e / sqrtf((float)head_dim) * (kv_fp8 ? k_scale : 1.f);
  if (dtype == 1) {
    const uint16_t* qq = (const uint16_t*)q;
#define PDEC_ATTN_BF16(DH_, RW_, PW_, KT_)                                                   \
  return launch_timed(attn_split_bf16<DH_, RW_, PW_, KT_>, grid, dim3(64 * RW_ * PW_), stream,  \
                      ev_start, ev_stop, items, qblocks, qq, (const KT_*)k_pages,             \
                      (const KT_*)v_pages, page_stride_elems, block_table, bt_stride,         \
                      n_q_heads, n_kv_heads, scale_log2, v_scale, part_ml, part_acc)
#define PDEC_ATTN_KT(KT_)                                                                    \
  if (head_dim == 128) {                                                                     \
    PDEC_ATTN_BF16(128, 1, 4, KT_);                                                          \
  } else {                                                                                   \
    if (rows_per_item == 64) PDEC_ATTN_BF16(64, 4, 1, KT_); else PDEC_ATTN_BF16(64, 1, 4, KT_); \
  }
    // Prefill with 128-dim heads (128- or 256-row items, bf16 or E4M3 pages):
    // the LDS-staged prefill kernel.  Prefill with 64-dim heads (64-row
    // items): the split kernel with waves splitting rows.  Decode (16-row
    // items): the split kernel with waves splitting pages.
    if (head_dim == 128 && (rows_per_item == 128 || rows_per_item == 256))
      return launch_attention_prefill_bf16(n_items, rows_per_item, n_q_heads, n_kv_heads, kv_fp8,
                                           items, qblocks, q, k_pages, v_pages, page_stride_elems,
                                           block_table, bt_stride, scale_log2, v_scale, part_ml,
                                           part_acc, stream, ev_start, ev_stop);
    const bool rows_ok = rows_per_item == 16 || (head_dim == 64 && rows_per_item == 64);
    if (!rows_ok || (head_dim != 128 && head_dim != 64)) return hipErrorInvalidValue;
    if (kv_fp8) {
      PDEC_ATTN_KT(uint8_t)
    } else {
      PDEC_ATTN_KT(uint16_t)
    }
#undef PDEC_ATTN_KT
#undef PDEC_ATTN_BF16
  } else {
    if (head_dim == 128)
      return launch_timed(attn_split_f32<128>, grid, dim3(64), stream, ev_start, ev_stop, items,
                          qblocks, (const float*)q, (const float*)k_pages,
                          (const float*)v_pages, page_stride_elems, block_table, bt_stride,
                          n_q_heads, n_kv_heads, rows_per_item, scale_log2, part_ml, part_acc);
    else
      return launch_timed(attn_split_f32<64>, grid, dim3(64), stream, ev_start, ev_stop, items,
                          qblocks, (const float*)q, (const float*)k_pages,
                          (const float*)v_pages, page_stride_elems, block_table, bt_stride,
                          n_q_heads, n_kv_heads, rows_per_item, scale_log2, part_ml, part_acc);
  }
  return hipGetLastError();
}

hipError_t launch_attention_combine(int head_dim, int rows_per_item, int n_qblocks,
                                    int max_items, int n_q_heads, int n_kv_heads,
                                    const AttnQBlock* qblocks, const float* part_ml,
                                    const float* part_acc, void* out, int out_bf16,
                                    hipStream_t stream) {
  if (n_qblocks == 0) return hipSuccess;
  const dim3 grid(n_qblocks, n_kv_heads);
  // Each wave merges four items per round: enough waves that the query block
  // with the most items (the longest context) needs a single round, up to 16.
  const int nw = max_items <= 16 ? 4 : max_items <= 32 ? 8 : 16;
#define PDEC_COMBINE_NW(DH_, T_, NW_)                                                        \
  attn_combine<DH_, T_, NW_><<<grid, dim3(64 * NW_), 0, stream>>>(                           \
      qblocks, part_ml, part_acc, n_q_heads, n_kv_heads, rows_per_item, (T_*)out)
#define PDEC_COMBINE(DH_, T_)                                                                \
  do {                                                                                       \
    if (nw == 4) PDEC_COMBINE_NW(DH_, T_, 4);                                                \
    else if (nw == 8) PDEC_COMBINE_NW(DH_, T_, 8);                                           \
    else PDEC_COMBINE_NW(DH_, T_, 16);                                                       \
  } while (0)
  if (head_dim == 128) {
    if (out_bf16) PDEC_COMBINE(128, uint16_t); else PDEC_COMBINE(128, float);
  } else {
    if (out_bf16) PDEC_COMBINE(64, uint16_t); else PDEC_COMBINE(64, float);
  }
#undef PDEC_COMBINE
#undef PDEC_COMBINE_NW
  return hipGetLastError();
}

}  // namespace pdec

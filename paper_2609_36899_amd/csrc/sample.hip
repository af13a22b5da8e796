// Temperature / nucleus (top-p) sampling with caller-supplied uniforms.
//
// RL rollouts sample their actions rather than taking the argmax (paper:
// Background, "RL Post-Training Workflow"); the paper does not state the
// sampler, so this is the common temperature + top-p rule, defined so that
// every decision is exact integer arithmetic after one exponential:
//
//   e_v = exp((z_v - max z) / T)            (fp64)
//   q_v = rint(e_v * 2^40)                  (integer mass, 0 .. 2^40)
//   S   = sum_v q_v
//   nucleus: the shortest prefix of the tokens ordered by (q desc, index asc)
//            whose mass reaches ceil(p24 * S / 2^24), p24 = rint(top_p * 2^24)
//   Z   = nucleus mass, target = floor(u24 * Z / 2^24), u24 = floor(u * 2^24)
//   token = the first nucleus token, in index order, whose running nucleus
//           mass exceeds target.
//
// One work group of 1024 threads per row.  The nucleus threshold key is
// found by a radix select over the 41-bit keys (digits of 11, 11, 11 and 8
// bits) with 64-bit integer mass histograms in LDS (integer atomics: the
// result does not depend on their order); the final index-order walk uses
// wave-level scans over each wave's contiguous range.  Only the first round
// needs every token's mass.  Later passes need only the tokens whose mass can
// fall in the current key range.  A conservative test on x = (z - max z)/T
// (the mass is monotone in x) selects them, and only they recompute the
// exponential, so every decision stays exact without a stored row of keys.
#include "hip_common.h"
#include "kernels.h"

#include <climits>
#include <mutex>

namespace pdec {

namespace {

constexpr int kThreads = 1024, kWaves = kThreads / 64;
constexpr int kUnroll = 8;  // loads in flight per lane: index slabs of 64
constexpr int kUnroll4 = 4;  // 16-byte loads in flight per lane (vectorised passes)
constexpr int kRounds = 4, kMaxBins = 2048;
// Radix digits of the 41-bit keys, most significant first: bits 40..30,
// 29..19, 18..8, 7..0.
__device__ constexpr int kShift[kRounds] = {30, 19, 8, 0};
__device__ constexpr int kWidth[kRounds] = {11, 11, 11, 8};
typedef unsigned __int128 u128;

// Integer mass of one logit.  Below x = -28.5 the exponential is under
// 2^-41 and the mass rounds to exactly 0, so the exponential is skipped.
__device__ __forceinline__ uint64_t mass_of(float z, double m, double inv_t) {
  const double x = ((double)z - m) * inv_t;
  if (x < -28.5) return 0;
  return (uint64_t)rint(exp(x) * 0x1p40);
}

__device__ __forceinline__ uint64_t wave_scan_incl(uint64_t v, int lane) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint64_t o = __shfl_up(v, off, 64);
    if (lane >= off) v += o;
  }
  return v;
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Lowest x whose mass can reach key k (k >= 1): rint(e * 2^40) >= k needs
// e * 2^40 >= k - 1/2; a margin far above the exponential's error keeps the
// test conservative.
__device__ __forceinline__ double x_floor(uint64_t k) {
  return k == 0 ? -INFINITY : log(((double)k - 0.5) * 0x1p-40) - 1e-9;
}

__global__ __launch_bounds__(kThreads) void sample_top_p_kernel(
    int V, const float* __restrict__ logits, double inv_t, uint32_t p24,
    const float* __restrict__ uniforms, int32_t* __restrict__ tokens) {
  __shared__ uint64_t hist[kMaxBins];
  __shared__ uint64_t wave_a[kWaves], wave_b[kWaves];
  __shared__ float red_f[kWaves];
  __shared__ uint64_t sel[3];  // digit, mass above it, T_p
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const float* z = logits + (int64_t)blockIdx.x * V;
  // Wave w owns the index range [w0, w1), read coalesced in blocks of
  // kUnroll slabs of 64 (all loads of a block issued before any use); index
  // order is (wave, block, slab, lane).  Out-of-range slots read as -inf.
  const int span = ((V + kWaves * 64 - 1) / (kWaves * 64)) * 64;
  const int w0 = min(V, wave * span), w1 = min(V, w0 + span);
  auto load_block = [&](int base, float (&zv)[kUnroll]) {
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int i = base + u * 64 + lane;
      zv[u] = i < w1 ? z[i] : -INFINITY;
    }
  };

  // The passes whose results are sums (max, histograms, tie counts) may see
  // a wave's tokens in any order: with V % 4 == 0 (rows 16-byte aligned) they
  // read 16 bytes per lane, four times the bytes in flight of the scalar
  // blocks, which is what bounds one work group's pass over a long row.  Only
  // the final walk needs index order and keeps the scalar blocks.
  const bool vec4 = (V & 3) == 0;
  auto for_each = [&](auto&& f) {
    if (vec4) {
      for (int base = w0; base < w1; base += 256 * kUnroll4) {
        float4 zv[kUnroll4];
#pragma unroll
        for (int u = 0; u < kUnroll4; ++u) {
          const int i = base + (u * 64 + lane) * 4;  // i < w1 implies i + 3 < w1
          zv[u] = i < w1 ? *(const float4*)(z + i)
                         : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
        }
#pragma unroll
        for (int u = 0; u < kUnroll4; ++u) {
          f(zv[u].x);
          f(zv[u].y);
          f(zv[u].z);
          f(zv[u].w);
        }
      }
    } else {
      for (int base = w0; base < w1; base += 64 * kUnroll) {
        float zv[kUnroll];
        load_block(base, zv);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) f(zv[u]);
      }
    }
  };

  // Row max.
  float mx = -INFINITY;
  for_each([&](float v) { mx = fmaxf(mx, v); });
  mx = wave_max(mx);
  if (lane == 0) red_f[wave] = mx;
  __syncthreads();
  if (t == 0) {
    float bmax = red_f[0];
    for (int w = 1; w < kWaves; ++w) bmax = fmaxf(bmax, red_f[w]);
    red_f[0] = bmax;
  }
  __syncthreads();
  const double m = (double)red_f[0];

  // Radix select of the threshold key kappa: the largest key with
  // mass{q >= kappa} >= T_p, where T_p = ceil(p24 * S / 2^24).  Each thread
  // adds runs of equal digits in a register and flushes a run to the LDS
  // histogram only when the digit changes: most tokens share one bin, and
  // per-element atomics on one address would serialise.
  uint64_t prefix = 0, above = 0, t_p = 0;
  for (int r = 0; r < kRounds; ++r) {
    const int shift = kShift[r], bins = 1 << kWidth[r];
    for (int bin = t; bin < bins; bin += kThreads) hist[bin] = 0;
    __syncthreads();
    int run_bin = -1;
    uint64_t run_sum = 0;
    // keys of this round's range: [prefix << top, (prefix + 1) << top)
    const int top = shift + kWidth[r];
    const double xlo = x_floor(prefix << top), xhi = x_floor((prefix + 1) << top);
    for_each([&](float zz) {
      const double x = ((double)zz - m) * inv_t;
      if (x < xlo || (r > 0 && x > xhi + 2e-9)) return;
      const uint64_t q = mass_of(zz, m, inv_t);
      if (q != 0 && (q >> top) == prefix) {
        const int d = (int)((q >> shift) & (uint64_t)(bins - 1));
        if (d != run_bin) {
          if (run_bin >= 0) atomicAdd((unsigned long long*)&hist[run_bin], run_sum);
          run_bin = d;
          run_sum = 0;
        }
        run_sum += q;
      }
    });
    if (run_bin >= 0) atomicAdd((unsigned long long*)&hist[run_bin], run_sum);
    __syncthreads();
    if (r == 0) {  // S = total mass, T_p from it
      uint64_t part = 0;
      for (int bin = t; bin < bins; bin += kThreads) part += hist[bin];
      part = wave_sum_u64(part);
      if (lane == 0) wave_a[wave] = part;
      __syncthreads();
      if (t == 0) {
        uint64_t total = 0;
        for (int w = 0; w < kWaves; ++w) total += wave_a[w];
        sel[2] = (uint64_t)(((u128)p24 * total + ((u128)1 << 24) - 1) >> 24);
      }
      __syncthreads();
    }
    t_p = sel[2];
    // Select the digit: walking bins from the top, the first whose
    // cumulative mass (from `above`) reaches T_p.  Thread t holds the bins
    // ranked 2t and 2t+1 from the top; a block scan gives the cumulative sums.
    const int per = (bins + kThreads - 1) / kThreads;  // 2 or 1
    uint64_t mine = 0;
    for (int j = 0; j < per; ++j) {
      const int rank = t * per + j;
      if (rank < bins) mine += hist[bins - 1 - rank];
    }
    const uint64_t incl_w = wave_scan_incl(mine, lane);
    if (lane == 63) wave_b[wave] = incl_w;
    __syncthreads();
    uint64_t before = above + incl_w - mine;
    for (int w = 0; w < wave; ++w) before += wave_b[w];
    for (int j = 0; j < per; ++j) {
      const int rank = t * per + j;
      if (rank >= bins) break;
      const uint64_t h = hist[bins - 1 - rank];
      // The digit is the first bin reaching T_p; the lowest bin (rank
      // bins-1) always does, by the invariant mass(prefix range) >= T_p.
      if (before < t_p && (before + h >= t_p || rank == bins - 1)) {
        sel[0] = (uint64_t)(bins - 1 - rank);
        sel[1] = before;
      }
      before += h;
    }
    __syncthreads();
    prefix = (prefix << kWidth[r]) | sel[0];
    above = sel[1];
    __syncthreads();
  }
  const uint64_t kappa = prefix;  // >= 1: zero-mass keys never enter the histograms
  // Tokens with q == kappa join the nucleus in index order until the mass
  // reaches T_p: the first n_tie of them.
  const uint64_t n_tie = (t_p - above + kappa - 1) / kappa;

  // One pass: ties and strict-member mass per wave (only x >= x_floor(kappa)
  // can reach kappa).
  const double xk = x_floor(kappa);
  uint64_t ties = 0, strict = 0;
  for_each([&](float zz) {
    if (((double)zz - m) * inv_t < xk) return;
    const uint64_t q = mass_of(zz, m, inv_t);
    ties += q == kappa;
    strict += q > kappa ? q : 0;
  });
  ties = wave_sum_u64(ties);
  strict = wave_sum_u64(strict);
  if (lane == 0) {
    wave_a[wave] = ties;
    wave_b[wave] = strict;
  }
  __syncthreads();
  // Wave w holds ties ranked [tie_base, tie_base + ties); its member ties
  // are those ranked below n_tie.
  uint64_t tie_base = 0, mass_base = 0, Z = 0, own = 0, tb = 0;
  for (int w = 0; w < kWaves; ++w) {
    const uint64_t nt = wave_a[w];
    const uint64_t member_ties = n_tie > tb ? min(nt, n_tie - tb) : 0;
    const uint64_t wm = wave_b[w] + member_ties * kappa;
    if (w < wave) mass_base += wm;
    if (w == wave) {
      own = wm;
      tie_base = tb;
    }
    Z += wm;
    tb += nt;
  }
  float u = uniforms[blockIdx.x];
  u = fminf(fmaxf(u, 0.f), 0x1.fffffep-1f);
  const uint64_t u24 = (uint64_t)(u * 0x1p24f);
  const uint64_t target = (uint64_t)(((u128)u24 * Z) >> 24);
  // The wave whose nucleus mass range [mass_base, mass_base + own) holds
  // target walks its range in index order.
  if (own > 0 && mass_base <= target && target < mass_base + own) {
    uint64_t run = mass_base, rank = tie_base;
    bool found = false;
    for (int base = w0; base < w1 && !found; base += 64 * kUnroll) {
      float zv[kUnroll];
      load_block(base, zv);
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int i = base + u * 64 + lane;
        uint64_t q = 0;
        if (((double)zv[u] - m) * inv_t >= xk) q = mass_of(zv[u], m, inv_t);
        const bool tie = q == kappa;  // out-of-range slots have q = 0 < kappa
        const uint64_t tie_mask = __ballot(tie);
        const uint64_t my_rank = rank + __popcll(tie_mask & ((1ull << lane) - 1));
        const uint64_t mass = (q > kappa || (tie && my_rank < n_tie)) ? q : 0;
        const uint64_t incl = run + wave_scan_incl(mass, lane);
        const uint64_t hit = __ballot(mass > 0 && incl > target);
        if (hit) {
          if (lane == __ffsll((unsigned long long)hit) - 1) tokens[blockIdx.x] = i;
          found = true;
          break;
        }
        run = __shfl(incl, 63, 64);
        rank += __popcll(tie_mask);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Split form for batches below the CU count.  One work group per row leaves
// most CUs idle and each pass over a 513 KB row runs at one CU's bandwidth;
// here every pass is spread over C work groups per row, each owning a
// contiguous chunk of the row, and the per-row decisions run in small
// one-group kernels between them:
//   chunk_max -> (chunk_hist(r) -> select(r)) x 4 -> chunk_ties -> walk.
// All cross-chunk results are integer sums (or a max), so the token is the
// one-group form's.  Workspace per row: the row state, C chunk maxima, C
// partial histograms of 2048 bins and C (ties, strict mass) pairs.
// ---------------------------------------------------------------------------
constexpr int kST = 256, kSW = kST / 64;  // threads / waves of the split kernels

// Per row, after the rounds so far: the key prefix, the mass of keys above
// its range, and T_p.
struct RowState {
  uint64_t prefix, above, t_p;
};

struct SplitWs {
  RowState* st;       // [B]
  float* cmax;        // [B][C]
  uint64_t* hist;     // [B][C][kMaxBins]
  uint64_t* ties;     // [B][C][2]: tie count, strict-member mass
};

// Chunk c of a row: [i0, i1), the chunk length a multiple of 4 so that with
// V % 4 == 0 every chunk start is 16-byte aligned.
__device__ __forceinline__ void chunk_range(int V, int C, int c, int& i0, int& i1) {
  const int span = (((V + C - 1) / C) + 3) & ~3;
  i0 = min(V, c * span);
  i1 = min(V, i0 + span);
}

// Calls f(z) for every token of [i0, i1) in some order, 16-byte loads when
// the row length allows.
template <typename F>
__device__ __forceinline__ void chunk_for_each(const float* z, int V, int i0, int i1, F&& f) {
  const int t = threadIdx.x;
  if ((V & 3) == 0) {
    for (int base = i0 + 4 * t; base < i1; base += 4 * kST * kUnroll4) {
      float4 zv[kUnroll4];
#pragma unroll
      for (int u = 0; u < kUnroll4; ++u) {
        const int i = base + 4 * kST * u;  // i < i1 implies i + 3 < i1
        zv[u] = i < i1 ? *(const float4*)(z + i)
                       : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
      }
#pragma unroll
      for (int u = 0; u < kUnroll4; ++u) {
        f(zv[u].x);
        f(zv[u].y);
        f(zv[u].z);
        f(zv[u].w);
      }
    }
  } else {
    for (int i = i0 + t; i < i1; i += kST) f(z[i]);
  }
}

__device__ __forceinline__ uint64_t block_sum_u64(uint64_t v, uint64_t* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  v = wave_sum_u64(v);
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  uint64_t total = 0;
  for (int w = 0; w < kSW; ++w) total += red[w];
  return total;
}

__global__ __launch_bounds__(kST) void split_chunk_max(int V, int C, const float* __restrict__ logits,
                                                       SplitWs ws) {
  __shared__ float red[kSW];
  const int c = blockIdx.x, b = blockIdx.y, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int i0, i1;
  chunk_range(V, C, c, i0, i1);
  float mx = -INFINITY;
  chunk_for_each(logits + (int64_t)b * V, V, i0, i1, [&](float v) { mx = fmaxf(mx, v); });
  mx = wave_max(mx);
  if (lane == 0) red[wave] = mx;
  __syncthreads();
  if (threadIdx.x == 0) {
    float bm = red[0];
    for (int w = 1; w < kSW; ++w) bm = fmaxf(bm, red[w]);
    ws.cmax[(int64_t)b * C + c] = bm;
  }
}

// Row max from the chunk maxima (the same float max as one pass).
__device__ __forceinline__ double row_max(const SplitWs& ws, int b, int C) {
  float m = -INFINITY;
  for (int c = 0; c < C; ++c) m = fmaxf(m, ws.cmax[(int64_t)b * C + c]);
  return (double)m;
}

// Round r's histogram of one chunk: the tokens whose key lies in the
// current prefix range, by their round-r digit, as in the one-group form.
__global__ __launch_bounds__(kST) void split_chunk_hist(int V, int C, int r,
                                                        const float* __restrict__ logits,
                                                        double inv_t, SplitWs ws) {
  __shared__ uint64_t hist[kMaxBins];
  const int c = blockIdx.x, b = blockIdx.y;
  const int shift = kShift[r], bins = 1 << kWidth[r], top = shift + kWidth[r];
  const double m = row_max(ws, b, C);
  const uint64_t prefix = r ? ws.st[b].prefix : 0;
  for (int bin = threadIdx.x; bin < bins; bin += kST) hist[bin] = 0;
  __syncthreads();
  const double xlo = x_floor(prefix << top), xhi = x_floor((prefix + 1) << top);
  int i0, i1;
  chunk_range(V, C, c, i0, i1);
  int run_bin = -1;
  uint64_t run_sum = 0;
  chunk_for_each(logits + (int64_t)b * V, V, i0, i1, [&](float zz) {
    const double x = ((double)zz - m) * inv_t;
    if (x < xlo || (r > 0 && x > xhi + 2e-9)) return;
    const uint64_t q = mass_of(zz, m, inv_t);
    if (q != 0 && (q >> top) == prefix) {
      const int d = (int)((q >> shift) & (uint64_t)(bins - 1));
      if (d != run_bin) {
        if (run_bin >= 0) atomicAdd((unsigned long long*)&hist[run_bin], run_sum);
        run_bin = d;
        run_sum = 0;
      }
      run_sum += q;
    }
  });
  if (run_bin >= 0) atomicAdd((unsigned long long*)&hist[run_bin], run_sum);
  __syncthreads();
  uint64_t* dst = ws.hist + ((int64_t)b * C + c) * kMaxBins;
  for (int bin = threadIdx.x; bin < bins; bin += kST) dst[bin] = hist[bin];
}

// Round r's decision for one row: sum the chunk histograms, then pick the
// digit exactly as the one-group form (walking bins from the top, the first
// whose cumulative mass from `above` reaches T_p).
__global__ __launch_bounds__(kThreads) void split_select(int C, int r, uint32_t p24,
                                                         SplitWs ws) {
  __shared__ uint64_t hist[kMaxBins];
  __shared__ uint64_t wave_a[kWaves], wave_b[kWaves];
  __shared__ uint64_t sel[2];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6, b = blockIdx.x;
  const int bins = 1 << kWidth[r];
  const uint64_t* h0 = ws.hist + (int64_t)b * C * kMaxBins;
  for (int bin = t; bin < bins; bin += kThreads) {
    uint64_t v = 0;
    for (int c = 0; c < C; ++c) v += h0[(int64_t)c * kMaxBins + bin];
    hist[bin] = v;
  }
  __syncthreads();
  RowState st = ws.st[b];
  if (r == 0) {
    st.prefix = 0;
    st.above = 0;
    uint64_t part = 0;
    for (int bin = t; bin < bins; bin += kThreads) part += hist[bin];
    part = wave_sum_u64(part);
    if (lane == 0) wave_a[wave] = part;
    __syncthreads();
    uint64_t total = 0;
    for (int w = 0; w < kWaves; ++w) total += wave_a[w];
    st.t_p = (uint64_t)(((u128)p24 * total + ((u128)1 << 24) - 1) >> 24);
  }
  const int per = (bins + kThreads - 1) / kThreads;
  uint64_t mine = 0;
  for (int j = 0; j < per; ++j) {
    const int rank = t * per + j;
    if (rank < bins) mine += hist[bins - 1 - rank];
  }
  const uint64_t incl_w = wave_scan_incl(mine, lane);
  if (lane == 63) wave_b[wave] = incl_w;
  __syncthreads();
  uint64_t before = st.above + incl_w - mine;
  for (int w = 0; w < wave; ++w) before += wave_b[w];
  for (int j = 0; j < per; ++j) {
    const int rank = t * per + j;
    if (rank >= bins) break;
    const uint64_t h = hist[bins - 1 - rank];
    if (before < st.t_p && (before + h >= st.t_p || rank == bins - 1)) {
      sel[0] = (uint64_t)(bins - 1 - rank);
      sel[1] = before;
    }
    before += h;
  }
  __syncthreads();
  if (t == 0) {
    st.prefix = (st.prefix << kWidth[r]) | sel[0];
    st.above = sel[1];
    ws.st[b] = st;
  }
}

// Per chunk: the number of keys equal to kappa and the mass of keys above it.
__global__ __launch_bounds__(kST) void split_chunk_ties(int V, int C,
                                                        const float* __restrict__ logits,
                                                        double inv_t, SplitWs ws) {
  __shared__ uint64_t red[kSW];
  const int c = blockIdx.x, b = blockIdx.y;
  const double m = row_max(ws, b, C);
  const uint64_t kappa = ws.st[b].prefix;
  const double xk = x_floor(kappa);
  int i0, i1;
  chunk_range(V, C, c, i0, i1);
  uint64_t ties = 0, strict = 0;
  chunk_for_each(logits + (int64_t)b * V, V, i0, i1, [&](float zz) {
    if (((double)zz - m) * inv_t < xk) return;
    const uint64_t q = mass_of(zz, m, inv_t);
    ties += q == kappa;
    strict += q > kappa ? q : 0;
  });
  ties = block_sum_u64(ties, red);
  strict = block_sum_u64(strict, red);
  if (threadIdx.x == 0) {
    ws.ties[((int64_t)b * C + c) * 2] = ties;
    ws.ties[((int64_t)b * C + c) * 2 + 1] = strict;
  }
}

// The row's token: the chunk whose nucleus mass range holds the target is
// walked in index order, 256 tokens at a time, with a work-group scan.
__global__ __launch_bounds__(kST) void split_walk(int V, int C, const float* __restrict__ logits,
                                                  double inv_t,
                                                  const float* __restrict__ uniforms,
                                                  int32_t* __restrict__ tokens, SplitWs ws) {
  __shared__ uint64_t wsum[kSW], wtie[kSW];
  __shared__ int found_at;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6, b = blockIdx.x;
  const RowState st = ws.st[b];
  const uint64_t kappa = st.prefix;
  const uint64_t n_tie = (st.t_p - st.above + kappa - 1) / kappa;
  const uint64_t* tc = ws.ties + (int64_t)b * C * 2;
  // Nucleus mass of every chunk (its strict members plus its member ties,
  // ties ranked in index order across chunks).
  uint64_t Z = 0, tb = 0;
  for (int c = 0; c < C; ++c) {
    const uint64_t nt = tc[2 * c];
    const uint64_t mt = n_tie > tb ? min(nt, n_tie - tb) : 0;
    Z += tc[2 * c + 1] + mt * kappa;
    tb += nt;
  }
  float u = uniforms[b];
  u = fminf(fmaxf(u, 0.f), 0x1.fffffep-1f);
  const uint64_t u24 = (uint64_t)(u * 0x1p24f);
  const uint64_t target = (uint64_t)(((u128)u24 * Z) >> 24);
  uint64_t mass_base = 0, tie_base = 0;
  int cs = -1;
  tb = 0;
  for (int c = 0; c < C; ++c) {
    const uint64_t nt = tc[2 * c];
    const uint64_t mt = n_tie > tb ? min(nt, n_tie - tb) : 0;
    const uint64_t own = tc[2 * c + 1] + mt * kappa;
    if (own > 0 && mass_base <= target && target < mass_base + own) {
      cs = c;
      tie_base = tb;
      break;
    }
    mass_base += own;
    tb += nt;
  }
  if (cs < 0) return;  // cannot happen: Z > 0 (the max token has mass 2^40)
  const double m = row_max(ws, b, C);
  const double xk = x_floor(kappa);
  const float* z = logits + (int64_t)b * V;
  int i0, i1;
  chunk_range(V, C, cs, i0, i1);
  if (t == 0) found_at = INT_MAX;
  uint64_t run = mass_base, rank = tie_base;
  for (int base = i0; base < i1; base += kST) {
    const int i = base + t;
    uint64_t q = 0;
    if (i < i1) {
      const float zz = z[i];
      if (((double)zz - m) * inv_t >= xk) q = mass_of(zz, m, inv_t);
    }
    const bool tie = q == kappa;  // out-of-range slots have q = 0 < kappa
    // Tie ranks and member masses in index order: wave scans, then the
    // waves before this one.
    const uint64_t tie_mask = __ballot(tie);
    const uint64_t tie_before_w = __popcll(tie_mask & ((1ull << lane) - 1));
    if (lane == 0) wtie[wave] = __popcll(tie_mask);
    __syncthreads();
    uint64_t tie_before = rank + tie_before_w;
    for (int w = 0; w < wave; ++w) tie_before += wtie[w];
    const uint64_t mass = (q > kappa || (tie && tie_before < n_tie)) ? q : 0;
    const uint64_t incl_w = wave_scan_incl(mass, lane);
    if (lane == 63) wsum[wave] = incl_w;
    __syncthreads();
    uint64_t incl = run + incl_w;
    for (int w = 0; w < wave; ++w) incl += wsum[w];
    // The first token (lowest index) whose running mass passes the target.
    const uint64_t hit = __ballot(mass > 0 && incl > target);
    if (hit && lane == __ffsll((unsigned long long)hit) - 1) atomicMin(&found_at, i);
    __syncthreads();
    if (found_at != INT_MAX) {
      if (t == 0) tokens[b] = found_at;
      return;  // uniform: found_at is shared
    }
    for (int w = 0; w < kSW; ++w) {
      run += wsum[w];
      rank += wtie[w];
    }
    __syncthreads();
  }
}

}  // namespace

namespace {

constexpr int sample_split_chunks(int B) {
  // About 256 work groups per pass: 16 chunks per row up to 16 rows, 8 up
  // to 32, none above (at 64 rows the split form's eleven launches already
  // cost more than its wider passes save).
  return (B > 0 ? 256 / B : 1) >= 16 ? 16 : (B > 0 ? 256 / B : 1) >= 8 ? 8 : 1;
}

constexpr int64_t split_workspace_bytes(int B) {
  return sample_split_chunks(B) == 1
             ? 0
             : (int64_t)B * ((int64_t)sizeof(RowState) + sample_split_chunks(B) * 4 +
                             (int64_t)sample_split_chunks(B) * kMaxBins * 8 +
                             sample_split_chunks(B) * 16) +
                   1024;
}

constexpr int64_t max_split_workspace_bytes() {
  int64_t m = 0;
  for (int B = 1; B <= 256; ++B) m = split_workspace_bytes(B) > m ? split_workspace_bytes(B) : m;
  return m;
}

// ---------------------------------------------------------------------------
// Scratch of the no-allocation entry point (sample_top_p_noalloc): the split
// form's row states and per-chunk partial results in a static device array
// sized for the largest batch that takes the split form (about 4 MiB).  Each
// GPU the library runs on holds its own copy until the process ends; every
// call on a GPU shares that GPU's copy, so such calls must not overlap.  No
// entry of it needs clearing: every kernel of the split form writes what
// the next one reads before it is read.
// ---------------------------------------------------------------------------
constexpr int64_t kSampleScratchBytes = max_split_workspace_bytes();
__device__ __align__(256) char sample_scratch[kSampleScratchBytes];

std::mutex g_scratch_mu;
constexpr int kMaxDevices = 64;
void* g_scratch_dev[kMaxDevices] = {};

}  // namespace

int64_t sample_workspace_bytes(int B) { return split_workspace_bytes(B); }

int64_t sample_scratch_bytes() { return kSampleScratchBytes; }

// The device address of this GPU's copy of the scratch array.  In host code
// the array's name is only a host-side stand-in, so the address is looked up
// once per device (with that device current) and kept.
hipError_t sample_scratch_ptr(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(sample_scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return hipSuccess;
}

hipError_t launch_sample_top_p(int B, int V, const float* logits, float temperature, float top_p,
                               const float* uniforms, int32_t* tokens, void* workspace,
                               int64_t ws_bytes, hipStream_t stream) {
  if (B == 0) return hipSuccess;
  const double inv_t = 1.0 / (double)temperature;
  uint32_t p24 = (uint32_t)rint((double)top_p * 16777216.0);
  p24 = p24 < 1 ? 1 : (p24 > (1u << 24) ? (1u << 24) : p24);
  const int C = sample_split_chunks(B);
  if (C == 1 || !workspace || ws_bytes < sample_workspace_bytes(B)) {
    sample_top_p_kernel<<<B, kThreads, 0, stream>>>(V, logits, inv_t, p24, uniforms, tokens);
    return hipGetLastError();
  }
  // Workspace layout (256-byte aligned pieces): row states, chunk maxima,
  // histograms, tie pairs.
  auto al = [](int64_t x) { return (x + 255) & ~(int64_t)255; };
  char* p = (char*)workspace;
  SplitWs ws;
  ws.st = (RowState*)p;
  p += al((int64_t)B * sizeof(RowState));
  ws.cmax = (float*)p;
  p += al((int64_t)B * C * 4);
  ws.hist = (uint64_t*)p;
  p += al((int64_t)B * C * kMaxBins * 8);
  ws.ties = (uint64_t*)p;
  const dim3 grid(C, B);
  split_chunk_max<<<grid, kST, 0, stream>>>(V, C, logits, ws);
  for (int r = 0; r < kRounds; ++r) {
    split_chunk_hist<<<grid, kST, 0, stream>>>(V, C, r, logits, inv_t, ws);
    split_select<<<B, kThreads, 0, stream>>>(C, r, p24, ws);
  }
  split_chunk_ties<<<grid, kST, 0, stream>>>(V, C, logits, inv_t, ws);
  split_walk<<<B, kST, 0, stream>>>(V, C, logits, inv_t, uniforms, tokens, ws);
  return hipGetLastError();
}

}  // namespace pdec

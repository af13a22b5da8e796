// Weight-streaming projections: out[s][m][n] = sum_{k in split s} A[m][k] W[n][k].
//
// Each decode step reads the weights once for the whole active batch (paper:
// Introduction; Design Principles, "Specialization in Heterogeneous Pools"),
// so at decode batch sizes the weight stream from HBM is the bound.  bf16
// weights are stored packed so that this stream is long contiguous runs:
// columns form groups of 128 (8 strips of 16), a 16-column x 32-k block is
// 1 KiB in the lane order of the v_mfma_f32_16x16x32_bf16 B operand (one
// 16-byte load per lane at lane * 8 is exactly one fragment), and the eight
// blocks of one k-block of a group are adjacent, so a group's weight tile for
// a k-step of 64 is one contiguous 16 KiB run (layout at pack_weight_kernel).
// Row-wise [N][K] weights give 128-byte runs in many rows at once and stream
// 10-25% slower.
//
// Kernels by batch rows: the streaming kernel (up to 32 rows, weights straight
// into registers), the 128- and 256-row LDS tiles (up to 256 rows), and the
// 256 x 256 tile above that.  When the column tiles alone cannot fill 256 CUs
// the K axis is split and the fp32 partial sums are reduced in a fixed order
// by the next kernel.
#include "hip_common.h"
#include "kernels.h"

namespace pdec {

namespace {

constexpr int kGroupCols = 128;  // columns per packed group (8 strips of 16)

// Group g of a bf16 weight given as up to three packed segments.
struct GroupRef {
  const uint16_t* base;  // the group's K/32 x 8 blocks of 512 elements
  int col0;              // its first output column
  int col_end;           // end of its segment's output columns
};
__device__ __forceinline__ GroupRef group_ref(const WSegs& w, int g, int K) {
  int s = 0;
  while (s < w.n_seg - 1 && g >= w.grp_end[s]) ++s;
  const int g0 = s ? w.grp_end[s - 1] : 0, c0 = s ? w.row_end[s - 1] : 0;
  return {(const uint16_t*)w.ptr[s] + (int64_t)(g - g0) * kGroupCols * K,
          c0 + (g - g0) * kGroupCols, w.row_end[s]};
}

// Packed bf16 layout (group-major): element (n, k) of an [N][K] matrix is at
//   (((G * K/32 + b) * 8 + s) * 64 + q * 16 + c) * 8 + e,
//   n = 128 G + 16 s + c,  k = 32 b + 8 q + e,
// columns past N zero.  A 16 x 32 block (s, b) is 1 KiB in the lane order of
// the MFMA B operand, and the eight blocks of one k-block of a group are
// adjacent: per k-step of 64 a group's weight tile is one contiguous 16 KiB
// run, so the streams a projection reads from HBM are few and long.
__global__ __launch_bounds__(256) void pack_weight_kernel(const uint16_t* __restrict__ W, int N,
                                                          int K, uint16_t* __restrict__ P) {
  const int KB = K / 32;
  const int64_t chunk = (int64_t)blockIdx.x * 256 + threadIdx.x;  // one 8-element chunk
  if (chunk >= (int64_t)((N + kGroupCols - 1) / kGroupCols) * KB * 8 * 64) return;
  const int l = (int)(chunk & 63);
  const int64_t r = chunk >> 6;
  const int s = (int)(r & 7);
  const int64_t gb = r >> 3;
  const int b = (int)(gb % KB), G = (int)(gb / KB);
  const int n = G * kGroupCols + 16 * s + (l & 15), k = 32 * b + 8 * (l >> 4);
  u32x4 v = {0u, 0u, 0u, 0u};
  if (n < N) v = *(const u32x4*)(W + (int64_t)n * K + k);
  *(u32x4*)(P + chunk * 8) = v;
}

// SwiGLU-fused form (GLU = true, gate and up given as the two segments of
// w, N = the FFN width F, no K split): work group v takes half h = v % 2 of
// group G = v / 2 of both matrices, and each wave the same 16 columns of the
// gate and of the up matrix.  The two results of a column then sit in one
// lane, and the epilogue writes silu(gate) * up as bf16 to u [M][F]: the
// fp32 gate/up products never reach memory.
__device__ __forceinline__ float silu_mul(float g, float u) { return g / (1.f + expf(-g)) * u; }

// Small batches (M <= 32): a work group owns one 128-column group, each of
// its four waves two strips of it and every row of the batch (MT tiles of 16
// rows), so no two waves share weight bytes and no LDS or barrier is needed.
// The weight fragments and the matching activation fragments (L2-resident)
// of the next NS k-steps are in flight in a register ring.  The steady-state
// loop is branch-free (the prefetch index is clamped to the last step) and
// pinned to consume-then-refill order per slot, so the compiler keeps all NS
// slots in flight instead of draining the ring.
template <int MT, int NS, bool GLU>
__global__ __launch_bounds__(256) void gemm_bf16_stream(int M, int N, int K, int k_split,
                                                        const uint16_t* __restrict__ A,
                                                        int64_t lda, WSegs w,
                                                        float* __restrict__ out,
                                                        uint16_t* __restrict__ glu_out) {
  constexpr int WS = 2;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c16 = lane & 15, q4 = lane >> 4;
  const int kbeg = blockIdx.z * k_split;
  const int n_iter = (min(K, kbeg + k_split) - kbeg) / 64;
  if (n_iter <= 0) return;  // no barriers in this kernel

  // Strip s of this wave, k-block kb: wp[s] + kb * 4096 (a k-block of a
  // group is 8 strips of 512 elements).  Plain: strips 2 wave and 2 wave + 1
  // of group blockIdx.x.  GLU: strip 4 h + wave of the gate and of the up
  // matrix's group G.
  const uint16_t* wp[WS];
  int col_s[WS], col_end;
  if constexpr (GLU) {
    const int G = blockIdx.x >> 1, h = blockIdx.x & 1;
    const int64_t off =
        (int64_t)G * kGroupCols * K + ((int64_t)(kbeg / 32) * 8 + 4 * h + wave) * 512 + lane * 8;
    wp[0] = (const uint16_t*)w.ptr[0] + off;
    wp[1] = (const uint16_t*)w.ptr[1] + off;
    col_s[0] = col_s[1] = G * kGroupCols + (4 * h + wave) * 16 + c16;
    col_end = N;
  } else {
    const GroupRef gr = group_ref(w, blockIdx.x, K);
    wp[0] = gr.base + ((int64_t)(kbeg / 32) * 8 + 2 * wave) * 512 + lane * 8;
    wp[1] = wp[0] + 512;
    col_s[0] = gr.col0 + 2 * wave * 16 + c16;
    col_s[1] = col_s[0] + 16;
    col_end = gr.col_end;
  }
  const uint16_t* ap[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t)
    ap[t] = A + (int64_t)min(t * 16 + c16, M - 1) * lda + kbeg + q4 * 8;

  f32x4 acc[MT][WS];
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int s = 0; s < WS; ++s) acc[t][s] = f32x4{0.f, 0.f, 0.f, 0.f};
  bf16x8 rw[NS][WS][2], ra[NS][MT][2];
  auto load = [&](int i, bf16x8(&wr)[WS][2], bf16x8(&ar)[MT][2]) {
#pragma unroll
    for (int s = 0; s < WS; ++s) {
      wr[s][0] = load_stream<bf16x8>(wp[s] + (int64_t)(2 * i) * 4096);
      wr[s][1] = load_stream<bf16x8>(wp[s] + (int64_t)(2 * i + 1) * 4096);
    }
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      ar[t][0] = *(const bf16x8*)(ap[t] + i * 64);
      ar[t][1] = *(const bf16x8*)(ap[t] + i * 64 + 32);
    }
  };
  auto mma = [&](const bf16x8(&wr)[WS][2], const bf16x8(&ar)[MT][2]) {
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int s = 0; s < WS; ++s)
          acc[t][s] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ar[t][h], wr[s][h], acc[t][s], 0, 0, 0);
  };
  const int last = n_iter - 1;
#pragma unroll
  for (int s = 0; s < NS; ++s) load(min(s, last), rw[s], ra[s]);
  int it0 = 0;
  for (; it0 + NS <= n_iter; it0 += NS) {
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      mma(rw[s], ra[s]);
      load(min(it0 + s + NS, last), rw[s], ra[s]);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  const int rem = n_iter - it0;
#pragma unroll
  for (int s = 0; s < NS; ++s)
    if (s < rem) mma(rw[s], ra[s]);

  if constexpr (GLU) {
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int row = t * 16 + 4 * q4 + rr;
        if (row < M && col_s[0] < col_end)
          glu_out[(int64_t)row * N + col_s[0]] = f32_to_bf16(silu_mul(acc[t][0][rr], acc[t][1][rr]));
      }
  } else {
    float* o = out + (int64_t)blockIdx.z * M * N;
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
      for (int s = 0; s < WS; ++s)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          const int row = t * 16 + 4 * q4 + rr;
          if (row < M && col_s[s] < col_end) o[(int64_t)row * N + col_s[s]] = acc[t][s][rr];
        }
  }
}

// Larger batches (M > 32): (64 WM) x 128 output tiles, 2 WM waves in a WM x 2
// grid of 64 x 64 sub-tiles.  Per k-step of 64 the A tile and the W tile are
// staged once through LDS and each is shared by the waves that need it.  The
// tiles travel from memory straight into LDS (16-byte LDS-DMA loads, no
// register staging), through a ring of three stages: while step it is
// computed, steps it+1 and it+2 are in flight.  One barrier per step: after
// it, every wave has finished step it-1, whose stage then takes step it+2.
// The W tile (one packed group, 2 k-blocks x 8 strips) is one contiguous
// 16 KiB run in HBM, copied in packed order (fragment reads from LDS are
// linear, hence free of bank conflicts) with the non-temporal hint, so the
// weight stream does not push the re-read A tiles out of L2; the A tile is row-major with its
// 16-byte chunks XOR-swizzled by
// row (the swizzle is applied to the source address, as the DMA writes each
// wave's 64 chunks contiguously).  WM = 4 covers 256 rows, so up to that
// batch size W is read from HBM exactly once per step.  Larger batches take
// several M-blocks, laid out so the M-blocks of one column tile are
// dispatched back to back (ids L and L+8 share an XCD).
// GLU (gate and up as the two segments of w, N = F, no K split): column tile
// v holds half v % 2 of group v / 2 of both matrices, its eight strips
// staged as gate, up, gate, up, ... so that each wave's four strips are two
// (gate, up) pairs of the same columns; the epilogue writes silu(gate) * up
// as bf16 to u [M][F].
template <int WM, bool GLU>
__global__ __launch_bounds__(128 * WM) void gemm_bf16_tile(int M, int N, int K, int k_split,
                                                          int n_mb, int n_nb,
                                                          const uint16_t* __restrict__ A,
                                                          int64_t lda, WSegs w,
                                                          float* __restrict__ out,
                                                          uint16_t* __restrict__ glu_out) {
  constexpr int MT = 4, NT = 4, D = 3;
  constexpr int THREADS = 128 * WM, ROWS = 64 * WM;
  constexpr int ACH = ROWS * 8 / THREADS;  // A chunks per thread per stage (4)
  constexpr int WCH = 1024 / THREADS;      // W chunks per thread per stage (16 KiB tile)
  constexpr int LPS = ACH + WCH;           // loads per thread per stage
  constexpr int SA = ROWS * 64, STAGE = SA + 128 * 64;
  // One array per stage: the compiler then tells the stages' LDS apart and
  // does not wait for every DMA in flight before reading a landed stage.
  __shared__ __attribute__((aligned(16))) uint16_t lds0[STAGE];
  __shared__ __attribute__((aligned(16))) uint16_t lds1[STAGE];
  __shared__ __attribute__((aligned(16))) uint16_t lds2[STAGE];
  auto stage_ptr = [&](int b) -> uint16_t* { return b == 0 ? lds0 : b == 1 ? lds1 : lds2; };
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int c16 = lane & 15, q4 = lane >> 4;
  const int L = blockIdx.x;
  const int grp = L / (8 * n_mb), rem = L % (8 * n_mb);
  const int mb = rem / 8, nb = grp * 8 + rem % 8;
  if (nb >= n_nb) return;  // padding of the id layout; uniform over the group
  const int kbeg = blockIdx.z * k_split;
  const int n_iter = (min(K, kbeg + k_split) - kbeg) / 64;
  if (n_iter <= 0) return;
  const int m_blk = mb * ROWS;
  const int wm = wave >> 1, wn = wave & 1;
  GroupRef gr;
  if constexpr (GLU) gr = {nullptr, (nb >> 1) * kGroupCols + (nb & 1) * 64, N};
  else gr = group_ref(w, nb, K);

  // Chunk id = j * THREADS + tid lands at LDS chunk id of the stage (the DMA
  // of wave w, load j, fills chunks j * THREADS + 64 w .. +63).  A: chunk id
  // is row id >> 3, slot id & 7, holding source chunk slot ^ (row & 7).
  const uint16_t* asrc[ACH];
#pragma unroll
  for (int j = 0; j < ACH; ++j) {
    const int id = j * THREADS + tid, r = id >> 3, slot = id & 7;
    asrc[j] = A + (int64_t)min(m_blk + r, M - 1) * lda + kbeg + ((slot ^ (r & 7)) * 8);
  }
  // W: chunk id of step i is chunk id of the step's 16 KiB run (k-block
  // 2i + (id >> 9), strip (id >> 6) & 7, lane id & 63).
  const uint16_t* wsrc[WCH];
#pragma unroll
  for (int j = 0; j < WCH; ++j) {
    const int id = j * THREADS + tid;
    if constexpr (GLU) {  // staged strip sp: strip 4 h + sp / 2 of gate (sp even) or up
      const int kb = id >> 9, sp = (id >> 6) & 7, ln = id & 63;
      wsrc[j] = (const uint16_t*)w.ptr[sp & 1] + (int64_t)(nb >> 1) * kGroupCols * K +
                ((int64_t)(kbeg / 32 + kb) * 8 + 4 * (nb & 1) + (sp >> 1)) * 512 + ln * 8;
    } else {
      wsrc[j] = gr.base + (int64_t)(kbeg / 32) * 4096 + id * 8;
    }
  }
  int aoff[MT][2];
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int ra = wm * 64 + t * 16 + c16, cc = h * 4 + q4;
      aoff[t][h] = ra * 64 + ((cc ^ (ra & 7)) * 8);
    }

  f32x4 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto issue = [&](int i, int b) {
    uint16_t* base = stage_ptr(b) + wave * 64 * 8;
#pragma unroll
    for (int j = 0; j < ACH; ++j) dma16(asrc[j] + i * 64, base + j * THREADS * 8);
#pragma unroll
    for (int j = 0; j < WCH; ++j)
      dma16_stream(wsrc[j] + (int64_t)i * 8192, base + SA + j * THREADS * 8);
  };
  auto compute = [&](int b) {
    const uint16_t* la = stage_ptr(b);
    const uint16_t* lw = la + SA;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      bf16x8 af[MT], bf[NT];
#pragma unroll
      for (int t = 0; t < MT; ++t) af[t] = *(const bf16x8*)(la + aoff[t][h]);
#pragma unroll
      for (int t = 0; t < NT; ++t)
        bf[t] = *(const bf16x8*)(lw + ((h * 8 + wn * 4 + t) * 64 + lane) * 8);
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
  };
  // Every step issues one stage (the prefetch index clamped to the last
  // step, so the tail re-reads it into a stage nobody reads), which keeps
  // the count of loads in flight fixed: waiting until D - 2 stages are
  // outstanding means this wave's part of step it has landed; the barrier
  // then covers the other waves' parts.
  const int last = n_iter - 1;
#pragma unroll
  for (int s = 0; s < D - 1; ++s) issue(min(s, last), s);
  int it = 0;
  for (; it + D <= n_iter; it += D) {
#pragma unroll
    for (int s = 0; s < D; ++s) {
      wait_vmem<(D - 2) * LPS>();
      wg_barrier();
      issue(min(it + s + D - 1, last), (s + D - 1) % D);
      __builtin_amdgcn_sched_barrier(0);
      compute(s);
    }
  }
  const int tail = n_iter - it;  // uniform over the work group
#pragma unroll
  for (int s = 0; s < D; ++s)
    if (s < tail) {
      wait_vmem<(D - 2) * LPS>();
      wg_barrier();
      issue(min(it + s + D - 1, last), (s + D - 1) % D);
      __builtin_amdgcn_sched_barrier(0);
      compute(s);
    }
  wait_vmem<0>();  // no LDS write may still be in flight when the group ends

  if constexpr (GLU) {
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int p = 0; p < NT / 2; ++p) {
        const int col = gr.col0 + (2 * wn + p) * 16 + c16;
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          const int row = m_blk + wm * 64 + i * 16 + 4 * q4 + rr;
          if (row < M && col < gr.col_end)
            glu_out[(int64_t)row * N + col] =
                f32_to_bf16(silu_mul(acc[i][2 * p][rr], acc[i][2 * p + 1][rr]));
        }
      }
  } else {
    float* o = out + (int64_t)blockIdx.z * M * N;
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        const int col = gr.col0 + wn * 64 + j * 16 + c16;
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          const int row = m_blk + wm * 64 + i * 16 + 4 * q4 + rr;
          if (row < M && col < gr.col_end) o[(int64_t)row * N + col] = acc[i][j][rr];
        }
      }
  }
}

// Batches above 256 rows (prefill chunks, B = 512 decode): 256 x 256 output
// tiles, 8 waves in a 4 x 2 grid of 64 x 128 sub-tiles (each wave's columns
// are one packed group, NT = 8 strips).  Against the 256 x 128 tile this
// halves the A bytes each output needs from L2 (the A tile is shared by two
// column groups) and reads 12 fragments from LDS per 32 MFMAs instead of 16.
// Stages hold one k-block (32): A 256 rows x 64 B (16-byte chunks swizzled
// by row so that the 16 rows of a fragment read hit distinct banks) and W
// 2 groups x 8 strips (two contiguous 8 KiB runs); a ring of four stages
// keeps three k-blocks in flight.  Column tile v covers groups 2v and 2v + 1
// (the second clamped to a valid group and its outputs dropped when the
// group count is odd); GLU: column tile v is group v of both matrices, wave
// column wn taking half wn of it with its strips staged as gate, up, gate,
// up, ... (four (gate, up) pairs per wave), and the epilogue writes
// silu(gate) * up as bf16.
template <bool GLU>
__global__ __launch_bounds__(512) void gemm_bf16_wide(int M, int N, int K, int k_split,
                                                     int n_mb, int n_nb, int n_groups,
                                                     const uint16_t* __restrict__ A,
                                                     int64_t lda, WSegs w,
                                                     float* __restrict__ out,
                                                     uint16_t* __restrict__ glu_out) {
  constexpr int MT = 4, NT = 8, D = 4, THREADS = 512, ROWS = 256;
  constexpr int ACH = ROWS * 4 / THREADS;  // A chunks per thread per stage (2)
  constexpr int WCH = 1024 / THREADS;      // W chunks per thread per stage (2)
  constexpr int LPS = ACH + WCH;
  constexpr int SA = ROWS * 32, STAGE = SA + 2 * 8 * 512;  // elements
  __shared__ __attribute__((aligned(16))) uint16_t lds0[STAGE];
  __shared__ __attribute__((aligned(16))) uint16_t lds1[STAGE];
  __shared__ __attribute__((aligned(16))) uint16_t lds2[STAGE];
  __shared__ __attribute__((aligned(16))) uint16_t lds3[STAGE];
  auto stage_ptr = [&](int b) -> uint16_t* {
    return b == 0 ? lds0 : b == 1 ? lds1 : b == 2 ? lds2 : lds3;
  };
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int c16 = lane & 15, q4 = lane >> 4;
  const int L = blockIdx.x;
  const int grp = L / (8 * n_mb), rem = L % (8 * n_mb);
  const int mb = rem / 8, nb = grp * 8 + rem % 8;
  if (nb >= n_nb) return;  // padding of the id layout; uniform over the group
  const int kbeg = blockIdx.z * k_split;
  const int n_iter = (min(K, kbeg + k_split) - kbeg) / 32;
  if (n_iter <= 0) return;
  const int m_blk = mb * ROWS;
  const int wm = wave >> 1, wn = wave & 1;

  // This wave's output columns: strip t covers col0 + 16 t .. + 15 (plain) or
  // the pair p = t / 2 covers col0 + 16 p .. + 15 (GLU).
  int col0, col_end;
  if constexpr (GLU) {
    col0 = nb * kGroupCols + wn * 64;
    col_end = N;
  } else {
    const int gw = 2 * nb + wn;
    const GroupRef gr = group_ref(w, min(gw, n_groups - 1), K);
    col0 = gr.col0;
    col_end = gw < n_groups ? gr.col_end : 0;  // a clamped second group writes nothing
  }

  // A: chunk id = row * 4 + slot, holding source chunk slot ^ ((row >> 1) & 3).
  // A row is 64 bytes, so two rows share one 128-byte span of the banks; a
  // fragment read (eight consecutive lanes = eight consecutive rows, one
  // logical chunk) then lands on eight distinct 16-byte bank groups: even and
  // odd rows take the two halves, and (row >> 1) & 3 spreads the four of each.
  const uint16_t* asrc[ACH];
#pragma unroll
  for (int j = 0; j < ACH; ++j) {
    const int id = j * THREADS + tid, r = id >> 2, slot = id & 3;
    asrc[j] = A + (int64_t)min(m_blk + r, M - 1) * lda + kbeg + ((slot ^ ((r >> 1) & 3)) * 8);
  }
  // W: chunk id = (g2 * 8 + sp) * 64 + lane of staged group g2 (the wave
  // column that reads it), staged strip sp.
  const uint16_t* wsrc[WCH];
#pragma unroll
  for (int j = 0; j < WCH; ++j) {
    const int id = j * THREADS + tid, g2 = id >> 9, sp = (id >> 6) & 7, ln = id & 63;
    if constexpr (GLU) {
      wsrc[j] = (const uint16_t*)w.ptr[sp & 1] + (int64_t)nb * kGroupCols * K +
                ((int64_t)(kbeg / 32) * 8 + 4 * g2 + (sp >> 1)) * 512 + ln * 8;
    } else {
      const GroupRef gs = group_ref(w, min(2 * nb + g2, n_groups - 1), K);
      wsrc[j] = gs.base + ((int64_t)(kbeg / 32) * 8 + sp) * 512 + ln * 8;
    }
  }
  int aoff[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    const int ra = wm * 64 + t * 16 + c16;
    aoff[t] = ra * 32 + ((q4 ^ ((ra >> 1) & 3)) * 8);
  }

  f32x4 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto issue = [&](int i, int b) {
    uint16_t* base = stage_ptr(b) + wave * 64 * 8;
#pragma unroll
    for (int j = 0; j < ACH; ++j) dma16(asrc[j] + i * 32, base + j * THREADS * 8);
#pragma unroll
    for (int j = 0; j < WCH; ++j)
      dma16_stream(wsrc[j] + (int64_t)i * 4096, base + SA + j * THREADS * 8);
  };
  auto compute = [&](int b) {
    const uint16_t* la = stage_ptr(b);
    const uint16_t* lw = la + SA + wn * 8 * 512;
    bf16x8 af[MT], bf[NT];
#pragma unroll
    for (int t = 0; t < MT; ++t) af[t] = *(const bf16x8*)(la + aoff[t]);
#pragma unroll
    for (int t = 0; t < NT; ++t) bf[t] = *(const bf16x8*)(lw + (t * 64 + lane) * 8);
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NT; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
  };
  // As in the 256 x 128 tile: every step issues one stage (the prefetch index
  // clamped to the last step), so waiting until D - 2 stages are outstanding
  // means this wave's part of step it has landed; the barrier covers the
  // other waves' parts and frees the stage that step it + D - 1 refills.
  const int last = n_iter - 1;
#pragma unroll
  for (int s = 0; s < D - 1; ++s) issue(min(s, last), s);
  int it = 0;
  for (; it + D <= n_iter; it += D) {
#pragma unroll
    for (int s = 0; s < D; ++s) {
      wait_vmem<(D - 2) * LPS>();
      wg_barrier();
      issue(min(it + s + D - 1, last), (s + D - 1) % D);
      __builtin_amdgcn_sched_barrier(0);
      compute(s);
    }
  }
  const int tail = n_iter - it;  // uniform over the work group
#pragma unroll
  for (int s = 0; s < D; ++s)
    if (s < tail) {
      wait_vmem<(D - 2) * LPS>();
      wg_barrier();
      issue(min(it + s + D - 1, last), (s + D - 1) % D);
      __builtin_amdgcn_sched_barrier(0);
      compute(s);
    }
  wait_vmem<0>();  // no LDS write may still be in flight when the group ends

  if constexpr (GLU) {
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int p = 0; p < NT / 2; ++p) {
        const int col = col0 + p * 16 + c16;
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          const int row = m_blk + wm * 64 + i * 16 + 4 * q4 + rr;
          if (row < M && col < col_end)
            glu_out[(int64_t)row * N + col] =
                f32_to_bf16(silu_mul(acc[i][2 * p][rr], acc[i][2 * p + 1][rr]));
        }
      }
  } else {
    float* o = out + (int64_t)blockIdx.z * M * N;
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        const int col = col0 + j * 16 + c16;
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          const int row = m_blk + wm * 64 + i * 16 + 4 * q4 + rr;
          if (row < M && col < col_end) o[(int64_t)row * N + col] = acc[i][j][rr];
        }
      }
  }
}

// fp32 weights are row-major [N][K] (the packed layout is for bf16 only).
__device__ __forceinline__ const void* seg_row(const WSegs& w, int n, int64_t row_elems,
                                               int elem_bytes) {
  int start = 0;
  for (int s = 0; s < w.n_seg; ++s) {
    if (n < w.row_end[s])
      return (const char*)w.ptr[s] + (int64_t)(n - start) * row_elems * elem_bytes;
    start = w.row_end[s];
  }
  return w.ptr[0];
}

// fp32: 32 x 64 tiles through LDS, 2 x 4 outputs per thread.
__global__ __launch_bounds__(256) void gemm_f32_tiled(int M, int N, int K, int k_split,
                                                      const float* __restrict__ A, int64_t lda,
                                                      WSegs w, float* __restrict__ out) {
  __shared__ float As[16][33];
  __shared__ float Ws[16][65];
  const int tid = threadIdx.x;
  const int m0 = blockIdx.y * 32, n0 = blockIdx.x * 64;
  const int kbeg = blockIdx.z * k_split;
  const int kend = min(K, kbeg + k_split);
  const int tm = tid >> 4, tn = tid & 15;
  float acc[2][4] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
  for (int k0 = kbeg; k0 < kend; k0 += 16) {
    for (int e = tid; e < 32 * 16; e += 256) {
      const int mm = e >> 4, kk = e & 15, row = m0 + mm, k = k0 + kk;
      As[kk][mm] = (row < M && k < kend) ? A[(int64_t)row * lda + k] : 0.f;
    }
    for (int e = tid; e < 64 * 16; e += 256) {
      const int nn = e >> 4, kk = e & 15, n = n0 + nn, k = k0 + kk;
      Ws[kk][nn] = (n < N && k < kend) ? ((const float*)seg_row(w, n, K, 4))[k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      const float a0 = As[kk][tm * 2], a1 = As[kk][tm * 2 + 1];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float b = Ws[kk][tn * 4 + j];
        acc[0][j] += a0 * b;
        acc[1][j] += a1 * b;
      }
    }
    __syncthreads();
  }
  float* o = out + (int64_t)blockIdx.z * M * N;
  for (int i = 0; i < 2; ++i)
    for (int j = 0; j < 4; ++j) {
      const int row = m0 + tm * 2 + i, col = n0 + tn * 4 + j;
      if (row < M && col < N) o[(int64_t)row * N + col] = acc[i][j];
    }
}

}  // namespace

// Kernel choice for bf16, from measurements on the 8B projection shapes:
//  * M <= 32: the streaming kernel (two strips per wave, ring depth 2);
//    6.0-6.6 TB/s of weights up to M = 16;
//  * larger M: the 128 x 128 tile (M <= 128) or 256 x 128 tile, and above
//    256 rows the 256 x 256 tile where its grid fills the GPU.
constexpr int kStreamMaxRows = 32;

// Rows per tile: 128 (4 waves) up to 128-row batches, 256 (8 waves) beyond,
// so W is read once per step for batches up to 256.  Above 256 rows the
// 256 x 256 tile (two column groups per work group).
int tile_rows(int M) { return M <= 128 ? 128 : 256; }
// The 256 x 256 tile is taken only where its grid alone fills the GPU
// (gate/up and the LM head at any M > 256, qkv only past ~2300 rows): where
// it would need more K splits than the 256 x 128 tile (o, down, qkv at
// 384-1024 rows) the extra partial traffic made it 5-45% slower.
bool wide_tiles(int M, int64_t groups) {
  return M > 256 && ((groups + 1) / 2) * ((M + 255) / 256) >= 224;
}

int gemm_plan_splits(int dtype, int M, int N, int K, int* k_split) {
  const int kq = (dtype == 1) ? 64 : 16;
  const int ksteps = (K + kq - 1) / kq;
  int s = 1;
  if (dtype == 1) {
    // Work groups per split: one per 128-column group (times the M-blocks).
    int64_t groups = (N + kGroupCols - 1) / kGroupCols;
    if (wide_tiles(M, groups)) groups = ((groups + 1) / 2) * ((M + 255) / 256);
    else if (M > kStreamMaxRows) groups *= (M + tile_rows(M) - 1) / tile_rows(M);
    // Measured on the 8B shapes with weights streamed from HBM: the best
    // split count fills one round of work groups on the 256 CUs (a partial
    // second round costs 15-30%).
    s = (int)std::max<int64_t>(1, 256 / groups);
    s = std::min(s, 8);
    // Above 256 rows (prefill chunks, large batches) with a long K (the down
    // projection), a grid of 129-255 work groups fills one round poorly; up
    // to 4 splits are weighed by rounds per unit of work,
    // ceil(groups * s / 256) / s, ties to fewer splits.  Measured at 640-1536
    // rows this picked the best count every time (1242 rows: 160 groups,
    // 3 splits, 142 against 189 us).  With K = 4096 the shorter split loops
    // and the partials cost more than the rounds save, so those keep the
    // rule above.
    if (M > 256 && groups < 256 && K >= 8192) {
      double best = 1e30;
      for (int c = 1; c <= 4; ++c) {
        const double cost = (double)((groups * c + 255) / 256) / c;
        if (cost < best - 1e-9) best = cost, s = c;
      }
    }
  } else {
    const int64_t groups = (int64_t)((N + 63) / 64) * ((M + 31) / 32);
    if (groups < 512) s = (int)std::min<int64_t>((512 + groups - 1) / groups, 8);
  }
  s = std::max(1, std::min(s, ksteps));
  const int steps_per = (ksteps + s - 1) / s;
  *k_split = steps_per * kq;
  return (K + *k_split - 1) / *k_split;
}

hipError_t launch_pack_weight(int dtype, int N, int K, const void* w, void* packed,
                              hipStream_t stream) {
  if (N <= 0 || K <= 0) return hipSuccess;
  if (dtype != 1)
    return hipMemcpyAsync(packed, w, (size_t)N * K * 4, hipMemcpyDeviceToDevice, stream);
  const int64_t chunks = (int64_t)((N + kGroupCols - 1) / kGroupCols) * (K / 32) * 8 * 64;
  pack_weight_kernel<<<(unsigned)((chunks + 255) / 256), 256, 0, stream>>>(
      (const uint16_t*)w, N, K, (uint16_t*)packed);
  return hipGetLastError();
}

namespace {

// The bf16 kernels over n_groups column groups (GLU: half-groups).
template <bool GLU>
hipError_t launch_gemm_bf16(int M, int N, int K, const uint16_t* a, int64_t lda, const WSegs& w,
                            int n_groups, float* out, uint16_t* glu_out, int splits, int k_split,
                            hipStream_t stream, hipEvent_t ev_start, hipEvent_t ev_stop) {
  // Plain matrices given as several segments (q|k|v) keep the 256 x 128 tile.
  const bool wide = wide_tiles(M, n_groups) && (GLU || w.n_seg == 1);
  if (M <= kStreamMaxRows) {
    const dim3 grid(n_groups, 1, splits);
    if (M <= 16)
      return launch_timed(gemm_bf16_stream<1, 2, GLU>, grid, dim3(256), stream, ev_start,
                          ev_stop, M, N, K, k_split, a, lda, w, out, glu_out);
    return launch_timed(gemm_bf16_stream<2, 2, GLU>, grid, dim3(256), stream, ev_start, ev_stop,
                        M, N, K, k_split, a, lda, w, out, glu_out);
  }
  if (wide) {
    // GLU: n_groups counts half-groups; a wide column tile is one whole group.
    const int n_mb = (M + 255) / 256, n_nb = GLU ? n_groups / 2 : (n_groups + 1) / 2;
    const dim3 grid(((n_nb + 7) / 8) * 8 * n_mb, 1, splits);
    return launch_timed(gemm_bf16_wide<GLU>, grid, dim3(512), stream, ev_start, ev_stop, M, N, K,
                        k_split, n_mb, n_nb, n_groups, a, lda, w, out, glu_out);
  }
  const int rows = tile_rows(M);
  const int n_mb = (M + rows - 1) / rows, n_nb = n_groups;
  const dim3 grid(((n_nb + 7) / 8) * 8 * n_mb, 1, splits);
  if (rows == 128)
    return launch_timed(gemm_bf16_tile<2, GLU>, grid, dim3(256), stream, ev_start, ev_stop, M, N,
                        K, k_split, n_mb, n_nb, a, lda, w, out, glu_out);
  return launch_timed(gemm_bf16_tile<4, GLU>, grid, dim3(512), stream, ev_start, ev_stop, M, N, K,
                      k_split, n_mb, n_nb, a, lda, w, out, glu_out);
}

}  // namespace

namespace {

// The fused gate/up grid has one work group per half column-group of both
// matrices (up to 256 rows: one M-block).  When that count is whole rounds
// of the 256 CUs plus a last round at most half full (F = 17408: 272
// half-groups), the last round runs nearly as long as a full one while most
// CUs idle: at K = 5120 and 128 rows, 272 half-groups took 112 us against
// 70 us for 256.  Those tail columns then take the plain kernels with their
// K axis split (up to 16 ways, so that the tail fills one round of short
// work groups) and a SwiGLU pass over the summed partials.
struct GluPlan {
  int fused_halves;  // half-groups of the fused launch (a multiple of 256 when split)
  int tail_halves;   // half-groups left to the split launch (0: none)
  int splits, k_split;
};

GluPlan plan_glu(int M, int F, int K) {
  const int halves = 2 * ((F + kGroupCols - 1) / kGroupCols);
  GluPlan p{halves, 0, 1, K};
  const int tail = halves % 256;
  if (M > 256 || halves < 256 || tail == 0 || tail > 128) return p;
  const int ksteps = K / 64, want = std::min(16, 256 / tail);
  const int per = (ksteps + want - 1) / want;  // k-steps of 64 per split
  const int splits = (ksteps + per - 1) / per;
  if (splits < 2) return p;
  return {halves - tail, tail, splits, per * 64};
}

}  // namespace

int64_t swiglu_tail_part_elems(int M, int F, int K) {
  const GluPlan g = plan_glu(M, F, K);
  if (g.tail_halves == 0) return 0;
  const int64_t ft = F - (int64_t)(g.fused_halves / 2) * kGroupCols;  // tail columns per matrix
  return (int64_t)g.splits * M * 2 * ft;
}

hipError_t launch_gemm_swiglu(int M, int F, int K, const void* A, int64_t lda, const void* w_gate,
                              const void* w_up, void* u, float* tail_part, hipStream_t stream,
                              hipEvent_t ev_start, hipEvent_t ev_stop) {
  if (M <= 0 || F <= 0) return hipSuccess;
  WSegs w{};
  w.ptr[0] = w_gate;
  w.ptr[1] = w_up;
  w.row_end[0] = F;
  w.row_end[1] = 2 * F;
  w.n_seg = 2;
  const GluPlan g = plan_glu(M, F, K);
  if (g.tail_halves == 0 || !tail_part)
    return launch_gemm_bf16<true>(M, F, K, (const uint16_t*)A, lda, w, 2 * ((F + 127) / 128),
                                  nullptr, (uint16_t*)u, 1, K, stream, ev_start, ev_stop);
  // Whole groups [0, g0) of both matrices fused; groups [g0, ...) split.
  hipError_t e = launch_gemm_bf16<true>(M, F, K, (const uint16_t*)A, lda, w, g.fused_halves,
                                        nullptr, (uint16_t*)u, 1, K, stream, ev_start, nullptr);
  if (e != hipSuccess) return e;
  const int g0 = g.fused_halves / 2, ft = F - g0 * kGroupCols, tg = (ft + kGroupCols - 1) / kGroupCols;
  WSegs t{};
  t.ptr[0] = (const uint16_t*)w_gate + (int64_t)g0 * kGroupCols * K;
  t.ptr[1] = (const uint16_t*)w_up + (int64_t)g0 * kGroupCols * K;
  t.row_end[0] = ft;
  t.row_end[1] = 2 * ft;
  t.grp_end[0] = tg;
  t.grp_end[1] = 2 * tg;
  t.n_seg = 2;
  e = launch_gemm_bf16<false>(M, 2 * ft, K, (const uint16_t*)A, lda, t, 2 * tg, tail_part, nullptr,
                              g.splits, g.k_split, stream, nullptr, nullptr);
  if (e != hipSuccess) return e;
  e = launch_swiglu(1, M, ft, tail_part, g.splits, (uint16_t*)u + (int64_t)g0 * kGroupCols, stream,
                    F);
  if (e == hipSuccess && ev_stop) e = hipEventRecord(ev_stop, stream);
  return e;
}

hipError_t launch_gemm(int dtype, int M, int N, int K, const void* A, int64_t lda,
                       const WSegs& w_in, float* out, int splits, int k_split, hipStream_t stream,
                       hipEvent_t ev_start, hipEvent_t ev_stop) {
  if (M <= 0 || N <= 0) return hipSuccess;
  const dim3 block(256);
  if (dtype == 1) {
    // Each segment is padded to whole groups; count them.
    WSegs w = w_in;
    int start = 0, n_groups = 0;
    for (int s = 0; s < w.n_seg; ++s) {
      n_groups += (w.row_end[s] - start + kGroupCols - 1) / kGroupCols;
      w.grp_end[s] = n_groups;
      start = w.row_end[s];
    }
    return launch_gemm_bf16<false>(M, N, K, (const uint16_t*)A, lda, w, n_groups, out, nullptr,
                                   splits, k_split, stream, ev_start, ev_stop);
  } else {
    const dim3 grid((N + 63) / 64, (M + 31) / 32, splits);
    return launch_timed(gemm_f32_tiled, grid, block, stream, ev_start, ev_stop, M, N, K, k_split,
                        (const float*)A, lda, w_in, out);
  }
  return hipGetLastError();
}

}  // namespace pdec

// Weight-streaming projections: out[s][m][n] = sum_{k in split s} A[m][k] W[n][k].
//
// Each decode step reads the weights once for the whole active batch (paper:
// Introduction; Design Principles, "Specialization in Heterogeneous Pools").
// A work group owns a 64-column slice of W and every row of the batch, so W
// is streamed from HBM exactly once per step; the activations (at most a few
// MB) stay in L2.  When the column slices alone cannot fill 256 CUs the K
// axis is split and the fp32 partial sums are reduced by the next kernel.
//
// bf16: v_mfma_f32_16x16x32_bf16 tiles of 16 rows x 16 columns.  The
// weight stream is the bound at small batch, so weight tiles are prefetched
// several k-steps ahead to keep enough bytes in flight per CU.
#include "hip_common.h"
#include "kernels.h"

namespace pdec {

namespace {

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

// Small batches (M <= 4 with long K in practice, up to 64 supported).  Each
// wave owns 16 columns of the 64-column
// block and every row of the batch, so no two waves share weight bytes.  The
// weight fragments are prefetched NS k-steps ahead through a register ring so
// that enough HBM bytes are in flight to hide the memory latency; the
// activations (L2-resident) are prefetched one step ahead.
template <int MT, int NS>
__global__ __launch_bounds__(256, 2) void gemm_bf16_small_m(int M, int N, int K, int k_split,
                                                            const uint16_t* __restrict__ A,
                                                            int64_t lda, WSegs w,
                                                            float* __restrict__ out) {
  static_assert(NS % 2 == 0, "ring depth must be even");
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c16 = lane & 15, q4 = lane >> 4;
  const int n0 = blockIdx.x * 64 + wave * 16;
  const int kbeg = blockIdx.z * k_split;
  const int n_iter = (min(K, kbeg + k_split) - kbeg) / 64;
  if (n0 >= N || n_iter <= 0) return;  // no barriers in this kernel

  const uint16_t* wrow = (const uint16_t*)seg_row(w, min(n0 + c16, N - 1), K, 2) + kbeg + q4 * 8;
  const uint16_t* arow[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t)
    arow[t] = A + (int64_t)min(t * 16 + c16, M - 1) * lda + kbeg + q4 * 8;

  f32x4 acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  bf16x8 wr[NS][2];
  bf16x8 ar[2][MT][2];
#pragma unroll
  for (int s = 0; s < NS; ++s)
    if (s < n_iter) {
      wr[s][0] = load_stream<bf16x8>(wrow + s * 64);
      wr[s][1] = load_stream<bf16x8>(wrow + s * 64 + 32);
    }
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    ar[0][t][0] = *(const bf16x8*)(arow[t]);
    ar[0][t][1] = *(const bf16x8*)(arow[t] + 32);
  }
  for (int it0 = 0; it0 < n_iter; it0 += NS) {
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const int it = it0 + s;
      if (it >= n_iter) break;
      const bf16x8 b0 = wr[s][0], b1 = wr[s][1];
      if (it + NS < n_iter) {
        wr[s][0] = load_stream<bf16x8>(wrow + (it + NS) * 64);
        wr[s][1] = load_stream<bf16x8>(wrow + (it + NS) * 64 + 32);
      }
      if (it + 1 < n_iter) {
#pragma unroll
        for (int t = 0; t < MT; ++t) {
          ar[(s + 1) & 1][t][0] = *(const bf16x8*)(arow[t] + (it + 1) * 64);
          ar[(s + 1) & 1][t][1] = *(const bf16x8*)(arow[t] + (it + 1) * 64 + 32);
        }
      }
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ar[s & 1][t][0], b0, acc[t], 0, 0, 0);
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ar[s & 1][t][1], b1, acc[t], 0, 0, 0);
      }
    }
  }

  float* o = out + (int64_t)blockIdx.z * M * N;
  const int col = n0 + c16;
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int row = t * 16 + 4 * q4 + rr;
      if (row < M && col < N) o[(int64_t)row * N + col] = acc[t][rr];
    }
}

// Larger batches (M > 4): (64 WM) x 128 output tiles, 2 WM waves in a WM x 2
// grid of 64 x 64 sub-tiles.  Per k-step of 64 the A tile and the W tile are
// staged once through LDS (double-buffered, 16-byte chunks XOR-swizzled by
// row) and each is shared by the waves that need it; the tiles of the next
// NS k-steps are prefetched into a register ring meanwhile (NS even: ring
// slot s also names the LDS buffer s & 1).  WM = 4 covers 256 rows, so up to
// that batch size W is read from HBM exactly once per step.  Larger batches
// take several M-blocks, laid out so the M-blocks of one column tile are
// dispatched back to back (ids L and L+8 share an XCD).
template <int WM, int NS, int NA>
__global__ __launch_bounds__(128 * WM) void gemm_bf16_tile(int M, int N, int K, int k_split,
                                                          int n_mb, int n_nb,
                                                          const uint16_t* __restrict__ A,
                                                          int64_t lda, WSegs w,
                                                          float* __restrict__ out) {
  constexpr int MT = 4, NT = 4;
  constexpr int THREADS = 128 * WM, ROWS = 64 * WM;
  constexpr int RSTEP = THREADS / 8;  // rows covered by one chunk column of the group
  constexpr int ACH = ROWS / RSTEP;   // A chunks per thread (4)
  constexpr int WCH = 128 / RSTEP;    // W chunks per thread
  __shared__ __attribute__((aligned(16))) uint16_t la_s[2][ROWS * 64];
  __shared__ __attribute__((aligned(16))) uint16_t lw_s[2][128 * 64];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int c16 = lane & 15, q4 = lane >> 4;
  const int L = blockIdx.x;
  const int grp = L / (8 * n_mb), rem = L % (8 * n_mb);
  const int mb = rem / 8, nb = grp * 8 + rem % 8;
  if (nb >= n_nb) return;  // padding of the id layout; uniform over the group
  const int kbeg = blockIdx.z * k_split;
  const int n_iter = (min(K, kbeg + k_split) - kbeg) / 64;
  if (n_iter <= 0) return;
  const int m_blk = mb * ROWS, n_blk = nb * 128;
  const int wm = wave >> 1, wn = wave & 1;

  const int r = tid >> 3, c = tid & 7;
  const int dst = r * 64 + ((c ^ (r & 7)) * 8);  // + j * RSTEP * 64 for chunk j
  const uint16_t* asrc[ACH];
  const uint16_t* wsrc[WCH];
#pragma unroll
  for (int j = 0; j < ACH; ++j)
    asrc[j] = A + (int64_t)min(m_blk + r + RSTEP * j, M - 1) * lda + kbeg + c * 8;
#pragma unroll
  for (int j = 0; j < WCH; ++j)
    wsrc[j] = (const uint16_t*)seg_row(w, min(n_blk + r + RSTEP * j, N - 1), K, 2) + kbeg + c * 8;
  int aoff[MT][2], boff[NT][2];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int ra = wm * 64 + t * 16 + c16, rb = wn * 64 + t * 16 + c16, cc = h * 4 + q4;
      aoff[t][h] = ra * 64 + ((cc ^ (ra & 7)) * 8);
      boff[t][h] = rb * 64 + ((cc ^ (rb & 7)) * 8);
    }

  f32x4 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // W (from HBM) is prefetched NS k-steps ahead, A (L2-resident) NA.
  static_assert(NS % NA == 0 && NA % 2 == 0, "ring depths");
  u16x8 ra_[NA][ACH], rw_[NS][WCH];
#pragma unroll
  for (int s = 0; s < NS; ++s)
    if (s < n_iter) {
#pragma unroll
      for (int j = 0; j < WCH; ++j) rw_[s][j] = *(const u16x8*)(wsrc[j] + s * 64);
      if (s < NA) {
#pragma unroll
        for (int j = 0; j < ACH; ++j) ra_[s][j] = *(const u16x8*)(asrc[j] + s * 64);
      }
    }
  for (int it0 = 0; it0 < n_iter; it0 += NS) {
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const int it = it0 + s;
      if (it >= n_iter) break;
      uint16_t* la = la_s[s & 1];
      uint16_t* lw = lw_s[s & 1];
#pragma unroll
      for (int j = 0; j < ACH; ++j) *(u16x8*)(la + dst + j * RSTEP * 64) = ra_[s % NA][j];
#pragma unroll
      for (int j = 0; j < WCH; ++j) *(u16x8*)(lw + dst + j * RSTEP * 64) = rw_[s][j];
      __syncthreads();
      if (it + NS < n_iter) {
#pragma unroll
        for (int j = 0; j < WCH; ++j) rw_[s][j] = *(const u16x8*)(wsrc[j] + (it + NS) * 64);
      }
      if (it + NA < n_iter) {
#pragma unroll
        for (int j = 0; j < ACH; ++j) ra_[s % NA][j] = *(const u16x8*)(asrc[j] + (it + NA) * 64);
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        bf16x8 af[MT], bf[NT];
#pragma unroll
        for (int t = 0; t < MT; ++t) af[t] = *(const bf16x8*)(la + aoff[t][h]);
#pragma unroll
        for (int t = 0; t < NT; ++t) bf[t] = *(const bf16x8*)(lw + boff[t][h]);
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
          for (int j = 0; j < NT; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
      }
    }
  }

  float* o = out + (int64_t)blockIdx.z * M * N;
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const int col = n_blk + wn * 64 + j * 16 + c16;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int row = m_blk + wm * 64 + i * 16 + 4 * q4 + rr;
        if (row < M && col < N) o[(int64_t)row * N + col] = acc[i][j][rr];
      }
    }
}

// VALU weight-streaming GEMV for tiny batches (M <= 4): out[m][n] =
// sum_k x[m][k] W[n][k] with v_dot2_f32_bf16.  Each wave streams whole
// contiguous weight rows (a row of K bf16 is K*2 contiguous bytes, read 1 KiB
// per instruction), so the weight stream is long sequential runs; the batch's
// activations sit in LDS.  Every wave covers the full K of its rows: no
// split-K, results go straight to out (splits = 1).
// Whole vectors are reinterpreted and split by shuffles (bit-casting a
// single vector element would read the vector's first element).
__device__ __forceinline__ float dot8(const u32x4 w, const u32x4 x, float acc) {
  const bf16x8 wb = __builtin_bit_cast(bf16x8, w), xb = __builtin_bit_cast(bf16x8, x);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(wb, wb, 0, 1),
                                        __builtin_shufflevector(xb, xb, 0, 1), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(wb, wb, 2, 3),
                                        __builtin_shufflevector(xb, xb, 2, 3), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(wb, wb, 4, 5),
                                        __builtin_shufflevector(xb, xb, 4, 5), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(wb, wb, 6, 7),
                                        __builtin_shufflevector(xb, xb, 6, 7), acc, false);
  return acc;
}

template <int M>
__global__ __launch_bounds__(256) void gemv_bf16(int N, int K, int rows_per_wave,
                                                 const uint16_t* __restrict__ x, int64_t ldx,
                                                 WSegs w, float* __restrict__ out) {
  extern __shared__ __attribute__((aligned(16))) uint16_t xs[];  // [M][K]
  for (int i = threadIdx.x * 8; i < M * K; i += 256 * 8) {
    const int m = i / K, k = i % K;
    *(u32x4*)(xs + i) = *(const u32x4*)(x + (int64_t)m * ldx + k);
  }
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int n0 = (blockIdx.x * 4 + wave) * rows_per_wave;
  const int n1 = min(N, n0 + rows_per_wave);
  for (int n = n0; n < n1; ++n) {
    const uint16_t* wr = (const uint16_t*)seg_row(w, n, K, 2);
    float acc[M];
#pragma unroll
    for (int m = 0; m < M; ++m) acc[m] = 0.f;
    int k = lane * 8;
    for (; k + 3 * 512 < K; k += 4 * 512) {
      u32x4 wv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) wv[u] = load_stream<u32x4>(wr + k + u * 512);
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int m = 0; m < M; ++m)
          acc[m] = dot8(wv[u], *(const u32x4*)(xs + m * K + k + u * 512), acc[m]);
    }
    for (; k < K; k += 512) {
      const u32x4 wv = load_stream<u32x4>(wr + k);
#pragma unroll
      for (int m = 0; m < M; ++m) acc[m] = dot8(wv, *(const u32x4*)(xs + m * K + k), acc[m]);
    }
#pragma unroll
    for (int m = 0; m < M; ++m) {
      const float v = wave_sum(acc[m]);
      if (lane == m) out[(int64_t)m * N + n] = v;
    }
  }
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
//  * GEMV (VALU dot2, whole-row streaming) while the batch's activations fit
//    in 64 KB of LDS and M <= 4: 6.2-6.6 TB/s at M = 1, ahead of MFMA up to
//    M = 4;
//  * the register-ring MFMA kernel for the remaining M <= 4 (long K);
//  * the 128 x 128 tile MFMA kernel above that.
enum class GemmPath { kGemv, kSmallM, kTile128 };

GemmPath bf16_path(int M, int K) {
  if (M <= 4 && (int64_t)M * K * 2 <= 64 * 1024) return GemmPath::kGemv;
  if (M <= 4) return GemmPath::kSmallM;
  return GemmPath::kTile128;
}

constexpr int kGemvWaves = 2048;

// Rows per tile: 128 (4 waves) up to 128-row batches, 256 (8 waves) beyond,
// so W is read once per step for batches up to 256.
int tile_rows(int M) { return M <= 128 ? 128 : 256; }

int gemm_plan_splits(int dtype, int M, int N, int K, int* k_split) {
  const int kq = (dtype == 1) ? 64 : 16;
  if (dtype == 1 && bf16_path(M, K) == GemmPath::kGemv) {
    *k_split = K;
    return 1;
  }
  const bool tile = dtype == 1 && bf16_path(M, K) == GemmPath::kTile128;
  const int mblk = (dtype == 1) ? (tile ? tile_rows(M) : 64) : 32;
  const int nblk = tile ? 128 : 64;
  const int64_t tiles = (int64_t)((N + nblk - 1) / nblk) * ((M + mblk - 1) / mblk);
  // Small batches: aim for two work groups per CU; the partial sums are
  // small.  Larger batches: about one per CU, since every extra split writes
  // and re-reads an M x N fp32 slab; the 256-row tile holds a whole CU.
  const int64_t target = !tile || M <= 64 ? 512 : (M <= 128 ? 256 : 224);
  const int ksteps = (K + kq - 1) / kq;
  int s = 1;
  if (tiles < target) s = (int)std::min<int64_t>((target + tiles - 1) / tiles, 8);
  s = std::max(1, std::min(s, ksteps));
  const int steps_per = (ksteps + s - 1) / s;
  *k_split = steps_per * kq;
  return (K + *k_split - 1) / *k_split;
}

hipError_t launch_gemm(int dtype, int M, int N, int K, const void* A, int64_t lda,
                       const WSegs& w, float* out, int splits, int k_split, hipStream_t stream) {
  if (M <= 0 || N <= 0) return hipSuccess;
  const dim3 block(256);
  if (dtype == 1) {
    const uint16_t* a = (const uint16_t*)A;
    const GemmPath path = bf16_path(M, K);
    if (path == GemmPath::kGemv) {
      const int rpw = (N + kGemvWaves - 1) / kGemvWaves;
      const dim3 grid((N + 4 * rpw - 1) / (4 * rpw));
      const size_t lds = (size_t)M * K * 2;
      switch (M) {
        case 1: gemv_bf16<1><<<grid, block, lds, stream>>>(N, K, rpw, a, lda, w, out); break;
        case 2: gemv_bf16<2><<<grid, block, lds, stream>>>(N, K, rpw, a, lda, w, out); break;
        case 3: gemv_bf16<3><<<grid, block, lds, stream>>>(N, K, rpw, a, lda, w, out); break;
        default: gemv_bf16<4><<<grid, block, lds, stream>>>(N, K, rpw, a, lda, w, out); break;
      }
    } else if (path == GemmPath::kSmallM) {
      const dim3 grid((N + 63) / 64, 1, splits);
      switch ((M + 15) / 16) {
        case 1: gemm_bf16_small_m<1, 8><<<grid, block, 0, stream>>>(M, N, K, k_split, a, lda, w, out); break;
        case 2: gemm_bf16_small_m<2, 8><<<grid, block, 0, stream>>>(M, N, K, k_split, a, lda, w, out); break;
        case 3: gemm_bf16_small_m<3, 8><<<grid, block, 0, stream>>>(M, N, K, k_split, a, lda, w, out); break;
        default: gemm_bf16_small_m<4, 8><<<grid, block, 0, stream>>>(M, N, K, k_split, a, lda, w, out); break;
      }
    } else {
      const int rows = tile_rows(M);
      const int n_mb = (M + rows - 1) / rows, n_nb = (N + 127) / 128;
      const dim3 grid(((n_nb + 7) / 8) * 8 * n_mb, 1, splits);
      if (rows == 128)
        gemm_bf16_tile<2, 2, 2><<<grid, dim3(256), 0, stream>>>(M, N, K, k_split, n_mb, n_nb, a,
                                                               lda, w, out);
      else
        gemm_bf16_tile<4, 2, 2><<<grid, dim3(512), 0, stream>>>(M, N, K, k_split, n_mb, n_nb, a,
                                                               lda, w, out);
    }
  } else {
    const dim3 grid((N + 63) / 64, (M + 31) / 32, splits);
    gemm_f32_tiled<<<grid, block, 0, stream>>>(M, N, K, k_split, (const float*)A, lda, w, out);
  }
  return hipGetLastError();
}

}  // namespace pdec

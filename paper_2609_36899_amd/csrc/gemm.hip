// Weight-streaming projections: out[s][m][n] = sum_{k in split s} A[m][k] W[n][k].
//
// Each decode step reads the weights once for the whole active batch (paper:
// Introduction; Design Principles, "Specialization in Heterogeneous Pools").
// A work group owns a 64-column slice of W and every row of the batch, so W
// is streamed from HBM exactly once per step; the activations (at most a few
// MB) stay in L2.  When the column slices alone cannot fill 256 CUs the K
// axis is split and the fp32 partial sums are reduced by the next kernel.
//
// bf16: v_mfma_f32_16x16x32_bf16 tiles of 16 rows x 16 columns, four waves
// per work group arranged WM x WN over the (rows, columns) tile.
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

template <int WM, int WN, int MT, int NT>
__global__ __launch_bounds__(256) void gemm_bf16_mfma(int M, int N, int K, int k_split,
                                                      const uint16_t* __restrict__ A,
                                                      int64_t lda, WSegs w,
                                                      float* __restrict__ out) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c16 = lane & 15, q4 = lane >> 4;
  const int wm = wave / WN, wn = wave % WN;
  const int m0 = blockIdx.y * (WM * MT * 16) + wm * MT * 16;
  const int n0 = blockIdx.x * (WN * NT * 16) + wn * NT * 16;
  const int kbeg = blockIdx.z * k_split;
  const int kend = min(K, kbeg + k_split);
  if (m0 >= M || n0 >= N) return;  // no barriers below: idle waves may leave

  const uint16_t* arow[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) arow[t] = A + (int64_t)min(m0 + t * 16 + c16, M - 1) * lda + q4 * 8;
  const uint16_t* wrow[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
    wrow[t] = (const uint16_t*)seg_row(w, min(n0 + t * 16 + c16, N - 1), K, 2) + q4 * 8;

  f32x4 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int k = kbeg; k < kend; k += 64) {
    bf16x8 a0[MT], a1[MT], b0[NT], b1[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      b0[j] = *(const bf16x8*)(wrow[j] + k);
      b1[j] = *(const bf16x8*)(wrow[j] + k + 32);
    }
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      a0[i] = *(const bf16x8*)(arow[i] + k);
      a1[i] = *(const bf16x8*)(arow[i] + k + 32);
    }
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0[i], b0[j], acc[i][j], 0, 0, 0);
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1[i], b1[j], acc[i][j], 0, 0, 0);
      }
  }

  float* o = out + (int64_t)blockIdx.z * M * N;
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const int col = n0 + j * 16 + c16;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int row = m0 + i * 16 + 4 * q4 + rr;
        if (row < M && col < N) o[(int64_t)row * N + col] = acc[i][j][rr];
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

struct BfCfg {
  int mblk;
};

BfCfg bf_cfg(int M) {
  if (M <= 16) return {16};
  if (M <= 32) return {32};
  if (M <= 64) return {64};
  if (M <= 128) return {128};
  if (M <= 256) return {256};
  return {512};
}

}  // namespace

int gemm_plan_splits(int dtype, int M, int N, int K, int* k_split) {
  const int kq = (dtype == 1) ? 64 : 16;
  const int mblk = (dtype == 1) ? bf_cfg(M).mblk : 32;
  const int64_t tiles = (int64_t)((N + 63) / 64) * ((M + mblk - 1) / mblk);
  const int ksteps = (K + kq - 1) / kq;
  int s = 1;
  if (tiles < 512) s = (int)std::min<int64_t>((512 + tiles - 1) / tiles, 8);
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
    const int mblk = bf_cfg(M).mblk;
    const dim3 grid((N + 63) / 64, (M + mblk - 1) / mblk, splits);
    const uint16_t* a = (const uint16_t*)A;
    switch (mblk) {
      case 16: gemm_bf16_mfma<1, 4, 1, 1><<<grid, block, 0, stream>>>(M, N, K, k_split, a, lda, w, out); break;
      case 32: gemm_bf16_mfma<1, 4, 2, 1><<<grid, block, 0, stream>>>(M, N, K, k_split, a, lda, w, out); break;
      case 64: gemm_bf16_mfma<1, 4, 4, 1><<<grid, block, 0, stream>>>(M, N, K, k_split, a, lda, w, out); break;
      case 128: gemm_bf16_mfma<2, 2, 4, 2><<<grid, block, 0, stream>>>(M, N, K, k_split, a, lda, w, out); break;
      case 256: gemm_bf16_mfma<4, 1, 4, 4><<<grid, block, 0, stream>>>(M, N, K, k_split, a, lda, w, out); break;
      default: gemm_bf16_mfma<4, 1, 8, 4><<<grid, block, 0, stream>>>(M, N, K, k_split, a, lda, w, out); break;
    }
  } else {
    const dim3 grid((N + 63) / 64, (M + 31) / 32, splits);
    gemm_f32_tiled<<<grid, block, 0, stream>>>(M, N, K, k_split, (const float*)A, lda, w, out);
  }
  return hipGetLastError();
}

}  // namespace pdec

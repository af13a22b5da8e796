// Per-row and elementwise steps of the decoder layer, each fused with the
// reduction of the preceding projection's split-K partial sums:
//   embedding gather + RMSNorm, residual add + RMSNorm, q/k rotary embedding
//   + KV page write, SwiGLU, greedy argmax, block-table updates and the
//   rotary cos/sin table.
#include "hip_common.h"
#include "kernels.h"

namespace pdec {

namespace {

constexpr int kRowThreads = 256;

// Token ids from the caller's device buffer cannot be checked on the host
// without a synchronisation; out-of-range ids are clamped so that they read
// a valid embedding row instead of faulting.
template <typename WT, typename HT>
__global__ __launch_bounds__(kRowThreads) void embed_norm_kernel(
    int d, int vocab, const int32_t* __restrict__ tokens, const WT* __restrict__ embed,
    const float* __restrict__ gain, float eps, float* __restrict__ x, HT* __restrict__ h) {
  __shared__ float red[kRowThreads / 64];
  const int row = blockIdx.x;
  const int tok = min(max(tokens[row], 0), vocab - 1);
  const WT* e = embed + (int64_t)tok * d;
  float* xr = x + (int64_t)row * d;
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += kRowThreads) {
    const float v = Store<WT>::load(e + i);
    xr[i] = v;
    ss += v * v;
  }
  const float inv = rsqrtf(block_sum(ss, red) / (float)d + eps);
  HT* hr = h + (int64_t)row * d;
  for (int i = threadIdx.x; i < d; i += kRowThreads)
    hr[i] = Store<HT>::from(xr[i] * inv * gain[i]);
}

template <typename HT>
__global__ __launch_bounds__(kRowThreads) void resid_norm_kernel(
    int M, int d, const float* __restrict__ part, int splits, float* __restrict__ x,
    const float* __restrict__ gain, float eps, HT* __restrict__ h) {
  __shared__ float red[kRowThreads / 64];
  const int row = blockIdx.x;
  float* xr = x + (int64_t)row * d;
  const int64_t slab = (int64_t)M * d;
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += kRowThreads) {
    float v = xr[i];
    for (int s = 0; s < splits; ++s) v += part[s * slab + (int64_t)row * d + i];
    xr[i] = v;
    ss += v * v;
  }
  const float inv = rsqrtf(block_sum(ss, red) / (float)d + eps);
  HT* hr = h + (int64_t)row * d;
  for (int i = threadIdx.x; i < d; i += kRowThreads)
    hr[i] = Store<HT>::from(xr[i] * inv * gain[i]);
}

// One work group per row.  Pairs (i, i + Dh/2) of every q and k head are
// rotated by the table angle of the row's position; v is copied.  K goes to
// [page][g][slot][Dh], V to the transposed block [page][g][Dh][slot].
template <typename T>
__global__ __launch_bounds__(kRowThreads) void qkv_rope_kv_kernel(
    int M, int head_dim, int n_q_heads, int n_kv_heads, const float* __restrict__ part,
    int splits, const RowMeta* __restrict__ rows, const float2* __restrict__ rope_cs,
    const int32_t* __restrict__ bt, int32_t bt_stride, T* __restrict__ q_out,
    T* __restrict__ kpool, T* __restrict__ vpool, int64_t page_stride) {
  const int row = blockIdx.x;
  const RowMeta rm = rows[row];
  const int half = head_dim / 2;
  const int ncols = (n_q_heads + 2 * n_kv_heads) * head_dim;
  const int64_t slab = (int64_t)M * ncols;
  const float* pr = part + (int64_t)row * ncols;
  const int page = bt[(int64_t)rm.slot * bt_stride + rm.pos / kPage];
  const int slot = rm.pos % kPage;
  const int64_t page_base = (int64_t)page * page_stride;
  const float2* cs = rope_cs + (int64_t)rm.pos * half;

  const int n_pairs = (n_q_heads + n_kv_heads) * half;
  for (int p = threadIdx.x; p < n_pairs; p += kRowThreads) {
    const int hh = p / half, i = p % half;
    const int c0 = hh * head_dim + i, c1 = c0 + half;
    float a = 0.f, b = 0.f;
    for (int s = 0; s < splits; ++s) {
      a += pr[s * slab + c0];
      b += pr[s * slab + c1];
    }
    const float2 t = cs[i];
    const float ra = a * t.x - b * t.y;
    const float rb = a * t.y + b * t.x;
    if (hh < n_q_heads) {
      T* qr = q_out + ((int64_t)row * n_q_heads + hh) * head_dim;
      qr[i] = Store<T>::from(ra);
      qr[i + half] = Store<T>::from(rb);
    } else {
      T* kr = kpool + page_base + ((int64_t)(hh - n_q_heads) * kPage + slot) * head_dim;
      kr[i] = Store<T>::from(ra);
      kr[i + half] = Store<T>::from(rb);
    }
  }
  const int vcol0 = (n_q_heads + n_kv_heads) * head_dim;
  for (int idx = threadIdx.x; idx < n_kv_heads * head_dim; idx += kRowThreads) {
    float v = 0.f;
    for (int s = 0; s < splits; ++s) v += pr[s * slab + vcol0 + idx];
    const int g = idx / head_dim, dd = idx % head_dim;
    vpool[page_base + ((int64_t)g * head_dim + dd) * kPage + slot] = Store<T>::from(v);
  }
}

template <typename HT>
__global__ __launch_bounds__(256) void swiglu_kernel(int M, int F, const float* __restrict__ part,
                                                     int splits, HT* __restrict__ u) {
  const int64_t n = (int64_t)M * F;
  const int64_t slab = (int64_t)M * 2 * F;
  for (int64_t idx = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; idx < n;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t m = idx / F, c = idx % F;
    float gt = 0.f, up = 0.f;
    for (int s = 0; s < splits; ++s) {
      gt += part[s * slab + m * 2 * F + c];
      up += part[s * slab + m * 2 * F + F + c];
    }
    u[idx] = Store<HT>::from(gt / (1.f + expf(-gt)) * up);
  }
}

__global__ __launch_bounds__(256) void argmax_kernel(int V, const float* __restrict__ logits,
                                                     int32_t* __restrict__ tokens) {
  __shared__ float sv[256];
  __shared__ int si[256];
  const float* lr = logits + (int64_t)blockIdx.x * V;
  float best = -INFINITY;
  int bi = 0x7FFFFFFF;
  for (int i = threadIdx.x; i < V; i += 256) {
    const float v = lr[i];
    if (v > best) {  // strict: the first (lowest) index wins within a thread
      best = v;
      bi = i;
    }
  }
  sv[threadIdx.x] = best;
  si[threadIdx.x] = bi;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) {
      const float v2 = sv[threadIdx.x + o];
      const int i2 = si[threadIdx.x + o];
      if (v2 > sv[threadIdx.x] || (v2 == sv[threadIdx.x] && i2 < si[threadIdx.x])) {
        sv[threadIdx.x] = v2;
        si[threadIdx.x] = i2;
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) tokens[blockIdx.x] = (si[0] == 0x7FFFFFFF) ? 0 : si[0];
}

__global__ void bt_deltas_kernel(int n, const BtDelta* __restrict__ d, int32_t* __restrict__ bt,
                                 int32_t stride) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) bt[(int64_t)d[i].slot * stride + d[i].idx] = d[i].page;
}

__global__ void rope_table_kernel(int max_pos, int half, double base, float2* __restrict__ cs) {
  const int64_t n = (int64_t)max_pos * half;
  for (int64_t idx = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; idx < n;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t p = idx / half;
    const int i = (int)(idx % half);
    const double ang = (double)p * pow(base, -2.0 * (double)i / (double)(2 * half));
    cs[idx] = make_float2((float)cos(ang), (float)sin(ang));
  }
}

inline int grid_for(int64_t n, int block) {
  return (int)std::min<int64_t>((n + block - 1) / block, 65536);
}

}  // namespace

hipError_t launch_embed_norm(int dtype, int M, int d, int vocab, const int32_t* tokens,
                             const void* embed,
                             const float* gain, float eps, float* x, void* h, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  if (dtype == 1)
    embed_norm_kernel<uint16_t, uint16_t><<<M, kRowThreads, 0, stream>>>(
        d, vocab, tokens, (const uint16_t*)embed, gain, eps, x, (uint16_t*)h);
  else
    embed_norm_kernel<float, float><<<M, kRowThreads, 0, stream>>>(
        d, vocab, tokens, (const float*)embed, gain, eps, x, (float*)h);
  return hipGetLastError();
}

hipError_t launch_resid_norm(int dtype, int M, int d, const float* part, int splits, float* x,
                             const float* gain, float eps, void* h, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  if (dtype == 1)
    resid_norm_kernel<uint16_t><<<M, kRowThreads, 0, stream>>>(M, d, part, splits, x, gain, eps,
                                                               (uint16_t*)h);
  else
    resid_norm_kernel<float><<<M, kRowThreads, 0, stream>>>(M, d, part, splits, x, gain, eps,
                                                            (float*)h);
  return hipGetLastError();
}

hipError_t launch_qkv_rope_kv(int dtype, int M, int head_dim, int n_q_heads, int n_kv_heads,
                              const float* part, int splits, const RowMeta* rows,
                              const float2* rope_cs, const int32_t* block_table, int32_t bt_stride,
                              void* q_out, void* k_pages, void* v_pages, int64_t page_stride_elems,
                              hipStream_t stream) {
  if (M == 0) return hipSuccess;
  if (dtype == 1)
    qkv_rope_kv_kernel<uint16_t><<<M, kRowThreads, 0, stream>>>(
        M, head_dim, n_q_heads, n_kv_heads, part, splits, rows, rope_cs, block_table, bt_stride,
        (uint16_t*)q_out, (uint16_t*)k_pages, (uint16_t*)v_pages, page_stride_elems);
  else
    qkv_rope_kv_kernel<float><<<M, kRowThreads, 0, stream>>>(
        M, head_dim, n_q_heads, n_kv_heads, part, splits, rows, rope_cs, block_table, bt_stride,
        (float*)q_out, (float*)k_pages, (float*)v_pages, page_stride_elems);
  return hipGetLastError();
}

hipError_t launch_swiglu(int dtype, int M, int F, const float* part, int splits, void* u,
                         hipStream_t stream) {
  const int64_t n = (int64_t)M * F;
  if (n == 0) return hipSuccess;
  if (dtype == 1)
    swiglu_kernel<uint16_t><<<grid_for(n, 256), 256, 0, stream>>>(M, F, part, splits,
                                                                   (uint16_t*)u);
  else
    swiglu_kernel<float><<<grid_for(n, 256), 256, 0, stream>>>(M, F, part, splits, (float*)u);
  return hipGetLastError();
}

hipError_t launch_argmax(int B, int V, const float* logits, int32_t* tokens, hipStream_t stream) {
  if (B == 0) return hipSuccess;
  argmax_kernel<<<B, 256, 0, stream>>>(V, logits, tokens);
  return hipGetLastError();
}

hipError_t launch_bt_deltas(int n, const BtDelta* deltas, int32_t* bt, int32_t stride,
                            hipStream_t stream) {
  if (n == 0) return hipSuccess;
  bt_deltas_kernel<<<(n + 255) / 256, 256, 0, stream>>>(n, deltas, bt, stride);
  return hipGetLastError();
}

hipError_t launch_rope_table(int max_pos, int head_dim, double base, float2* cs,
                             hipStream_t stream) {
  const int64_t n = (int64_t)max_pos * (head_dim / 2);
  if (n == 0) return hipSuccess;
  rope_table_kernel<<<grid_for(n, 256), 256, 0, stream>>>(max_pos, head_dim / 2, base, cs);
  return hipGetLastError();
}

}  // namespace pdec

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

// Split-K partials: partial s of element i is at p[s * slab + i].  These add
// v + p[0] + p[slab] + ... + p[(n - 1) slab] in that order, with the loads of
// up to eight splits issued together so that their latencies overlap.
__device__ __forceinline__ float4 add_splits4(float4 v, const float* p, int64_t slab, int n) {
  for (int s0 = 0; s0 < n; s0 += 8) {
    float4 t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (s0 + u < n) t[u] = *(const float4*)(p + (int64_t)(s0 + u) * slab);
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (s0 + u < n) {
        v.x += t[u].x;
        v.y += t[u].y;
        v.z += t[u].z;
        v.w += t[u].w;
      }
  }
  return v;
}

__device__ __forceinline__ float add_splits1(float v, const float* p, int64_t slab, int n) {
  for (int s0 = 0; s0 < n; s0 += 8) {
    float t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (s0 + u < n) t[u] = p[(int64_t)(s0 + u) * slab];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (s0 + u < n) v += t[u];
  }
  return v;
}

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
struct Pack4;
template <>
struct Pack4<float> {
  static __device__ __forceinline__ void store(float* p, float4 v) { *(float4*)p = v; }
};
template <>
struct Pack4<uint16_t> {
  static __device__ __forceinline__ void store(uint16_t* p, float4 v) {
    const uint32_t lo = (uint32_t)f32_to_bf16(v.x) | ((uint32_t)f32_to_bf16(v.y) << 16);
    const uint32_t hi = (uint32_t)f32_to_bf16(v.z) | ((uint32_t)f32_to_bf16(v.w) << 16);
    *(uint2*)p = make_uint2(lo, hi);
  }
};

// KV page stores: bf16 / fp32 as above; fp8 pages hold E4M3 codes of x / scale.
template <typename T>
struct KvStore {
  static __device__ __forceinline__ void store4(T* p, float4 v, float) { Pack4<T>::store(p, v); }
  static __device__ __forceinline__ T one(float v, float) { return Store<T>::from(v); }
};
template <>
struct KvStore<uint8_t> {
  static __device__ __forceinline__ void store4(uint8_t* p, float4 v, float scale) {
    *(uint32_t*)p = e4m3_from_f32(v.x / scale) | (e4m3_from_f32(v.y / scale) << 8) |
                    (e4m3_from_f32(v.z / scale) << 16) | (e4m3_from_f32(v.w / scale) << 24);
  }
  static __device__ __forceinline__ uint8_t one(float v, float scale) {
    return (uint8_t)e4m3_from_f32(v / scale);
  }
};

// One work group of up to 1024 threads per row, float4 accesses (d % 4 == 0).
template <typename HT>
__global__ __launch_bounds__(1024) void resid_norm_kernel(
    int M, int d, const float* __restrict__ part, int splits, float* __restrict__ x,
    const float* __restrict__ gain, float eps, HT* __restrict__ h) {
  constexpr int RC = 4;  // float4s per thread kept in registers between the passes
  __shared__ float red[16];
  const int row = blockIdx.x;
  float* xr = x + (int64_t)row * d;
  const int64_t slab = (int64_t)M * d;
  const float* pr = part + (int64_t)row * d;
  const int stride = blockDim.x * 4;
  float4 keep[RC];
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < RC; ++k) {
    const int i = threadIdx.x * 4 + k * stride;
    if (i < d) {
      const float4 v = add_splits4(*(const float4*)(xr + i), pr + i, slab, splits);
      *(float4*)(xr + i) = v;
      keep[k] = v;
      ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
    }
  }
  for (int i = threadIdx.x * 4 + RC * stride; i < d; i += stride) {  // rows wider than kept
    const float4 v = add_splits4(*(const float4*)(xr + i), pr + i, slab, splits);
    *(float4*)(xr + i) = v;
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  const float inv = rsqrtf(block_sum(ss, red) / (float)d + eps);
  HT* hr = h + (int64_t)row * d;
  auto put = [&](int i, float4 v) {
    const float4 g = *(const float4*)(gain + i);
    Pack4<HT>::store(hr + i, make_float4(v.x * inv * g.x, v.y * inv * g.y, v.z * inv * g.z,
                                         v.w * inv * g.w));
  };
#pragma unroll
  for (int k = 0; k < RC; ++k) {
    const int i = threadIdx.x * 4 + k * stride;
    if (i < d) put(i, keep[k]);
  }
  for (int i = threadIdx.x * 4 + RC * stride; i < d; i += stride) put(i, *(const float4*)(xr + i));
}

// A row is handled by gridDim.y work groups.  Pairs (i, i + Dh/2) of every q and k head are
// rotated by the table angle of the row's position, four pairs per thread;
// v is copied.  KV pages take the element type KVT (fp8 pages store codes of
// k / k_scale and v / v_scale).  With q/k gains (the Qwen3 family's per-head norm), each q and
// k head is first RMS-normalised over Dh: the Dh/8 threads of a head are
// consecutive, aligned lanes, and reduce their sum of squares by shuffles.  K goes to [page][g][slot][Dh], V to the transposed block
// [page][g][Dh][slot].
template <typename T, typename KVT>
__global__ __launch_bounds__(kRowThreads) void qkv_rope_kv_kernel(
    int M, int head_dim, int n_q_heads, int n_kv_heads, const float* __restrict__ part,
    int splits, const RowMeta* __restrict__ rows, const float2* __restrict__ rope_cs,
    const int32_t* __restrict__ bt, int32_t bt_stride, T* __restrict__ q_out,
    KVT* __restrict__ kpool, KVT* __restrict__ vpool, int64_t page_stride,
    const float* __restrict__ q_gain, const float* __restrict__ k_gain, float eps,
    float k_scale, float v_scale) {
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

  // blockIdx.y splits the row's work across gridDim.y groups.
  const int part_id = blockIdx.y, n_parts = gridDim.y;
  const int quads_per_head = half / 4;
  const int n_quads = (n_q_heads + n_kv_heads) * quads_per_head;
  for (int qd = part_id * kRowThreads + threadIdx.x; qd < n_quads; qd += n_parts * kRowThreads) {
    const int hh = qd / quads_per_head, i = (qd % quads_per_head) * 4;
    const int c0 = hh * head_dim + i, c1 = c0 + half;
    float4 a = add_splits4(*(const float4*)(pr + c0), pr + slab + c0, slab, splits - 1);
    float4 b = add_splits4(*(const float4*)(pr + c1), pr + slab + c1, slab, splits - 1);
    if (q_gain) {
      // All quads_per_head lanes of this head run this iteration together
      // (heads are whole, aligned lane groups and n_quads is a multiple).
      float ss = a.x * a.x + a.y * a.y + a.z * a.z + a.w * a.w + b.x * b.x + b.y * b.y +
                 b.z * b.z + b.w * b.w;
      for (int off = quads_per_head / 2; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);
      const float r = rsqrtf(ss / (float)head_dim + eps);
      const float* gn = hh < n_q_heads ? q_gain : k_gain;
      const float4 ga = *(const float4*)(gn + i), gb = *(const float4*)(gn + i + half);
      a = make_float4(a.x * r * ga.x, a.y * r * ga.y, a.z * r * ga.z, a.w * r * ga.w);
      b = make_float4(b.x * r * gb.x, b.y * r * gb.y, b.z * r * gb.z, b.w * r * gb.w);
    }
    const float4 t01 = *(const float4*)(cs + i), t23 = *(const float4*)(cs + i + 2);
    const float4 ra = make_float4(a.x * t01.x - b.x * t01.y, a.y * t01.z - b.y * t01.w,
                                  a.z * t23.x - b.z * t23.y, a.w * t23.z - b.w * t23.w);
    const float4 rb = make_float4(a.x * t01.y + b.x * t01.x, a.y * t01.w + b.y * t01.z,
                                  a.z * t23.y + b.z * t23.x, a.w * t23.w + b.w * t23.z);
    if (hh < n_q_heads) {
      T* dst = q_out + ((int64_t)row * n_q_heads + hh) * head_dim;
      Pack4<T>::store(dst + i, ra);
      Pack4<T>::store(dst + i + half, rb);
    } else {
      KVT* dst = kpool + page_base + ((int64_t)(hh - n_q_heads) * kPage + slot) * head_dim;
      KvStore<KVT>::store4(dst + i, ra, k_scale);
      KvStore<KVT>::store4(dst + i + half, rb, k_scale);
    }
  }
  const int vcol0 = (n_q_heads + n_kv_heads) * head_dim;
  for (int idx = part_id * kRowThreads + threadIdx.x; idx < n_kv_heads * head_dim;
       idx += n_parts * kRowThreads) {
    const float v = add_splits1(0.f, pr + vcol0 + idx, slab, splits);
    const int g = idx / head_dim, dd = idx % head_dim;
    vpool[page_base + ((int64_t)g * head_dim + dd) * kPage + slot] = KvStore<KVT>::one(v, v_scale);
  }
}

// Four columns per thread (F % 4 == 0); row m of u starts at u + m * ldu.
template <typename HT>
__global__ __launch_bounds__(256) void swiglu_kernel(int M, int F, const float* __restrict__ part,
                                                     int splits, HT* __restrict__ u,
                                                     int64_t ldu) {
  const int64_t n4 = (int64_t)M * F / 4;
  const int64_t slab = (int64_t)M * 2 * F;
  for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < n4;
       q += (int64_t)gridDim.x * blockDim.x) {
    const int64_t idx = q * 4;
    const int64_t m = idx / F, c = idx % F;
    const float* pg = part + m * 2 * F + c;
    const float4 gt = add_splits4(*(const float4*)pg, pg + slab, slab, splits - 1);
    const float4 up = add_splits4(*(const float4*)(pg + F), pg + slab + F, slab, splits - 1);
    const float4 r = make_float4(gt.x / (1.f + expf(-gt.x)) * up.x, gt.y / (1.f + expf(-gt.y)) * up.y,
                                 gt.z / (1.f + expf(-gt.z)) * up.z, gt.w / (1.f + expf(-gt.w)) * up.w);
    Pack4<HT>::store(u + m * ldu + c, r);
  }
}

// out[i] = sum_s part[s][i] in split order (float4; n % 4 == 0).
__global__ __launch_bounds__(256) void sum_splits_kernel(int64_t n4, const float* __restrict__ part,
                                                         int splits, float* __restrict__ out) {
  for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < n4;
       q += (int64_t)gridDim.x * blockDim.x) {
    const float4 v =
        add_splits4(*(const float4*)(part + q * 4), part + n4 * 4 + q * 4, n4 * 4, splits - 1);
    *(float4*)(out + q * 4) = v;
  }
}

// One work group per row, 4-byte words.
__global__ __launch_bounds__(256) void gather_rows_kernel(const int32_t* __restrict__ idx,
                                                          const uint32_t* __restrict__ src,
                                                          int64_t row_words,
                                                          uint32_t* __restrict__ dst) {
  const uint32_t* s = src + (int64_t)idx[blockIdx.x] * row_words;
  uint32_t* d = dst + (int64_t)blockIdx.x * row_words;
  for (int64_t i = threadIdx.x; i < row_words; i += 256) d[i] = s[i];
}

__device__ __forceinline__ void argmax_merge(float& v, int& i, float v2, int i2) {
  if (v2 > v || (v2 == v && i2 < i)) {
    v = v2;
    i = i2;
  }
}

// One work group of 1024 threads per row.  Ties go to the lowest index.
__global__ __launch_bounds__(1024) void argmax_kernel(int V, const float* __restrict__ logits,
                                                      int32_t* __restrict__ tokens) {
  __shared__ float sv[16];
  __shared__ int si[16];
  const float* lr = logits + (int64_t)blockIdx.x * V;
  float best = -INFINITY;
  int bi = 0x7FFFFFFF;
  const int v4 = (((uintptr_t)lr & 15) == 0) ? V / 4 : 0;
  for (int q = threadIdx.x; q < v4; q += 1024) {
    const float4 v = *(const float4*)(lr + q * 4);
    argmax_merge(best, bi, v.x, q * 4);
    argmax_merge(best, bi, v.y, q * 4 + 1);
    argmax_merge(best, bi, v.z, q * 4 + 2);
    argmax_merge(best, bi, v.w, q * 4 + 3);
  }
  for (int i = v4 * 4 + threadIdx.x; i < V; i += 1024) argmax_merge(best, bi, lr[i], i);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float v2 = __shfl_xor(best, o, 64);
    const int i2 = __shfl_xor(bi, o, 64);
    argmax_merge(best, bi, v2, i2);
  }
  if ((threadIdx.x & 63) == 0) {
    sv[threadIdx.x >> 6] = best;
    si[threadIdx.x >> 6] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 16; ++w) argmax_merge(best, bi, sv[w], si[w]);
    tokens[blockIdx.x] = (bi == 0x7FFFFFFF) ? 0 : bi;
  }
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
  const int threads = std::max(64, std::min(1024, (d / 4 + 63) / 64 * 64));
  if (dtype == 1)
    resid_norm_kernel<uint16_t><<<M, threads, 0, stream>>>(M, d, part, splits, x, gain, eps,
                                                           (uint16_t*)h);
  else
    resid_norm_kernel<float><<<M, threads, 0, stream>>>(M, d, part, splits, x, gain, eps,
                                                        (float*)h);
  return hipGetLastError();
}

hipError_t launch_qkv_rope_kv(int dtype, int kv_fp8, float k_scale, float v_scale, int M,
                              int head_dim, int n_q_heads, int n_kv_heads, const float* part,
                              int splits, const RowMeta* rows, const float2* rope_cs,
                              const int32_t* block_table, int32_t bt_stride, void* q_out,
                              void* k_pages, void* v_pages, int64_t page_stride_elems,
                              const float* q_gain, const float* k_gain, float eps,
                              hipStream_t stream) {
  if (M == 0) return hipSuccess;
  // Enough groups per row that every thread has at most one (q or k) quad,
  // so no group runs a second, mostly idle pass; small batches take more
  // groups per row to fill the GPU.
  const int n_quads = (n_q_heads + n_kv_heads) * (head_dim / 8);
  const dim3 grid(M, std::max(M >= 64 ? 2 : 8, (n_quads + kRowThreads - 1) / kRowThreads));
#define PDEC_QKV(T_, KVT_)                                                                   \
  qkv_rope_kv_kernel<T_, KVT_><<<grid, kRowThreads, 0, stream>>>(                             \
      M, head_dim, n_q_heads, n_kv_heads, part, splits, rows, rope_cs, block_table, bt_stride, \
      (T_*)q_out, (KVT_*)k_pages, (KVT_*)v_pages, page_stride_elems, q_gain, k_gain, eps,     \
      k_scale, v_scale)
  if (dtype == 1 && kv_fp8)
    PDEC_QKV(uint16_t, uint8_t);
  else if (dtype == 1)
    PDEC_QKV(uint16_t, uint16_t);
  else
    PDEC_QKV(float, float);
#undef PDEC_QKV
  return hipGetLastError();
}

hipError_t launch_swiglu(int dtype, int M, int F, const float* part, int splits, void* u,
                         hipStream_t stream, int64_t ldu) {
  const int64_t n = (int64_t)M * F / 4;
  if (n == 0) return hipSuccess;
  if (ldu == 0) ldu = F;
  if (dtype == 1)
    swiglu_kernel<uint16_t><<<grid_for(n, 256), 256, 0, stream>>>(M, F, part, splits,
                                                                   (uint16_t*)u, ldu);
  else
    swiglu_kernel<float><<<grid_for(n, 256), 256, 0, stream>>>(M, F, part, splits, (float*)u,
                                                                ldu);
  return hipGetLastError();
}

hipError_t launch_sum_splits(int64_t n, const float* part, int splits, float* out,
                             hipStream_t stream) {
  if (n == 0) return hipSuccess;
  sum_splits_kernel<<<grid_for(n / 4, 256), 256, 0, stream>>>(n / 4, part, splits, out);
  return hipGetLastError();
}

hipError_t launch_gather_rows(int n, const int32_t* idx, const void* src, int64_t row_bytes,
                              void* dst, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  gather_rows_kernel<<<n, 256, 0, stream>>>(idx, (const uint32_t*)src, row_bytes / 4,
                                            (uint32_t*)dst);
  return hipGetLastError();
}

hipError_t launch_argmax(int B, int V, const float* logits, int32_t* tokens, hipStream_t stream) {
  if (B == 0) return hipSuccess;
  argmax_kernel<<<B, 1024, 0, stream>>>(V, logits, tokens);
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

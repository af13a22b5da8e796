// Device-side helpers shared by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pdec {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Streaming loads of data read exactly once per step (KV pages, weight
// tiles): the non-temporal hint keeps them from displacing reused lines.
template <typename V>
__device__ __forceinline__ V load_stream(const void* p) {
  const u32x4 v = __builtin_nontemporal_load((const u32x4*)p);
  return __builtin_bit_cast(V, v);
}

// bf16 storage is handled as raw 16-bit patterns.
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

// Round-to-nearest-even float -> bf16 bits (inputs here are finite or inf).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename T>
struct Store;
template <>
struct Store<float> {
  static __device__ __forceinline__ float from(float v) { return v; }
  static __device__ __forceinline__ float load(const float* p) { return *p; }
};
template <>
struct Store<uint16_t> {
  static __device__ __forceinline__ uint16_t from(float v) { return f32_to_bf16(v); }
  static __device__ __forceinline__ float load(const uint16_t* p) { return bf16_to_f32(*p); }
};

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Sum over a work group of up to 1024 threads (multiple of 64).  `red` is
// __shared__ scratch of at least blockDim.x / 64 floats.  All threads get it.
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}

}  // namespace pdec

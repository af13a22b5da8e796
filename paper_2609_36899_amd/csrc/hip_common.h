// Device-side helpers shared by the gfx950 kernels.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fp8_e4m3.h"

namespace pdec {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Streaming loads of data read exactly once per step (KV pages, weight
// tiles): the non-temporal hint keeps them from displacing reused lines.
template <typename V>
__device__ __forceinline__ V load_stream(const void* p) {
  static_assert(sizeof(V) == 16 || sizeof(V) == 8, "16- or 8-byte loads");
  if constexpr (sizeof(V) == 16) {
    return __builtin_bit_cast(V, __builtin_nontemporal_load((const u32x4*)p));
  } else {
    return __builtin_bit_cast(V, __builtin_nontemporal_load((const u32x2*)p));
  }
}

// 16 bytes per lane from global memory straight into LDS (gfx950 LDS-DMA):
// lane i's bytes land at lds + 16 i, where lds is uniform over the wave.  The
// load counts in the vector-memory counter until its data is in LDS.
__device__ __forceinline__ void dma16(const void* src, void* lds) {
  __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                   (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}
// The same with the non-temporal hint (nt), for data read once per launch
// (streamed weights): it leaves the L2 to the operands that are re-read.
__device__ __forceinline__ void dma16_stream(const void* src, void* lds) {
  __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                   (__attribute__((address_space(3))) void*)lds, 16, 0, 2);
}

// Wait until at most N vector-memory operations of this wave are outstanding
// (loads retire in issue order), leaving the other counters alone.
template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 64, "vmcnt is six bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Wait until this wave's LDS (and scalar memory) operations have completed,
// leaving the vector-memory counter alone.
__device__ __forceinline__ void wait_lds() {
  __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));
}

// Work-group barrier without the fence of __syncthreads, whose release would
// wait for every load in flight (LDS-DMA loads included).  Callers order
// their memory with explicit counter waits; the empty asm statements keep
// the compiler from moving memory accesses across the barrier.
__device__ __forceinline__ void wg_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
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

// IEEE maximum: one v_maximum3_f32, with no canonicalising self-max on its
// inputs as fmaxf needs.  Callers pass finite scores or -inf (masked keys are
// set to -inf before any maximum, so no NaN reaches it).
__device__ __forceinline__ float max2(float a, float b) {
  return __builtin_elementwise_maximum(a, b);
}

// Maximum and sum over the four lanes l, l^16, l^32, l^48 (the four key
// groups of an MFMA score column) with the gfx950 cross-row swaps, which stay
// in the VALU: a __shfl_xor is an LDS permute, and its wait also drains every
// LDS read in flight.  Swapping a value with itself leaves 16-lane rows
// (0,0,2,2) in one result and (1,1,3,3) in the other, or 32-lane halves (0,0)
// and (1,1), so combining the two gives the xor-16 / xor-32 reduction; each
// lane adds the same two operands as the shuffle form (in swapped order), so
// the sum is bit-identical to it.
__device__ __forceinline__ float max_over_key_groups(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = max2(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return max2(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float sum_over_key_groups(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
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

// ---- fp8 (OCP E4M3FN) KV codes: e4m3_from_f32 in fp8_e4m3.h --------------

// Eight codes (two dwords, code i in byte i) to eight bf16 values: the
// hardware fp8 -> f32 conversion, then f32 -> bf16, both exact (every e4m3
// value is a bf16 value).
__device__ __forceinline__ bf16x8 e4m3x8_to_bf16(u32x2 w) {
  const f32x2 a = __builtin_amdgcn_cvt_pk_f32_fp8((int)w.x, false);
  const f32x2 b = __builtin_amdgcn_cvt_pk_f32_fp8((int)w.x, true);
  const f32x2 c = __builtin_amdgcn_cvt_pk_f32_fp8((int)w.y, false);
  const f32x2 d = __builtin_amdgcn_cvt_pk_f32_fp8((int)w.y, true);
  const bf16x2 pa = __builtin_convertvector(a, bf16x2), pb = __builtin_convertvector(b, bf16x2);
  const bf16x2 pc = __builtin_convertvector(c, bf16x2), pd = __builtin_convertvector(d, bf16x2);
  return bf16x8{pa[0], pa[1], pb[0], pb[1], pc[0], pc[1], pd[0], pd[1]};
}

// Launch on stream s.  With a start/stop event pair the dispatch itself
// records the kernel's begin and end (hipExtLaunchKernelGGL), so timing a
// launch adds no marker packets, and no gaps, between kernels.
template <typename... KArgs, typename... Args>
hipError_t launch_timed(void (*kernel)(KArgs...), dim3 grid, dim3 block, hipStream_t s,
                        hipEvent_t ev_start, hipEvent_t ev_stop, Args... args) {
  if (ev_start)
    hipExtLaunchKernelGGL(kernel, grid, block, 0, s, ev_start, ev_stop, 0, (KArgs)args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, s, (KArgs)args...);
  return hipGetLastError();
}

}  // namespace pdec

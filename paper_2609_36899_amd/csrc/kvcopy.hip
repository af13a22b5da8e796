// KV snapshot and restore: page gather to, and scatter from, pinned host memory.
//
// A trajectory that departs is snapshotted from device memory to host memory
// over PCIe, freeing its pages while the host copy keeps it available (paper:
// Design, "KV Preparation for Late-Bound Placement", phase 1).  The host copy
// is page-major, [page][layer][K|V][Hkv][16 * Dh], so any prefix range of
// pages is one contiguous byte range.  Each work group moves one
// (page, layer, K|V) block of Hkv * 16 * Dh elements with 16-byte accesses.
#include "hip_common.h"
#include "kernels.h"

namespace pdec {

namespace {

__global__ __launch_bounds__(256) void kv_page_copy_kernel(
    const int32_t* __restrict__ pages, int n_layers, int64_t n_pool_pages, int64_t block_bytes,
    char* __restrict__ pool, char* __restrict__ host, int to_host) {
  const int i = blockIdx.x;                 // page index within the sequence
  const int lk = blockIdx.y;                // layer * 2 + kind
  const int64_t dev_off = ((int64_t)lk * n_pool_pages + pages[i]) * block_bytes;
  const int64_t host_off = ((int64_t)i * n_layers * 2 + lk) * block_bytes;
  const int64_t n16 = block_bytes / 16;
  u32x4* d = (u32x4*)(pool + dev_off);
  u32x4* h = (u32x4*)(host + host_off);
  for (int64_t j = threadIdx.x; j < n16; j += 256) {
    if (to_host)
      h[j] = d[j];
    else
      d[j] = h[j];
  }
}

}  // namespace

hipError_t launch_kv_page_copy(int n_pages, const int32_t* pages_dev, int n_layers,
                               int64_t n_pool_pages, int64_t block_bytes, void* pool,
                               void* host_dev_ptr, int to_host, hipStream_t stream) {
  if (n_pages == 0) return hipSuccess;
  const dim3 grid(n_pages, 2 * n_layers);
  kv_page_copy_kernel<<<grid, 256, 0, stream>>>(pages_dev, n_layers, n_pool_pages, block_bytes,
                                               (char*)pool, (char*)host_dev_ptr, to_host);
  return hipGetLastError();
}

}  // namespace pdec

// Streaming-read microbenchmark: the measured HBM read ceiling that the
// decode attention is compared with next to the 8 TB/s specification.  Not
// part of the decode path.
//
//   * sequential: a grid-stride read of the whole buffer, four 16-byte
//     non-temporal loads in flight per lane;
//   * pages: whole 8 KB pages in a caller-given order, one wave per page and
//     eight 1 KB wavefront loads, which is the decode attention's access
//     pattern (a (page, kv head) K + V tile pair is one 8 KB region).
// Each workgroup folds what it read into one 16-byte word of `sink` so the
// loads cannot be dropped.
#include "common.h"
#include "kernels.h"

namespace sevo {

__global__ __launch_bounds__(256) void read_seq_kernel(const u32x4* __restrict__ p, size_t n16,
                                                       u32x4* __restrict__ sink) {
  constexpr int U = 4;
  const size_t stride = (size_t)gridDim.x * 256;
  u32x4 acc = u32x4{0u, 0u, 0u, 0u};
  size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  for (; i + (U - 1) * stride < n16; i += U * stride) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u];
  }
  for (; i < n16; i += stride) acc ^= __builtin_nontemporal_load(p + i);
  __shared__ u32x4 red[256];
  red[threadIdx.x] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    u32x4 r = u32x4{0u, 0u, 0u, 0u};
    for (int t = 0; t < 256; ++t) r ^= red[t];
    sink[blockIdx.x] = r;
  }
}

__global__ __launch_bounds__(256) void read_pages_kernel(const u32x4* __restrict__ p,
                                                         const int32_t* __restrict__ order,
                                                         int64_t n_pages, u32x4* __restrict__ sink) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 6;
  const int64_t nw = (int64_t)gridDim.x * 4;
  u32x4 acc = u32x4{0u, 0u, 0u, 0u};
  for (int64_t k = wave; k < n_pages; k += nw) {
    const int32_t pg = order[k];
    if (pg < 0 || pg >= n_pages) continue;  // an id outside the buffer is skipped
    const u32x4* base = p + (size_t)pg * 512;
    u32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(base + u * 64 + lane);
#pragma unroll
    for (int u = 0; u < 8; ++u) acc ^= v[u];
  }
  __shared__ u32x4 red[256];
  red[threadIdx.x] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    u32x4 r = u32x4{0u, 0u, 0u, 0u};
    for (int t = 0; t < 256; ++t) r ^= red[t];
    sink[blockIdx.x] = r;
  }
}

hipError_t launch_hbm_read_probe(const void* buf, size_t bytes, const int32_t* page_order,
                                 int grid, void* sink, hipStream_t st) {
  if (page_order)
    hipLaunchKernelGGL(read_pages_kernel, dim3(grid), dim3(256), 0, st,
                       static_cast<const u32x4*>(buf), page_order, (int64_t)(bytes / 8192),
                       static_cast<u32x4*>(sink));
  else
    hipLaunchKernelGGL(read_seq_kernel, dim3(grid), dim3(256), 0, st,
                       static_cast<const u32x4*>(buf), bytes / 16, static_cast<u32x4*>(sink));
  return hipGetLastError();
}

}  // namespace sevo

// Measurement helper: a plain streaming read of a device buffer, the rate the
// HBM attention and precompute kernels are compared against (the achievable
// read bandwidth of this device, beside the 8 TB/s of its specification).
//
// Workgroups sweep consecutive 32 KB blocks (grid-stride over blocks), every
// lane keeping eight 16-byte loads in flight, and fold the data with XOR; one
// word per workgroup goes to `sink`, so the reads cannot be elided.
#include "common.hpp"
#include "kernels.hpp"

namespace prc {
namespace {

constexpr int SR_THREADS = 256;
constexpr int SR_UNROLL = 8;                         // 16-byte loads in flight per lane
constexpr int SR_BLOCK = SR_THREADS * SR_UNROLL;     // chunks per workgroup block (32 KB)

__global__ void __launch_bounds__(SR_THREADS) stream_read_kernel(const u32x4* src, int64_t n_chunks, uint32_t* sink) {
  u32x4 acc = {0u, 0u, 0u, 0u};
  // Workgroup g reads the 32 KB blocks g, g + grid, ...; within a block each
  // load instruction of a wave covers 1 KB of consecutive chunks.
  for (int64_t blk = blockIdx.x; blk * SR_BLOCK < n_chunks; blk += gridDim.x) {
    const int64_t base = blk * SR_BLOCK + threadIdx.x;
    if (base + (SR_UNROLL - 1) * SR_THREADS < n_chunks) {
      u32x4 v[SR_UNROLL];
#pragma unroll
      for (int u = 0; u < SR_UNROLL; ++u) v[u] = __builtin_nontemporal_load(src + base + u * SR_THREADS);
#pragma unroll
      for (int u = 0; u < SR_UNROLL; ++u) acc ^= v[u];
    } else {
      for (int u = 0; u < SR_UNROLL; ++u)
        if (base + u * SR_THREADS < n_chunks) acc ^= src[base + u * SR_THREADS];
    }
  }
  uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) x ^= (uint32_t)__shfl_xor((int)x, m, 64);
  __shared__ uint32_t red[SR_THREADS / 64];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t s = 0;
#pragma unroll
    for (int w = 0; w < SR_THREADS / 64; ++w) s ^= red[w];
    sink[blockIdx.x] = s;
  }
}

}  // namespace

hipError_t launch_stream_read(const void* src, int64_t bytes, uint32_t* sink, int grid, hipStream_t st) {
  hipLaunchKernelGGL(stream_read_kernel, dim3(grid), dim3(SR_THREADS), 0, st, static_cast<const u32x4*>(src),
                     bytes / 16, sink);
  return hipGetLastError();
}

}  // namespace prc

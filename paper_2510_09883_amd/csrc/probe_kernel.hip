// HBM read-ceiling probe: a plain streaming read of a device buffer, to measure the read
// bandwidth the memory system actually delivers (the denominator the attention kernels are
// compared with, next to the 8 TB/s data-sheet peak).
//
// Every thread reads 16-byte words in a grid-stride loop, UNROLL loads in flight at a time,
// and folds them with XOR so the loads cannot be removed; one word per workgroup is written.
#include "../../include/delta_probe.h"

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int UNROLL>
__global__ __launch_bounds__(256) void read_probe_kernel(const u32x4* __restrict__ src, size_t n,
                                                         uint32_t* __restrict__ sink) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (; i + (UNROLL - 1) * stride < n; i += UNROLL * stride) {
    u32x4 v[UNROLL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) v[u] = src[i + u * stride];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) acc ^= v[u];
  }
  for (; i < n; i += stride) acc ^= src[i];
  uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
  __shared__ uint32_t s[256];
  s[threadIdx.x] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = 0;
    for (int t = 0; t < 256; ++t) r ^= s[t];
    sink[blockIdx.x] = r;
  }
}

}  // namespace

#pragma GCC visibility push(default)
extern "C" int delta_hbm_read_probe(const void* buf, size_t bytes, uint32_t* sink,
                                    int32_t n_workgroups, int32_t unroll, void* stream) {
  if (!buf || !sink || bytes < 16 || n_workgroups < 1 || (reinterpret_cast<uintptr_t>(buf) & 15))
    return -1;
  const size_t n = bytes / 16;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  const dim3 grid(n_workgroups), block(256);
  const u32x4* src = static_cast<const u32x4*>(buf);
  switch (unroll) {
    case 1: hipLaunchKernelGGL(read_probe_kernel<1>, grid, block, 0, st, src, n, sink); break;
    case 2: hipLaunchKernelGGL(read_probe_kernel<2>, grid, block, 0, st, src, n, sink); break;
    case 4: hipLaunchKernelGGL(read_probe_kernel<4>, grid, block, 0, st, src, n, sink); break;
    case 8: hipLaunchKernelGGL(read_probe_kernel<8>, grid, block, 0, st, src, n, sink); break;
    default: return -1;
  }
  return hipGetLastError() == hipSuccess ? 0 : -4;
}
#pragma GCC visibility pop

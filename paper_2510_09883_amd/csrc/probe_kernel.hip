// HBM read-ceiling probe: a plain streaming read of a device buffer, to measure the read
// bandwidth the memory system actually delivers (the denominator the attention kernels are
// compared with, next to the 8 TB/s data-sheet peak).
//
// Every workgroup streams its own contiguous share of the buffer, as the attention kernels'
// workgroups stream their pages: per step the 256 threads read UNROLL x 4 KB contiguous bytes
// (16 bytes per thread and load, one 1 KB run per wave and load) with non-temporal loads, all
// UNROLL loads of a step in flight at once, folded with XOR so the loads cannot be removed;
// one word per workgroup is written.
#include "../../include/delta_probe.h"

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int UNROLL>
__global__ __launch_bounds__(256) void read_probe_kernel(const u32x4* __restrict__ src, size_t n,
                                                         uint32_t* __restrict__ sink) {
  // this workgroup's words [lo, hi)
  const size_t per = n / gridDim.x;
  const size_t lo = (size_t)blockIdx.x * per;
  const size_t hi = blockIdx.x + 1 == gridDim.x ? n : lo + per;
  const int t = threadIdx.x;
  u32x4 acc = {0u, 0u, 0u, 0u};
  size_t i = lo;
  for (; i + (size_t)UNROLL * 256 <= hi; i += (size_t)UNROLL * 256) {
    u32x4 v[UNROLL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) v[u] = __builtin_nontemporal_load(src + i + u * 256 + t);
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) acc ^= v[u];
  }
  for (i += t; i < hi; i += 256) acc ^= src[i];
  uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
  __shared__ uint32_t s[256];
  s[t] = x;
  __syncthreads();
  if (t == 0) {
    uint32_t r = 0;
    for (int k = 0; k < 256; ++k) r ^= s[k];
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

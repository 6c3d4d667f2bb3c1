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

// Gather of 4 KB chunks (delta_hbm_gather_probe): the workgroup's chunk list goes to LDS, then
// every thread walks the list with a ring of three 16-byte loads (the loads of the next two
// chunks in flight while one is folded in), as a wave of the attention kernel walks its tiles.
constexpr int kGatherMaxChunks = 4096;
constexpr int kGatherRing = 3;

__global__ __launch_bounds__(256) void gather_probe_kernel(const u32x4* __restrict__ src,
                                                           const int64_t* __restrict__ chunks,
                                                           int n_chunks,
                                                           uint32_t* __restrict__ sink) {
  __shared__ int64_t s_list[kGatherMaxChunks];
  const int w = blockIdx.x, W = gridDim.x, t = threadIdx.x;
  const int c0 = (int)((int64_t)n_chunks * w / W), c1 = (int)((int64_t)n_chunks * (w + 1) / W);
  const int nc = c1 - c0;   // <= kGatherMaxChunks (checked on the host)
  for (int i = t; i < nc; i += 256) s_list[i] = chunks[c0 + i];
  __syncthreads();
  u32x4 acc = {0u, 0u, 0u, 0u};
  if (nc > 0) {
    u32x4 v[kGatherRing];
    auto fetch = [&](u32x4& x, int k) {
      x = __builtin_nontemporal_load(src + s_list[k < nc ? k : nc - 1] * 256 + t);
    };
#pragma unroll
    for (int i = 0; i < kGatherRing - 1; ++i) fetch(v[i], i);
    for (int k = 0; k < nc; k += kGatherRing) {
#pragma unroll
      for (int r = 0; r < kGatherRing; ++r) {
        fetch(v[(r + kGatherRing - 1) % kGatherRing], k + r + kGatherRing - 1);
        if (k + r < nc) acc ^= v[r];
      }
    }
  }
  sink[(size_t)w * 256 + t] = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
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
extern "C" int delta_hbm_gather_probe(const void* buf, size_t bytes, const int64_t* chunks,
                                      int32_t n_chunks, uint32_t* sink, int32_t n_workgroups,
                                      void* stream) {
  if (!buf || !chunks || !sink || bytes < 4096 || n_chunks < 1 || n_workgroups < 1 ||
      (reinterpret_cast<uintptr_t>(buf) & 15) ||
      ((int64_t)n_chunks + n_workgroups - 1) / n_workgroups > kGatherMaxChunks)
    return -1;
  hipLaunchKernelGGL(gather_probe_kernel, dim3(n_workgroups), dim3(256), 0,
                     static_cast<hipStream_t>(stream), static_cast<const u32x4*>(buf), chunks,
                     n_chunks, sink);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}
#pragma GCC visibility pop

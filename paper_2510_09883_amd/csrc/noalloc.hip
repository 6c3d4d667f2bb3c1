// Library-held scratch memory for the allocation-free decode step (delta_decode_step_noalloc):
// the split partials, arrival counters, Delta-layer logits, log-sum-exp, unit scores and
// selection locations that delta_decode_step keeps in the caller's workspace live here instead,
// in one file-scope device array per GPU.
//
// The array is a static device symbol of this translation unit's code object, which the HIP
// runtime loads onto a device (and so allocates the array there) the first time the symbol is
// looked up on that device; it stays until the process ends.  In host code `scratch` names a
// host-side stand-in, not device memory: its device address is looked up once per device with
// hipGetSymbolAddress (with that device current) and only that address is handed to kernels.
#include <mutex>

#include "internal.h"

namespace delta {
namespace {

static __device__ __align__(256) uint8_t scratch[kNoallocScratchBytes];

constexpr int kMaxDevices = 64;

__global__ void fill_zero2_kernel(uint32_t* p0, uint32_t n0, uint32_t* p1, uint32_t n1) {
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n0 + n1; i += gridDim.x * blockDim.x) {
    if (i < n0) p0[i] = 0u;
    else p1[i - n0] = 0u;
  }
}

}  // namespace

hipError_t noalloc_scratch(void** ptr) {
  static std::mutex mu;
  static void* addr[kMaxDevices];
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

// Zero-fills two word ranges in one launch (a kernel, not a memset node, so that it behaves
// the same inside a captured graph).
hipError_t launch_fill_zero2(void* p0, size_t bytes0, void* p1, size_t bytes1, hipStream_t stream) {
  const size_t n0 = bytes0 / 4, n1 = bytes1 / 4;
  if (n0 + n1 == 0) return hipSuccess;
  if (n0 + n1 > 0xffffffffu) return hipErrorInvalidValue;
  size_t blocks = (n0 + n1 + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(fill_zero2_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                     static_cast<uint32_t*>(p0), (uint32_t)n0, static_cast<uint32_t*>(p1),
                     (uint32_t)n1);
  return hipGetLastError();
}

}  // namespace delta

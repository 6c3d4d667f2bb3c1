// Device-side precondition checks of debug builds (-DDELTA_DEBUG=1; see delta_build_flags in
// the C ABI): a failure is recorded as a bit of the workspace's status word and the kernel goes
// on with an in-range value.  Release builds compile them away.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace delta {

// ORs `bit` into the status word (debug builds; status may be null: nothing recorded).
__device__ __forceinline__ void debug_flag(uint32_t* status, uint32_t bit) {
  if (DELTA_DEBUG && status)
    __hip_atomic_fetch_or(status, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// A physical page read through a page table or a selection: in debug builds one outside
// [0, n_pages) (n_pages = 0: unknown, only the sign is checked) is flagged and replaced by page 0.
__device__ __forceinline__ int checked_page(int p, int64_t n_pages, uint32_t* status) {
  if (!DELTA_DEBUG) return p;
  if (p < 0 || (n_pages > 0 && p >= n_pages)) {
    debug_flag(status, DELTA_DEBUG_PAGE);
    return 0;
  }
  return p;
}

}  // namespace delta

// KV append (Sec. 2, Eq. kv_update): the decoding step's key and value are written into the
// paged cache before attention reads it.  The token is the last one counted by seq_lens[b]:
// row (s_b - 1) % 16 of physical page page_table[b, (s_b - 1) / 16], in every KV head.
//
// One thread per 16 bytes: the K row of every KV head, then the V row (each a contiguous
// d-element bf16 row in the cache, coalesced within a head).
#include "internal.h"

namespace delta {
namespace {

constexpr int kAppendThreads = 256;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kAppendThreads) void kv_append_kernel(const AppendArgs a) {
  const int b = blockIdx.y;
  const int s = a.seq_lens[b];
  if (s < 1 || s > 16 * a.max_pages) return;   // no token slot: nothing written
  const int t = s - 1;
  const int page = a.page_table[(size_t)b * a.max_pages + (t >> 4)];
  // debug builds: a page outside the cache is not written (there is no status word to flag it)
  if (DELTA_DEBUG && (page < 0 || (a.n_pages > 0 && page >= a.n_pages))) return;
  const int row = t & 15;
  const int per_row = a.head_dim / 8;             // 16-byte pieces of one head's row
  const int chunks = a.n_kv_heads * per_row;      // of the K (or V) row over all heads
  for (int i = blockIdx.x * kAppendThreads + threadIdx.x; i < 2 * chunks;
       i += gridDim.x * kAppendThreads) {
    const bool is_v = i >= chunks;
    const int c = is_v ? i - chunks : i;
    const int h = c / per_row, e = c - h * per_row;
    const uint16_t* src = (is_v ? a.v_new : a.k_new) + ((size_t)b * a.n_kv_heads + h) * a.head_dim + 8 * e;
    uint16_t* dst = (is_v ? a.v_cache : a.k_cache) + (size_t)page * a.page_stride +
                    ((size_t)h * 16 + row) * a.head_dim + 8 * e;
    *reinterpret_cast<u32x4*>(dst) = *reinterpret_cast<const u32x4*>(src);
  }
}

}  // namespace

hipError_t launch_kv_append(const AppendArgs& a, int batch, hipStream_t stream) {
  const int pieces = 2 * a.n_kv_heads * (a.head_dim / 8);
  const dim3 grid((pieces + kAppendThreads - 1) / kAppendThreads, batch);
  hipLaunchKernelGGL(kv_append_kernel, grid, dim3(kAppendThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace delta

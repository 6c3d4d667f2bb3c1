// Cross-lane primitives for gfx950 wave64, all on the vector ALU (DPP and the lane-swap
// instructions): none of them goes through the LDS crossbar as ds_bpermute does.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace delta {

// op(x[l], x[l ^ 16]) and op(x[l], x[l ^ 32]).  v_permlane16_swap / v_permlane32_swap with both
// operands x return the two members of every lane pair (lower lane first in both lanes), so the
// two lanes of a pair compute op on the same operands in the same order: identical results.
__device__ __forceinline__ float max_xor16(float x) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
}
__device__ __forceinline__ float max_xor32(float x) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
}
__device__ __forceinline__ float sum_xor16(float x) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}
__device__ __forceinline__ float sum_xor32(float x) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}

// DPP lane moves inside rows of 16 lanes: x of lane l ^ 1, l ^ 2 (quad permutations) and
// l ^ 8 (rotation of the row by 8).
__device__ __forceinline__ float lane_xor1(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xf, 0xf, false));
}
__device__ __forceinline__ float lane_xor2(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x4E, 0xf, 0xf, false));
}
__device__ __forceinline__ float lane_xor8(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x128, 0xf, 0xf, false));
}

// Inclusive prefix sum over the 64 lanes: row shifts by 1, 2, 4, 8 (lanes shifted in from
// outside the row add 0), then lane 15 of rows 0 / 2 is added to rows 1 / 3 and lane 31 to
// rows 2 and 3.
__device__ __forceinline__ int wave_incl_scan(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);
  return v;
}

// Bitwise OR / AND and unsigned minimum of all 64 lanes, returned in every lane (quad swaps,
// row half-mirror and mirror, then the 16- and 32-lane swaps; the three operations are
// idempotent, so any pairing works).
__device__ __forceinline__ uint32_t wave_or(uint32_t v) {
  v |= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xf, 0xf, false);
  v |= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xf, 0xf, false);
  v |= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x141, 0xf, 0xf, false);
  v |= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x140, 0xf, 0xf, false);
  const auto p = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  v = p[0] | p[1];
  const auto q = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return q[0] | q[1];
}
__device__ __forceinline__ uint32_t wave_and(uint32_t v) {
  v &= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xf, 0xf, false);
  v &= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xf, 0xf, false);
  v &= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x141, 0xf, 0xf, false);
  v &= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x140, 0xf, 0xf, false);
  const auto p = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  v = p[0] & p[1];
  const auto q = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return q[0] & q[1];
}

__device__ __forceinline__ uint32_t wave_min(uint32_t v) {
  v = min(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xf, 0xf, false));
  v = min(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xf, 0xf, false));
  v = min(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x141, 0xf, 0xf, false));
  v = min(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x140, 0xf, 0xf, false));
  const auto p = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  v = min(p[0], p[1]);
  const auto q = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return min(q[0], q[1]);
}

// Workgroup barrier that orders LDS accesses only: the waves wait for their own LDS operations,
// not for outstanding global loads (which __syncthreads would also drain), so loads issued
// before the barrier stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

}  // namespace delta

// Page scoring and page selection for Delta layers (Sec. 4 "Selection mechanism" and
// "Page-based DELTA"; App. A, Alg. 2 RefreshPages), gfx950.
//
// score_kernel: one thread per token.  With the Delta-layer attention's log2-domain logits
//   x_j(t) and per-head log-sum-exp lse_j, the softmax weight is alpha_j(t) = 2^(x_j(t) - lse_j).
//   Token score s_t = max_j alpha_j(t) = 2^(max_j (x_j(t) - lse_j)) (exp2 is increasing, so one
//   exp2 per token suffices), or sum_j alpha_j(t) with the sum aggregation.  Unit score
//   S_u = sum of s_t over the unit's tokens: a 16-lane butterfly for pages, the token itself
//   for token-level units.
//
// select_kernel: one wave per sequence (no workgroup barriers).  Units [n_u - L, n_u) are kept; among
//   the n_u - L older units the (K - L) largest scores are found by an exact radix select on
//   the float bit patterns (non-negative floats order like their uint32 bits): four 8-bit
//   digit histograms in LDS give the exact threshold key T and how many keys equal to T are
//   needed.  A final pass in index order takes every key > T and the lowest-index keys == T
//   (ballot prefix counts), writing them in ascending order.  While n_u <= K every unit is
//   kept.
#include "internal.h"

namespace delta {
namespace {

constexpr float kNegInf = -__builtin_huge_valf();
constexpr int kScoreThreads = 256;
constexpr int kSelectThreads = 64;   // one wave per sequence
constexpr int kLdsKeys = 8192;   // candidate keys cached in LDS when they fit

template <int AGG, int U>
__global__ __launch_bounds__(kScoreThreads) void score_kernel(const ScoreArgs a) {
  const int b = blockIdx.y;
  const int t = blockIdx.x * kScoreThreads + threadIdx.x;
  const int s_b = min(a.seq_lens[b], a.max_seq_len);
  if ((int)(blockIdx.x * kScoreThreads) >= s_b) return;
  const int Hq = a.n_q_heads;
  const float* lse = a.lse + (size_t)b * Hq;
  float sc = 0.f;
  if (t < s_b) {
    // page-major logits [b][page][head][16]: token t is row t%16 of page t/16
    const float* row = a.logits + ((size_t)b * a.logit_pages + (t >> 4)) * Hq * 16 + (t & 15);
    if (AGG == 0) {
      float m = kNegInf;
#pragma unroll 8
      for (int j = 0; j < Hq; ++j) m = fmaxf(m, row[j * 16] - lse[j]);
      sc = exp2f(m);
    } else {
#pragma unroll 8
      for (int j = 0; j < Hq; ++j) sc += exp2f(row[j * 16] - lse[j]);
    }
  }
  float* out = a.unit_scores + (size_t)b * a.nu_stride;
  if (U == 16) {
    sc += __shfl_xor(sc, 1);
    sc += __shfl_xor(sc, 2);
    sc += __shfl_xor(sc, 4);
    sc += __shfl_xor(sc, 8);
    if ((t & 15) == 0 && t < s_b) out[t >> 4] = sc;
  } else {
    if (t < s_b) out[t] = sc;
  }
}

__device__ __forceinline__ uint32_t key_of(float f) {
  return f > 0.f ? __float_as_uint(f) : 0u;   // scores are >= 0; NaN / -0 map to 0
}

// Wave-synchronous LDS ordering (one wave's LDS requests execute in order; this keeps the
// compiler from moving them).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// One wave per sequence: no workgroup barriers anywhere.
__global__ __launch_bounds__(kSelectThreads) void select_kernel(const SelectArgs a) {
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int U = a.unit_tokens;
  const int K = a.budget_units;
  const int L = a.recent_units;
  const int s_b = a.seq_lens[b];
  const int n_u = min((s_b + U - 1) / U, a.nu_stride);
  int32_t* idx_out = a.sel_idx + (size_t)b * K;

  if (n_u <= K) {   // the context fits the budget: keep every unit
    for (int i = lane; i < K; i += kSelectThreads) idx_out[i] = (i < n_u) ? i : -1;
    if (lane == 0) a.sel_cnt[b] = max(n_u, 0);
    return;
  }
  const int n_c = n_u - L;      // candidate (older) units
  const int need = K - L;       // >= 1
  const float* S = a.unit_scores + (size_t)b * a.nu_stride;
  const unsigned long long lt_mask = (1ull << lane) - 1ull;

  __shared__ uint32_t s_keys[kLdsKeys];
  __shared__ uint32_t s_hist[256];
  const bool in_lds = n_c <= kLdsKeys;
  if (in_lds) {
    // eight independent loads in flight per lane before any is stored
    for (int i0 = 0; i0 < n_c; i0 += 8 * kSelectThreads) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int i = i0 + u * kSelectThreads + lane;
        v[u] = (i < n_c) ? S[i] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int i = i0 + u * kSelectThreads + lane;
        if (i < n_c) s_keys[i] = key_of(v[u]);
      }
    }
  }
  auto key_at = [&](int i) -> uint32_t { return in_lds ? s_keys[i] : key_of(S[i]); };

  uint32_t prefix = 0;
  int remaining = need;   // rank of the threshold among the keys matching `prefix`
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    for (int i = lane; i < 256; i += kSelectThreads) s_hist[i] = 0;
    wave_lds_sync();
    for (int i = lane; i < n_c; i += kSelectThreads) {
      const uint32_t k = key_at(i);
      const bool match = (pass == 0) || ((k >> (shift + 8)) == (prefix >> (shift + 8)));
      if (match) atomicAdd(&s_hist[(k >> shift) & 255u], 1u);
    }
    wave_lds_sync();
    // lane l owns digits 255-4l .. 252-4l (descending); the lane where the running count
    // from the top reaches `remaining` holds the threshold's digit
    int c[4], sum = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      c[k] = (int)s_hist[255 - 4 * lane - k];
      sum += c[k];
    }
    int incl = sum;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int y = __shfl_up(incl, off);
      if (lane >= off) incl += y;
    }
    const int excl = incl - sum;
    int digit = 0, above = 0;
    int run = excl;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (run < remaining && remaining <= run + c[k]) {
        digit = 255 - 4 * lane - k;
        above = run;
      }
      run += c[k];
    }
    const unsigned long long hit = __ballot(excl < remaining && remaining <= incl);
    const int src = __ffsll((long long)hit) - 1;
    digit = __shfl(digit, src);
    above = __shfl(above, src);
    prefix |= (uint32_t)digit << shift;
    remaining -= above;
  }
  const uint32_t T = prefix;   // the need-th largest key; `remaining` keys equal to T are taken

  int carry_eq = 0, carry_sel = 0;
  for (int base = 0; base < n_c; base += kSelectThreads) {
    const int i = base + lane;
    const uint32_t k = (i < n_c) ? key_at(i) : 0u;
    const bool gt = (i < n_c) && k > T;
    const bool eq = (i < n_c) && k == T;
    const unsigned long long eqm = __ballot(eq);
    const bool take = gt || (eq && carry_eq + __popcll(eqm & lt_mask) < remaining);
    const unsigned long long tm = __ballot(take);
    const int pos = carry_sel + __popcll(tm & lt_mask);
    if (take && pos < need) idx_out[pos] = i;
    carry_eq += __popcll(eqm);
    carry_sel += __popcll(tm);
  }
  for (int j = lane; j < L; j += kSelectThreads) idx_out[need + j] = n_c + j;
  if (lane == 0) a.sel_cnt[b] = K;
}

__global__ void fill_zero_kernel(uint32_t* p, size_t n_words) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n_words;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

}  // namespace

hipError_t launch_score(int agg, int unit_tokens, const ScoreArgs& a, int batch,
                        hipStream_t stream) {
  const dim3 grid((a.max_seq_len + kScoreThreads - 1) / kScoreThreads, batch);
  const dim3 block(kScoreThreads);
  if (agg == 0 && unit_tokens == 16) hipLaunchKernelGGL((score_kernel<0, 16>), grid, block, 0, stream, a);
  else if (agg == 0 && unit_tokens == 1) hipLaunchKernelGGL((score_kernel<0, 1>), grid, block, 0, stream, a);
  else if (agg == 1 && unit_tokens == 16) hipLaunchKernelGGL((score_kernel<1, 16>), grid, block, 0, stream, a);
  else if (agg == 1 && unit_tokens == 1) hipLaunchKernelGGL((score_kernel<1, 1>), grid, block, 0, stream, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_select(const SelectArgs& a, int batch, hipStream_t stream) {
  hipLaunchKernelGGL(select_kernel, dim3(batch), dim3(kSelectThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* ptr, size_t bytes, hipStream_t stream) {
  const size_t words = bytes / 4;
  if (words == 0) return hipSuccess;
  size_t blocks = (words + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                     static_cast<uint32_t*>(ptr), words);
  return hipGetLastError();
}

}  // namespace delta

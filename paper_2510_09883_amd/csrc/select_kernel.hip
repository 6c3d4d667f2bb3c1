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
// select_kernel: one 1024-thread workgroup per sequence.  Units [n_u - L, n_u) are kept; among
//   the n_u - L older units the (K - L) largest scores are found by an exact radix select on
//   the float bit patterns (non-negative floats order like their uint32 bits): four 8-bit
//   digit histograms in LDS give the exact threshold key T and how many keys equal to T are
//   needed.  A final pass in index order takes every key > T and the lowest-index keys == T
//   (block-wide ballot scans), writing them in ascending order.  While n_u <= K every unit is
//   kept.
#include "internal.h"

namespace delta {
namespace {

constexpr float kNegInf = -__builtin_huge_valf();
constexpr int kScoreThreads = 256;
constexpr int kSelectThreads = 1024;
constexpr int kSelectWaves = kSelectThreads / 64;
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
    const float* row = a.logits + (size_t)b * Hq * a.logit_stride + t;
    if (AGG == 0) {
      float m = kNegInf;
#pragma unroll 8
      for (int j = 0; j < Hq; ++j) m = fmaxf(m, row[(size_t)j * a.logit_stride] - lse[j]);
      sc = exp2f(m);
    } else {
#pragma unroll 8
      for (int j = 0; j < Hq; ++j) sc += exp2f(row[(size_t)j * a.logit_stride] - lse[j]);
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

// Exclusive prefix count of `flag` over the workgroup in thread order; *total gets the sum.
__device__ __forceinline__ int block_scan_flag(bool flag, int* s_wave, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const unsigned long long m = __ballot(flag);
  const int pre = __popcll(m & ((1ull << lane) - 1ull));
  if (lane == 0) s_wave[w] = __popcll(m);
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < kSelectWaves; ++i) {
    const int c = s_wave[i];
    base += (i < w) ? c : 0;
    tot += c;
  }
  __syncthreads();
  *total = tot;
  return base + pre;
}

__global__ __launch_bounds__(kSelectThreads) void select_kernel(const SelectArgs a) {
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int U = a.unit_tokens;
  const int K = a.budget_units;
  const int L = a.recent_units;
  const int s_b = a.seq_lens[b];
  const int n_u = min((s_b + U - 1) / U, a.nu_stride);
  int32_t* idx_out = a.sel_idx + (size_t)b * K;

  if (n_u <= K) {   // the context fits the budget: keep every unit
    for (int i = tid; i < K; i += kSelectThreads) idx_out[i] = (i < n_u) ? i : -1;
    if (tid == 0) a.sel_cnt[b] = max(n_u, 0);
    return;
  }
  const int n_c = n_u - L;      // candidate (older) units
  const int need = K - L;       // >= 1
  const float* S = a.unit_scores + (size_t)b * a.nu_stride;

  __shared__ uint32_t s_keys[kLdsKeys];
  __shared__ uint32_t s_hist[256];
  __shared__ int s_wave[kSelectWaves];
  __shared__ uint32_t s_digit;
  __shared__ int s_above;
  const bool in_lds = n_c <= kLdsKeys;
  if (in_lds)
    for (int i = tid; i < n_c; i += kSelectThreads) s_keys[i] = key_of(S[i]);
  auto key_at = [&](int i) -> uint32_t { return in_lds ? s_keys[i] : key_of(S[i]); };

  uint32_t prefix = 0;
  int remaining = need;   // rank of the threshold among the keys matching `prefix`
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    for (int i = tid; i < 256; i += kSelectThreads) s_hist[i] = 0;
    __syncthreads();
    for (int i = tid; i < n_c; i += kSelectThreads) {
      const uint32_t k = key_at(i);
      const bool match = (pass == 0) || ((k >> (shift + 8)) == (prefix >> (shift + 8)));
      if (match) atomicAdd(&s_hist[(k >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid < 64) {
      // lane l owns digits 255-4l .. 252-4l (descending); find where the running count from
      // the top reaches `remaining`
      int c[4], sum = 0;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        c[k] = (int)s_hist[255 - 4 * tid - k];
        sum += c[k];
      }
      int incl = sum;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(incl, off);
        if (tid >= off) incl += y;
      }
      const int excl = incl - sum;
      if (excl < remaining && remaining <= incl) {
        int run = excl;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          if (run < remaining && remaining <= run + c[k]) {
            s_digit = (uint32_t)(255 - 4 * tid - k);
            s_above = run;
          }
          run += c[k];
        }
      }
    }
    __syncthreads();
    prefix |= s_digit << shift;
    remaining -= s_above;
    __syncthreads();
  }
  const uint32_t T = prefix;   // the need-th largest key; `remaining` keys equal to T are taken

  int carry_eq = 0, carry_sel = 0;
  for (int base = 0; base < n_c; base += kSelectThreads) {
    const int i = base + tid;
    const uint32_t k = (i < n_c) ? key_at(i) : 0u;
    const bool gt = (i < n_c) && k > T;
    const bool eq = (i < n_c) && k == T;
    int tot_eq, tot_sel;
    const int eq_rank = carry_eq + block_scan_flag(eq, s_wave, &tot_eq);
    const bool take = gt || (eq && eq_rank < remaining);
    const int pos = carry_sel + block_scan_flag(take, s_wave, &tot_sel);
    if (take && pos < need) idx_out[pos] = i;
    carry_eq += tot_eq;
    carry_sel += tot_sel;
  }
  for (int j = tid; j < L; j += kSelectThreads) idx_out[need + j] = n_c + j;
  if (tid == 0) a.sel_cnt[b] = K;
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

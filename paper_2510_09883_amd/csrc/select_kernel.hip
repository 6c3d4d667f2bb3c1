// Page scoring and page selection for Delta layers (Sec. 4 "Selection mechanism" and
// "Page-based DELTA"; App. A, Alg. 2 RefreshPages), gfx950.
//
// score_kernel: one thread per four tokens.  With the Delta-layer attention's log2-domain logits
//   x_j(t) and per-head log-sum-exp lse_j, the softmax weight is alpha_j(t) = 2^(x_j(t) - lse_j).
//   Token score s_t = max_j alpha_j(t) = 2^(max_j (x_j(t) - lse_j)) (exp2 is increasing, so one
//   exp2 per token suffices), or sum_j alpha_j(t) with the sum aggregation.  Unit score
//   S_u = sum of s_t over the unit's tokens: four tokens per thread and a 4-lane butterfly for
//   pages, the token itself for token-level units.
//
// select_kernel: one 256-thread workgroup per sequence, candidate keys in registers.  Units
//   [n_u - L, n_u) are kept; among
//   the n_u - L older units the (K - L) largest scores are found by an exact radix select on
//   the float bit patterns (non-negative floats order like their uint32 bits): after skipping
//   the leading bits common to all keys, 8-bit digit histograms in LDS give the exact
//   threshold key T and how many keys equal to T are needed.  A final pass in index order
//   takes every key > T and the lowest-index keys == T (block prefix sums), writing them in
//   ascending order.  While n_u <= K every unit is
//   kept.
#include "internal.h"

namespace delta {
namespace {

constexpr float kNegInf = -__builtin_huge_valf();
constexpr int kScoreThreads = 256;
constexpr int kSelectThreads = 256;
constexpr int kSelectWaves = kSelectThreads / 64;

typedef float f32x4 __attribute__((ext_vector_type(4)));

// One thread per four consecutive tokens (one 16-byte load per head; a page is four threads).
template <int AGG, int U>
__global__ __launch_bounds__(kScoreThreads) void score_kernel(const ScoreArgs a) {
  const int b = blockIdx.y;
  const int t0 = (blockIdx.x * kScoreThreads + threadIdx.x) * 4;
  const int s_b = min(a.seq_lens[b], a.max_seq_len);
  if ((int)(blockIdx.x * kScoreThreads * 4) >= s_b) return;
  const int Hq = a.n_q_heads;
  const float* lse = a.lse + (size_t)b * Hq;
  float sc[4] = {0.f, 0.f, 0.f, 0.f};
  if (t0 < s_b) {
    // group-major logits [b][g][page][h][16]: tokens t0..t0+3 are rows t0%16.. of page t0/16;
    // head j = g*G + h
    const int G = Hq / a.n_kv_heads;
    const size_t gstride = (size_t)a.logit_pages * G * 16;
    const float* row = a.logits + (size_t)b * a.n_kv_heads * gstride + (size_t)(t0 >> 4) * G * 16 + (t0 & 15);
    f32x4 acc;
    if (AGG == 0) acc = f32x4{kNegInf, kNegInf, kNegInf, kNegInf};
    else acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 16
    for (int j = 0; j < Hq; ++j) {
      const int g = j / G, h = j - g * G;
      const f32x4 x = *reinterpret_cast<const f32x4*>(row + g * gstride + h * 16);
      const float l = lse[j];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        if (AGG == 0) acc[c] = fmaxf(acc[c], x[c] - l);
        else acc[c] += exp2f(x[c] - l);
      }
    }
#pragma unroll
    for (int c = 0; c < 4; ++c)
      sc[c] = (t0 + c < s_b) ? (AGG == 0 ? exp2f(acc[c]) : acc[c]) : 0.f;
  }
  float* out = a.unit_scores + (size_t)b * a.nu_stride;
  if (U == 16) {
    float p = (sc[0] + sc[1]) + (sc[2] + sc[3]);
    p += __shfl_xor(p, 1);
    p += __shfl_xor(p, 2);
    if ((t0 & 15) == 0 && t0 < s_b) out[t0 >> 4] = p;
  } else {
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (t0 + c < s_b) out[t0 + c] = sc[c];
  }
}

__device__ __forceinline__ uint32_t key_of(float f) {
  return f > 0.f ? __float_as_uint(f) : 0u;   // scores are >= 0; NaN / -0 map to 0
}

// Exclusive prefix sum of one int per thread over the workgroup; *total gets the sum.
__device__ __forceinline__ int block_excl_scan(int v, int* s_wave, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(incl, off);
    if (lane >= off) incl += y;
  }
  if (lane == 63) s_wave[w] = incl;
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
  return base + incl - v;
}

// One workgroup per sequence.  Thread t owns the candidate keys [t*KPT, t*KPT + KPT) in
// registers, so index order is thread order then slot order and one block scan places every
// chosen unit.  KPT (keys per thread) is chosen on the host from the candidate bound.
template <int KPT>
__global__ __launch_bounds__(kSelectThreads) void select_kernel(const SelectArgs a) {
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
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
  const int n_c = min(n_u - L, KPT * kSelectThreads);   // candidate (older) units; the host bounds it
  const int need = K - L;       // >= 1
  const float* S = a.unit_scores + (size_t)b * a.nu_stride;
  const int i0 = tid * KPT;

  __shared__ uint32_t s_hist[256];
  __shared__ int s_wave[kSelectWaves];
  __shared__ uint32_t s_red[2][kSelectWaves];
  __shared__ int s_digit, s_above;

  // unconditional loads (indices clamped into the row) so that all of them are in flight at
  // once; slots past this thread's keys are zeroed afterwards
  uint32_t key[KPT];
#pragma unroll
  for (int j = 0; j < KPT; ++j) key[j] = key_of(S[min(i0 + j, n_c - 1)]);
#pragma unroll
  for (int j = 0; j < KPT; ++j)
    if (!(i0 + j < n_c)) key[j] = 0u;
  // Bits shared by every candidate key need no histogram: start the digit passes at the
  // highest bit where two keys differ (page scores mostly share sign and high exponent bits,
  // which would otherwise send every key of the first pass to the same bin).
  uint32_t k_or = 0u, k_and = 0xffffffffu;
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    if (i0 + j < n_c) {
      k_or |= key[j];
      k_and &= key[j];
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    k_or |= (uint32_t)__shfl_xor((int)k_or, off);
    k_and &= (uint32_t)__shfl_xor((int)k_and, off);
  }
  if (lane == 0) {
    s_red[0][tid >> 6] = k_or;
    s_red[1][tid >> 6] = k_and;
  }
  __syncthreads();
  k_or = 0u;
  k_and = 0xffffffffu;
#pragma unroll
  for (int w = 0; w < kSelectWaves; ++w) {
    k_or |= s_red[0][w];
    k_and &= s_red[1][w];
  }
  const uint32_t differ = k_or ^ k_and;
  int low = differ ? 32 - __clz((int)differ) : 0;   // bits [low, 32) are common to all keys
  uint32_t prefix = low >= 32 ? 0u : (k_and & ~((1u << low) - 1u));
  int remaining = need;   // rank of the threshold among the keys matching `prefix`
  while (low > 0) {
    const int width = min(8, low);
    const int shift = low - width;
    const int top = shift + width;                    // bits [top, 32) already fixed
    s_hist[tid] = 0u;                                 // kSelectThreads == 256 bins
    __syncthreads();
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
      const uint32_t k = key[j];
      const bool match = i0 + j < n_c && (top >= 32 || (k >> top) == (prefix >> top));
      if (match) atomicAdd(&s_hist[(k >> shift) & ((1u << width) - 1u)], 1u);
    }
    __syncthreads();
    if (tid < 64) {
      // lane l owns digits 255-4l .. 252-4l (descending); the lane where the running count
      // from the top reaches `remaining` holds the threshold's digit
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
            s_digit = 255 - 4 * tid - k;
            s_above = run;
          }
          run += c[k];
        }
      }
    }
    __syncthreads();
    prefix |= (uint32_t)s_digit << shift;
    remaining -= s_above;
    low = shift;
  }
  const uint32_t T = prefix;   // the need-th largest key; `remaining` keys equal to T are taken

  int n_eq = 0;
#pragma unroll
  for (int j = 0; j < KPT; ++j) n_eq += (i0 + j < n_c && key[j] == T);
  int tot;
  int eq_rank = block_excl_scan(n_eq, s_wave, &tot);
  int n_take = 0;
  uint32_t take_mask = 0u;
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    const bool valid = i0 + j < n_c;
    bool take = valid && key[j] > T;
    if (valid && key[j] == T) {
      take = eq_rank < remaining;
      ++eq_rank;
    }
    take_mask |= (take ? 1u : 0u) << j;
    n_take += take;
  }
  int pos = block_excl_scan(n_take, s_wave, &tot);
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    if ((take_mask >> j) & 1u) {
      if (pos < need) idx_out[pos] = i0 + j;
      ++pos;
    }
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
  const dim3 grid((a.max_seq_len + 4 * kScoreThreads - 1) / (4 * kScoreThreads), batch);
  const dim3 block(kScoreThreads);
  if (agg == 0 && unit_tokens == 16) hipLaunchKernelGGL((score_kernel<0, 16>), grid, block, 0, stream, a);
  else if (agg == 0 && unit_tokens == 1) hipLaunchKernelGGL((score_kernel<0, 1>), grid, block, 0, stream, a);
  else if (agg == 1 && unit_tokens == 16) hipLaunchKernelGGL((score_kernel<1, 16>), grid, block, 0, stream, a);
  else if (agg == 1 && unit_tokens == 1) hipLaunchKernelGGL((score_kernel<1, 1>), grid, block, 0, stream, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_select(const SelectArgs& a, int batch, hipStream_t stream) {
  // keys per thread: the smallest power of two covering the candidate bound
  const int bound = a.nu_stride - a.recent_units;
  const dim3 grid(batch), block(kSelectThreads);
  if (bound <= 1 * kSelectThreads) hipLaunchKernelGGL(select_kernel<1>, grid, block, 0, stream, a);
  else if (bound <= 2 * kSelectThreads) hipLaunchKernelGGL(select_kernel<2>, grid, block, 0, stream, a);
  else if (bound <= 4 * kSelectThreads) hipLaunchKernelGGL(select_kernel<4>, grid, block, 0, stream, a);
  else if (bound <= 8 * kSelectThreads) hipLaunchKernelGGL(select_kernel<8>, grid, block, 0, stream, a);
  else if (bound <= 16 * kSelectThreads) hipLaunchKernelGGL(select_kernel<16>, grid, block, 0, stream, a);
  else if (bound <= 32 * kSelectThreads) hipLaunchKernelGGL(select_kernel<32>, grid, block, 0, stream, a);
  else return hipErrorInvalidValue;
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

// Page scoring and page selection for Delta layers (Sec. 4 "Selection mechanism" and
// "Page-based DELTA"; App. A, Alg. 2 RefreshPages), gfx950.
//
// score_kernel: one workgroup per 256 tokens of a sequence, one lane per four tokens, the query
//   heads split over the four waves.  With the Delta-layer attention's log2-domain logits
//   x_j(t) and per-head log-sum-exp lse_j, the softmax weight is alpha_j(t) = 2^(x_j(t) - lse_j).
//   Token score s_t = max_j alpha_j(t) = 2^(max_j (x_j(t) - lse_j)) (exp2 is increasing, so one
//   exp2 per token suffices), or sum_j alpha_j(t) with the sum aggregation.  Unit score
//   S_u = sum of s_t over the unit's tokens: four tokens per lane and a 4-lane butterfly for
//   pages, the token itself for token-level units.
//
// select_kernel: one 256-thread workgroup per sequence runs the exact radix selection of
//   select_impl.h (last L units plus the top-(K - L) older units, ties to the lower index).
#include "internal.h"
#include "select_impl.h"
#include "wave.h"

namespace delta {
namespace {

constexpr float kNegInf = -__builtin_huge_valf();
constexpr int kScoreThreads = 256;
constexpr int kScoreWaves = kScoreThreads / 64;
constexpr int kScoreTokens = 256;   // tokens per scoring workgroup (four per lane)

typedef float f32x4 __attribute__((ext_vector_type(4)));

// One workgroup per 256 tokens (16 pages) of one sequence.  Lane l of every wave takes tokens
// 4l .. 4l+3 (one 16-byte load per head); wave w takes a contiguous quarter of the query heads,
// and all of its heads' loads are issued before the first is used, so each thread waits for
// memory once.  The four waves' partial reductions meet in LDS.
template <int AGG, int U, int NH>
__global__ __launch_bounds__(kScoreThreads) void score_kernel(const ScoreArgs a) {
  __shared__ f32x4 s_part[kScoreWaves][64];
  const int b = blockIdx.y;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int tb = blockIdx.x * kScoreTokens;
  const int s_b = min(a.seq_lens[b], a.max_seq_len);
  if (tb >= s_b) return;   // uniform over the workgroup
  const int t0 = tb + 4 * lane;
  const int Hq = a.n_q_heads;
  const int G = Hq / a.n_kv_heads;
  const int hpw = (Hq + kScoreWaves - 1) / kScoreWaves;
  const int j0 = wave * hpw;
  const int nj = min(hpw, Hq - j0);   // heads of this wave (<= 0 when Hq < 4 waves' worth)
  const float* lse = a.lse + (size_t)b * Hq;
  // group-major logits [b][g][page][h][16]: tokens t0..t0+3 are rows t0%16.. of page t0/16.
  // Lanes past the sequence read its last quad instead (inside the buffer; masked below).
  const int tl = min(t0, (s_b - 1) & ~3);
  const size_t gstride = (size_t)a.logit_pages * G * 16;
  const float* row = a.logits + (size_t)b * a.n_kv_heads * gstride + (size_t)(tl >> 4) * G * 16 + (tl & 15);

  f32x4 acc;
  if (AGG == 0) acc = f32x4{kNegInf, kNegInf, kNegInf, kNegInf};
  else acc = f32x4{0.f, 0.f, 0.f, 0.f};
  int gg = j0 / G, hh = j0 - (j0 / G) * G;   // kv group and head-in-group of head j0 + jb
  for (int jb = 0; jb < nj; jb += NH) {
    // heads j0 + jb .. j0 + jb + NH - 1, clamped to the wave's last head (re-reads are masked)
    f32x4 x[NH];
    float l[NH];
#pragma unroll
    for (int k = 0; k < NH; ++k) {
      x[k] = *reinterpret_cast<const f32x4*>(row + gg * gstride + hh * 16);
      l[k] = lse[j0 + min(jb + k, nj - 1)];
      if (jb + k + 1 < nj && ++hh == G) {
        hh = 0;
        ++gg;
      }
    }
    // keep every load of the batch ahead of the first use (one wait for memory per batch)
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int k = 0; k < NH; ++k) {
      const bool ok = jb + k < nj;   // branch-free: every load above stays unconditional
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        if (AGG == 0) acc[c] = fmaxf(acc[c], ok ? x[k][c] - l[k] : kNegInf);
        else acc[c] += ok ? exp2f(x[k][c] - l[k]) : 0.f;
      }
    }
  }
  s_part[wave][lane] = acc;
  lds_barrier();
  if (wave != 0) return;
#pragma unroll
  for (int w = 1; w < kScoreWaves; ++w) {
    const f32x4 y = s_part[w][lane];
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] = (AGG == 0) ? fmaxf(acc[c], y[c]) : acc[c] + y[c];
  }
  float sc[4];
#pragma unroll
  for (int c = 0; c < 4; ++c)
    sc[c] = (t0 + c < s_b) ? (AGG == 0 ? exp2f(acc[c]) : acc[c]) : 0.f;
  float* out = a.unit_scores + (size_t)b * a.nu_stride;
  if (U == 16) {
    float p = (sc[0] + sc[1]) + (sc[2] + sc[3]);
    p += lane_xor1(p);
    p += lane_xor2(p);
    if ((t0 & 15) == 0 && t0 < s_b) out[t0 >> 4] = p;
  } else {
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (t0 + c < s_b) out[t0 + c] = sc[c];
  }
}

// One workgroup per sequence.
template <int KPT, int U>
__global__ __launch_bounds__(kSelectThreads) void select_kernel(const SelectArgs a) {
  select_sequence<KPT, U>(a, blockIdx.x);
}

__global__ void fill_zero_kernel(uint32_t* p, size_t n_words) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n_words;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

}  // namespace

namespace {

template <int AGG, int U>
hipError_t launch_score_nh(int nh, const ScoreArgs& a, dim3 grid, hipStream_t stream) {
  const dim3 block(kScoreThreads);
  switch (nh) {
    case 1: hipLaunchKernelGGL((score_kernel<AGG, U, 1>), grid, block, 0, stream, a); break;
    case 2: hipLaunchKernelGGL((score_kernel<AGG, U, 2>), grid, block, 0, stream, a); break;
    case 4: hipLaunchKernelGGL((score_kernel<AGG, U, 4>), grid, block, 0, stream, a); break;
    default: hipLaunchKernelGGL((score_kernel<AGG, U, 8>), grid, block, 0, stream, a); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_score(int agg, int unit_tokens, const ScoreArgs& a, int batch,
                        hipStream_t stream) {
  const dim3 grid((a.max_seq_len + kScoreTokens - 1) / kScoreTokens, batch);
  // heads per wave, rounded up to the unrolled load batch (at most 8 loads per batch)
  const int hpw = (a.n_q_heads + kScoreWaves - 1) / kScoreWaves;
  const int nh = hpw <= 1 ? 1 : hpw <= 2 ? 2 : hpw <= 4 ? 4 : 8;
  if (agg == 0 && unit_tokens == 16) return launch_score_nh<0, 16>(nh, a, grid, stream);
  if (agg == 0 && unit_tokens == 1) return launch_score_nh<0, 1>(nh, a, grid, stream);
  if (agg == 1 && unit_tokens == 16) return launch_score_nh<1, 16>(nh, a, grid, stream);
  if (agg == 1 && unit_tokens == 1) return launch_score_nh<1, 1>(nh, a, grid, stream);
  return hipErrorInvalidValue;
}

namespace {

template <int U>
hipError_t launch_select_u(const SelectArgs& a, int batch, hipStream_t stream) {
  // keys per thread: the smallest power of two covering the candidate bound
  const int bound = a.nu_stride - a.recent_units;
  const dim3 grid(batch), block(kSelectThreads);
  if (bound <= 1 * kSelectThreads) hipLaunchKernelGGL((select_kernel<1, U>), grid, block, 0, stream, a);
  else if (bound <= 2 * kSelectThreads) hipLaunchKernelGGL((select_kernel<2, U>), grid, block, 0, stream, a);
  else if (bound <= 4 * kSelectThreads) hipLaunchKernelGGL((select_kernel<4, U>), grid, block, 0, stream, a);
  else if (bound <= 8 * kSelectThreads) hipLaunchKernelGGL((select_kernel<8, U>), grid, block, 0, stream, a);
  else if (bound <= 16 * kSelectThreads) hipLaunchKernelGGL((select_kernel<16, U>), grid, block, 0, stream, a);
  else if (bound <= 32 * kSelectThreads) hipLaunchKernelGGL((select_kernel<32, U>), grid, block, 0, stream, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace

hipError_t launch_select(const SelectArgs& a, int batch, hipStream_t stream) {
  if (a.unit_tokens == 16) return launch_select_u<16>(a, batch, stream);
  if (a.unit_tokens == 1) return launch_select_u<1>(a, batch, stream);
  return hipErrorInvalidValue;
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

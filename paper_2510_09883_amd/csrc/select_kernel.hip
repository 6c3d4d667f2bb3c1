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
// select_kernel: one 256-thread workgroup per sequence, candidate keys in registers.  Units
//   [n_u - L, n_u) are kept; among
//   the n_u - L older units the (K - L) largest scores are found by an exact radix select on
//   the float bit patterns (non-negative floats order like their uint32 bits): after skipping
//   the leading bits common to all keys, 8-bit digit histograms in LDS narrow the threshold
//   key T down until either every bit is fixed or all keys in the threshold's bin are needed
//   (then the remaining bits cannot change the set), and give how many keys equal to T are
//   needed.  A final pass in index order
//   takes every key > T and the lowest-index keys == T (one block prefix sum), writing them in
//   ascending order.  While n_u <= K every unit is kept.
#include "internal.h"
#include "wave.h"

namespace delta {
namespace {

constexpr float kNegInf = -__builtin_huge_valf();
constexpr int kScoreThreads = 256;
constexpr int kScoreWaves = kScoreThreads / 64;
constexpr int kScoreTokens = 256;   // tokens per scoring workgroup (four per lane)
constexpr int kSelectThreads = 256;
constexpr int kSelectWaves = kSelectThreads / 64;

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

__device__ __forceinline__ uint32_t key_of(float f) {
  return f > 0.f ? __float_as_uint(f) : 0u;   // scores are >= 0; NaN / -0 map to 0
}

// Exclusive prefix sum of one int per thread over the workgroup (one barrier: `s_wave` must not
// be reused by another scan); *total gets the sum.
__device__ __forceinline__ int block_excl_scan(int v, int* s_wave, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int incl = wave_incl_scan(v);
  if (lane == 63) s_wave[w] = incl;
  lds_barrier();
  int base = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < kSelectWaves; ++i) {
    const int c = s_wave[i];
    base += (i < w) ? c : 0;
    tot += c;
  }
  *total = tot;
  return base + incl - v;
}

// One workgroup per sequence.  Thread t owns the candidate keys [t*KPT, t*KPT + KPT) in
// registers, so index order is thread order then slot order and one block scan places every
// chosen unit.  KPT (keys per thread) is chosen on the host from the candidate bound.
// With a.sel_phys, the physical location of every chosen unit (its page, or for U = 1 its
// page * 16 + row) is written beside its index; the page-table entries of the thread's keys are
// loaded together with the keys.
template <int KPT, int U>
__global__ __launch_bounds__(kSelectThreads) void select_kernel(const SelectArgs a) {
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int K = a.budget_units;
  const int L = a.recent_units;
  const int s_b = a.seq_lens[b];
  const int n_u = min((s_b + U - 1) / U, a.nu_stride);
  int32_t* idx_out = a.sel_idx + (size_t)b * K;
  int32_t* phys_out = a.sel_phys ? a.sel_phys + (size_t)b * K : nullptr;
  const int32_t* pt = a.page_table + (size_t)b * a.max_pages;
  auto phys_of = [&](int u) { return U == 16 ? pt[u] : pt[u >> 4] * 16 + (u & 15); };

  const float* S = a.unit_scores + (size_t)b * a.nu_stride;
  const int i0 = tid * KPT;
  // The keys and their page-table entries are requested before the sequence length arrives
  // (indices clamped into the rows, so every load is in bounds): one wait for memory instead of
  // two.  Slots past the candidates are masked once the length is known.
  uint32_t key[KPT];
#pragma unroll
  for (int j = 0; j < KPT; ++j) key[j] = key_of(S[min(i0 + j, a.nu_stride - 1)]);
  // page-table entries of the keys (U = 1: KPT consecutive tokens span at most KPT/16 + 1 pages)
  constexpr int NP = U == 16 ? KPT : (KPT + 15) / 16 + 1;
  int pg[NP];
  if (phys_out) {
#pragma unroll
    for (int j = 0; j < NP; ++j)
      pg[j] = pt[min((U == 16 ? i0 : i0 >> 4) + j, a.max_pages - 1)];
  }

  if (n_u <= K) {   // the context fits the budget: keep every unit
    for (int i = tid; i < K; i += kSelectThreads) {
      idx_out[i] = (i < n_u) ? i : -1;
      if (phys_out) phys_out[i] = (i < n_u) ? phys_of(i) : -1;
    }
    if (tid == 0) a.sel_cnt[b] = max(n_u, 0);
    return;
  }
  const int n_c = min(n_u - L, KPT * kSelectThreads);   // candidate (older) units; the host bounds it
  const int need = K - L;       // >= 1
  const int rec_phys = (phys_out && tid < L) ? phys_of(n_c + tid) : 0;

  // Histograms rotate over three buffers: the one a pass fills was cleared two passes before,
  // so each digit pass needs a single barrier.
  __shared__ uint32_t s_hist[3][256];
  __shared__ int s_wave[kSelectWaves];
  __shared__ uint32_t s_red[2][kSelectWaves];
#pragma unroll
  for (int j = 0; j < KPT; ++j)
    if (!(i0 + j < n_c)) key[j] = 0u;
  s_hist[0][tid] = 0u;   // kSelectThreads == 256 bins
  s_hist[1][tid] = 0u;
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
  k_or = wave_or(k_or);
  k_and = wave_and(k_and);
  if (lane == 0) {
    s_red[0][tid >> 6] = k_or;
    s_red[1][tid >> 6] = k_and;
  }
  lds_barrier();
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
  for (int pass = 0; low > 0; ++pass) {
    const int width = min(8, low);
    const int shift = low - width;
    const int top = shift + width;                    // bits [top, 32) already fixed
    uint32_t* hist = s_hist[pass % 3];
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
      const uint32_t k = key[j];
      const bool match = i0 + j < n_c && (top >= 32 || (k >> top) == (prefix >> top));
      if (match) atomicAdd(&hist[(k >> shift) & ((1u << width) - 1u)], 1u);
    }
    lds_barrier();
    s_hist[(pass + 2) % 3][tid] = 0u;   // for pass + 2 (last read before this pass's barrier)
    // Every wave finds the digit itself: lane l owns digits 255-4l .. 252-4l (descending); the
    // lane where the running count from the top reaches `remaining` holds the threshold digit.
    int c[4], sum = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      c[k] = (int)hist[255 - 4 * lane - k];
      sum += c[k];
    }
    const int incl = wave_incl_scan(sum);
    const int excl = incl - sum;
    int digit = 0, above = 0, count = 0, run = excl;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (run < remaining && remaining <= run + c[k]) {
        digit = 255 - 4 * lane - k;
        above = run;
        count = c[k];
      }
      run += c[k];
    }
    const uint64_t owner = __ballot(excl < remaining && remaining <= incl);
    const int src = __ffsll((unsigned long long)owner) - 1;   // exactly one lane owns it
    digit = __builtin_amdgcn_readlane(digit, src);
    above = __builtin_amdgcn_readlane(above, src);
    count = __builtin_amdgcn_readlane(count, src);
    prefix |= (uint32_t)digit << shift;
    remaining -= above;
    low = shift;
    // Every key of the threshold's bin is needed: the bits below `low` cannot change the set.
    if (count == remaining) break;
  }
  // Keys are compared on their resolved bits [low, 32): T is the need-th largest key's value
  // there, and `remaining` keys with that value are taken (lowest index first).  When every
  // bit is resolved this is the exact threshold key.
  const uint32_t T = prefix >> low;

  // One scan of the packed counts (keys above T in the low half, keys equal to T in the high
  // half; each total is at most 8192) places every taken key: the equal keys are taken lowest
  // index first.
  int n_gt = 0, n_eq = 0;
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    const bool valid = i0 + j < n_c;
    n_gt += valid && (key[j] >> low) > T;
    n_eq += valid && (key[j] >> low) == T;
  }
  int tot;
  const int before = block_excl_scan(n_gt | (n_eq << 16), s_wave, &tot);
  int eq_rank = before >> 16;
  int pos = (before & 0xffff) + min(eq_rank, remaining);
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    const bool valid = i0 + j < n_c;
    bool take = valid && (key[j] >> low) > T;
    if (valid && (key[j] >> low) == T) {
      take = eq_rank < remaining;
      ++eq_rank;
    }
    if (take) {
      if (pos < need) {
        idx_out[pos] = i0 + j;
        if (phys_out)
          phys_out[pos] = U == 16 ? pg[j] : pg[((i0 + j) >> 4) - (i0 >> 4)] * 16 + ((i0 + j) & 15);
      }
      ++pos;
    }
  }
  for (int j = tid; j < L; j += kSelectThreads) {
    idx_out[need + j] = n_c + j;
    if (phys_out) phys_out[need + j] = (j == tid) ? rec_phys : phys_of(n_c + j);
  }
  if (tid == 0) a.sel_cnt[b] = K;
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

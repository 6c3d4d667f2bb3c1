// Page selection of one sequence by one workgroup (Sec. 4 "Selection mechanism" and
// "Page-based DELTA"; App. A, Alg. 2): units [n_u - L, n_u) are kept; among the n_u - L older
// units the (K - L) largest scores are found by an exact radix select on the float bit patterns
// (non-negative floats order like their uint32 bits): after skipping the leading bits common
// to all keys, 8-bit digit histograms in LDS narrow the threshold key T down until either every
// bit is fixed or all keys in the threshold's bin are needed (then the remaining bits cannot
// change the set), and give how many keys equal to T are needed.  A final pass in index order
// takes every key > T and the lowest-index keys == T (one block prefix sum), writing them in
// ascending order.  While n_u <= K every unit is kept.
#pragma once

#include "internal.h"
#include "wave.h"

namespace delta {

constexpr int kSelectThreads = 256;
constexpr int kSelectWaves = kSelectThreads / 64;

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

// Selection for sequence b by one workgroup of kSelectThreads threads.  Thread t owns the
// candidate keys [t*KPT, t*KPT + KPT) in registers, so index order is thread order then slot
// order and one block scan places every chosen unit.  KPT (keys per thread) is chosen on the
// host from the candidate bound.  With a.sel_phys, the physical location of every chosen unit
// (its page, or for U = 1 its page * 16 + row) is written beside its index; the page-table
// entries of the thread's keys are loaded together with the keys.  The unit scores are read
// with device-coherent loads, so they may have been written by other workgroups of the same
// launch (with device-coherent stores) as well as by an earlier launch.
template <int KPT, int U>
__device__ __forceinline__ void select_sequence(const SelectArgs& a, int b) {
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
  for (int j = 0; j < KPT; ++j)
    key[j] = key_of(__hip_atomic_load(S + min(i0 + j, a.nu_stride - 1), __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_AGENT));
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

}  // namespace delta

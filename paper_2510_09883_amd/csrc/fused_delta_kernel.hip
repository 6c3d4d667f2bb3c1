// Fused Delta layer for gfx950: full attention, token/page scoring and page selection of one
// Delta layer (App. A, Alg. 1 Delta branch and Alg. 2 RefreshPages; Sec. 4 "Selection
// mechanism", "Page-based DELTA") in one launch, with the logits kept in LDS.
//
// One workgroup per (chunk of kFusedChunkPages pages, sequence) covers every KV head of the
// chunk: wave w takes KV heads w, w + 4, ... and walks the chunk's pages with the register
// tile ring of the split attention kernel, putting every scaled log2-domain logit into LDS
// ([kv head][page][head in group][16]).  Then:
//   1. each wave stores its chunk partial (max, sum, o) per query head (device-coherent);
//   2. the workgroups of a sequence wait for each other (device-scope counter), for at most
//      a.spin_ticks of the 100 MHz real-time clock;
//   3. every workgroup forms the log-sum-exp of all query heads from the chunk partials (one
//      round trip for all of them);
//   4. workgroup c merges the outputs of heads c, c + n_active, ... in chunk order (n_active:
//      the chunks the sequence has), its loads in flight while it scores;
//   5. every workgroup scores its own tokens from its LDS logits, s_t = 2^(max_j (x_j(t) -
//      lse_j)) (or sum_j 2^(x_j(t) - lse_j)), sums them per page and stores the page scores;
//   6. the last workgroup of the sequence to finish scoring selects for it (select_impl.h).
// A plain launch does not guarantee that all workgroups of a sequence are resident together.
// When they are not (the wait of step 2 runs out), the waiting workgroup skips steps 3-5,
// writes its LDS logits to the workspace and flags its chunk; the sequence's last workgroup
// then does steps 3-5 for every flagged chunk from the workspace before selecting.  The
// arithmetic and its order are the same on both paths, so the results are the same bits; no
// workgroup ever waits without a bound.  When every workgroup is resident the logits never
// reach HBM; the split path (attention kernel + score kernel + select kernel) writes and
// re-reads them.
#include <type_traits>

#include "attn_tile.h"
#include "debug_check.h"
#include "internal.h"
#include "select_impl.h"
#include "wave.h"

namespace delta {
namespace {

constexpr int kWaves = kAttnThreads / 64;
constexpr int kC = kFusedChunkPages;
constexpr int kRawBufferFlags = 0x00020000;   // buffer-resource word 3, raw access (gfx950)
constexpr int kCoherent = 16;                 // device-coherent (sc1) cache policy
// Bound on the polls of the sequence barrier besides its time limit (each poll is a device
// round trip plus a short sleep, so this is about a second).
constexpr int kSpinLimit = 1 << 20;

__device__ __forceinline__ float2 load_ml(const __amdgpu_buffer_rsrc_t& r, int byte_off) {
  return __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(r, byte_off, 0, kCoherent));
}

template <int D, int G, int U>
__global__ __launch_bounds__(kAttnThreads) void fused_delta_kernel(const FusedArgs a) {
  using Gm = Geo<D>;
  constexpr int R = Gm::R;
  const int c = blockIdx.x;
  const int b = blockIdx.y;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int quad = lane >> 4, hcol = lane & 15;
  const int Hq = a.n_q_heads, Hkv = a.n_kv_heads;
  const int s_b = min(a.seq_lens[b], a.max_seq_len);
  const int n_pages = (s_b + 15) >> 4;
  const int n_active = (n_pages + kC - 1) / kC;   // workgroups of this sequence that run
  if (c >= n_active) return;                      // uniform over the workgroup
  const int p0 = c * kC;
  const int np = min(kC, n_pages - p0);

  __shared__ int s_pages[kC];
  __shared__ float s_p[kWaves][16 * 8 + 8];
  __shared__ __attribute__((aligned(16))) float s_logit[kFusedMaxQHeads * kC * 16];
  __shared__ float s_M[kFusedMaxQHeads], s_L[kFusedMaxQHeads], s_lse[kFusedMaxQHeads];
  __shared__ int s_last;
  if (tid < np) s_pages[tid] = checked_page(a.page_table[(size_t)b * a.max_pages + p0 + tid], a.n_pages, a.status);
  if (DELTA_DEBUG && c == 0 && tid == 0 && (a.seq_lens[b] < 1 || a.seq_lens[b] > a.max_seq_len))
    debug_flag(a.status, DELTA_DEBUG_SEQ_LEN);
  float* lp = s_p[wave];

  const size_t part_rows = (size_t)gridDim.y * Hkv * a.n_chunks * G;   // rows of G x D / G x 2
  const __amdgpu_buffer_rsrc_t ro = __builtin_amdgcn_make_buffer_rsrc(
      a.part_o, 0, (int)min(part_rows * D * 4, (size_t)0x7fffffff), kRawBufferFlags);
  const __amdgpu_buffer_rsrc_t rml = __builtin_amdgcn_make_buffer_rsrc(
      a.part_ml, 0, (int)min(part_rows * 8, (size_t)0x7fffffff), kRawBufferFlags);
  lds_barrier();   // page list

  // ---- 1. attention over the chunk -----------------------------------------------------
  for (int g = wave; g < Hkv; g += kWaves) {   // wave-uniform
    bf16x8 qb[Gm::NK];
    load_query<D, G>(qb, a.q, (size_t)b * Hq + g * G, lane);
    WaveSoftmax<G> st;
    st.init();
    const size_t head_off = (size_t)g * 16 * D;
    float* lg = s_logit + (size_t)g * kC * G * 16;
    // ring of R tiles as in the split kernel; prefetches past the chunk are one-line dummies
    auto fetch = [&](Tile<D>& t, int k) {
      const int kk = min(k, np - 1);
      const size_t page = (size_t)s_pages[kk] * a.page_stride + head_off;
      const int nrows = min(16, s_b - 16 * (p0 + kk));
      t.kmask = (nrows >= 16) ? 0xffffu : ((1u << max(nrows, 0)) - 1u);
      load_page_tile<D>(t, a.k_cache + page, a.v_cache + page, k < np, lane);
    };
    Tile<D> t[R];
#pragma unroll
    for (int i = 0; i < R - 1; ++i) fetch(t[i], i);
    for (int k = 0; k < np; k += R) {
#pragma unroll
      for (int r = 0; r < R; ++r) {
        fetch(t[(r + R - 1) % R], k + r + R - 1);
        if (k + r < np)
          process_tile<D, G, true>(t[r], qb, a.scale_log2, st, lp, lg + (k + r) * G * 16, lane);
      }
    }
    reduce_outputs<D, G>(st);
    const int prow = (((b * Hkv + g) * a.n_chunks) + c) * G;   // partial row of head 0
    if (quad == 0 && hcol < G)
      __builtin_amdgcn_raw_buffer_store_b64(
          __builtin_bit_cast(u32x2, make_float2(st.m_run, st.l_run)), rml, (prow + hcol) * 8, 0,
          kCoherent);
    if (lane < Gm::LPR) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const int off = ((prow + h) * D + 8 * lane) * 4;
        __builtin_amdgcn_raw_buffer_store_b128(
            __builtin_bit_cast(u32x4, f32x4{st.o[h][0], st.o[h][1], st.o[h][2], st.o[h][3]}), ro,
            off, 0, kCoherent);
        __builtin_amdgcn_raw_buffer_store_b128(
            __builtin_bit_cast(u32x4, f32x4{st.o[h][4], st.o[h][5], st.o[h][6], st.o[h][7]}), ro,
            off + 16, 0, kCoherent);
      }
    }
  }

  // ---- 2. sequence barrier, bounded in time ----------------------------------------------
  // A workgroup that does not see every chunk of its sequence arrive within a.spin_ticks (the
  // other workgroups are not resident: the launch shares the device, or it is larger than what
  // the device holds at once) does not wait longer: it writes its logits to the workspace and
  // leaves its chunk to the last workgroup of the sequence (step 6).  Either way the results
  // are the same bits.
  __builtin_amdgcn_s_waitcnt(0);   // this thread's partial stores are complete
  __syncthreads();
  __shared__ int s_ok;
  if (tid == 0) {
    // the last workgroup to arrive learns it from its own count and does not poll
    const int before = __hip_atomic_fetch_add(&a.counters[(size_t)b * kCounterStride], 1, __ATOMIC_RELAXED,
                                              __HIP_MEMORY_SCOPE_AGENT);
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    int ok = before + 1 >= n_active;
    for (int it = 0; !ok && it < kSpinLimit; ++it) {
      if (__hip_atomic_load(&a.counters[(size_t)b * kCounterStride], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= n_active) {
        ok = 1;
        break;
      }
      if ((int64_t)(__builtin_amdgcn_s_memrealtime() - t0) >= a.spin_ticks) break;
      __builtin_amdgcn_s_sleep(2);
    }
    s_ok = ok;
  }
  __syncthreads();
  const bool ok = s_ok != 0;

  // ---- 3. log-sum-exp of every query head ------------------------------------------------
  // (max, sum) of the chunk partials in chunk order, all n_active loads in flight at once
  // (n_active <= kFusedMaxChunks).  lse_heads is the work of threads tid < Hq; compute_lse
  // adds the barrier that publishes s_M, s_L and s_lse.
  constexpr int kNc = kFusedMaxChunks;
  auto lse_heads = [&]() {
    if (tid < Hq) {
      const int g = tid / G, h = tid - (tid / G) * G;
      const int row0 = ((b * Hkv + g) * a.n_chunks) * G + h;   // chunk cc: row0 + cc * G
      float2 ml[kNc];
#pragma unroll
      for (int i = 0; i < kNc; ++i) {   // chunks past the sequence's last are not loaded
        ml[i] = make_float2(kNegInfF, 0.f);
        if (i < n_active) ml[i] = load_ml(rml, (row0 + i * G) * 8);
      }
      float M = kNegInfF;
#pragma unroll
      for (int i = 0; i < kNc; ++i)
        if (i < n_active) M = fmaxf(M, ml[i].x);
      const float Mu = (M == kNegInfF) ? 0.f : M;
      float L = 0.f;
#pragma unroll
      for (int i = 0; i < kNc; ++i)
        if (i < n_active) L += (ml[i].x == kNegInfF ? 0.f : exp2f(ml[i].x - Mu)) * ml[i].y;
      s_M[tid] = M;
      s_L[tid] = L;
      s_lse[tid] = M + log2f(L);
    }
  };
  auto compute_lse = [&]() {
    lse_heads();
    __syncthreads();
  };

  // ---- 4. outputs of heads cc, cc + n_active, ... (chunk order: deterministic) -----------
  // Waves 1-3 merge, kQuads threads per head; each pass issues all of its partial loads at
  // once.  mid() runs on every thread once, after the first pass's loads are issued and before
  // they are used: it must leave s_M and s_L published (the log-sum-exp of step 3).
  auto merge_outputs = [&](int cc, auto&& mid) {
    constexpr int kQuads = D / 4;                            // threads per head
    constexpr int kPassHeads = (kAttnThreads - 64) / kQuads;
    const int mt = tid - 64;                                  // merge thread, waves 1-3
    const int dc = 4 * (max(mt, 0) % kQuads);
    const int n_heads = cc < Hq ? (Hq - cc + n_active - 1) / n_active : 0;
    const int n_pass = max(1, (n_heads + kPassHeads - 1) / kPassHeads);   // uniform
    for (int pass = 0; pass < n_pass; ++pass) {
      const int j = mt >= 0 ? cc + n_active * (pass * kPassHeads + mt / kQuads) : Hq;
      const bool act = j < Hq;
      const int g = act ? j / G : 0, h = act ? j - (j / G) * G : 0;
      const int row0 = ((b * Hkv + g) * a.n_chunks) * G + h;
      float m[kNc];
      f32x4 ov[kNc];
      if (act) {
#pragma unroll
        for (int i = 0; i < kNc; ++i) {
          m[i] = kNegInfF;
          ov[i] = f32x4{0.f, 0.f, 0.f, 0.f};
          if (i < n_active) {
            const int row = row0 + i * G;
            m[i] = load_ml(rml, row * 8).x;
            ov[i] = __builtin_bit_cast(
                f32x4, __builtin_amdgcn_raw_buffer_load_b128(ro, (row * D + dc) * 4, 0, kCoherent));
          }
        }
      }
      if (pass == 0) mid();
      if (act) {
        const float Mj = s_M[j];
        f32x4 O = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < kNc; ++i)
          if (i < n_active) O += (m[i] == kNegInfF ? 0.f : exp2f(m[i] - Mj)) * ov[i];
        const float lsum = s_L[j];
        uint2 packed;
        packed.x = (uint32_t)f32_to_bf16_rne(O[0] / lsum) | ((uint32_t)f32_to_bf16_rne(O[1] / lsum) << 16);
        packed.y = (uint32_t)f32_to_bf16_rne(O[2] / lsum) | ((uint32_t)f32_to_bf16_rne(O[3] / lsum) << 16);
        *reinterpret_cast<uint2*>(a.out + ((size_t)b * Hq + j) * D + dc) = packed;
      }
    }
  };

  // ---- 5. scores of chunk cc's tokens, from this workgroup's LDS logits or from the
  // workspace copy a timed-out workgroup left (layout [b][kv head][page][head in group][16])
  auto score_chunk = [&](int cc, bool from_lds) {
    const int pc = cc * kC;
    const int npc = min(kC, n_pages - pc);
    const int k = tid >> 2;           // page of the chunk (kC * 4 == kAttnThreads)
    const int r0 = 4 * (tid & 3);     // its rows r0 .. r0 + 3
    const int t0 = (pc + k) * 16 + r0;
    // x_j(t) - lse_j folded over the query heads in (KV head, head in group) order; the
    // reduction (max, or sum of 2^) is fixed at compile time so the loop carries no branch,
    // and a KV head's G logit reads are issued together
    auto fold = [&](auto max_mode, float (&acc)[4]) {
      constexpr bool kMax = decltype(max_mode)::value;
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[i] = kMax ? kNegInfF : 0.f;
      if (k >= npc) return;
      for (int g = 0; g < Hkv; ++g) {
        const float* glog = a.logits + (((size_t)b * Hkv + g) * a.logit_pages + pc + k) * G * 16 + r0;
        f32x4 x[G];
        float l[G];
#pragma unroll
        for (int h = 0; h < G; ++h) {
          l[h] = s_lse[g * G + h];
          if (from_lds) {
            x[h] = *reinterpret_cast<const f32x4*>(&s_logit[(((size_t)g * kC + k) * G + h) * 16 + r0]);
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i)
              x[h][i] = __hip_atomic_load(glog + h * 16 + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          }
        }
#pragma unroll
        for (int h = 0; h < G; ++h)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            acc[i] = kMax ? fmaxf(acc[i], x[h][i] - l[h]) : acc[i] + exp2f(x[h][i] - l[h]);
      }
    };
    float acc[4], sc[4];
    if (a.agg == 0) {
      fold(std::true_type{}, acc);
#pragma unroll
      for (int i = 0; i < 4; ++i) sc[i] = (k < npc && t0 + i < s_b) ? exp2f(acc[i]) : 0.f;
    } else {
      fold(std::false_type{}, acc);
#pragma unroll
      for (int i = 0; i < 4; ++i) sc[i] = (k < npc && t0 + i < s_b) ? acc[i] : 0.f;
    }
    float* S = a.unit_scores + (size_t)b * a.sel.nu_stride;
    if (U == 16) {
      float p = (sc[0] + sc[1]) + (sc[2] + sc[3]);
      p += lane_xor1(p);
      p += lane_xor2(p);
      if ((tid & 3) == 0 && k < npc)
        __hip_atomic_store(S + pc + k, p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (k < npc && t0 + i < s_b)
          __hip_atomic_store(S + t0 + i, sc[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  };

  int32_t* deferred = a.chunk_flags + (size_t)b * a.n_chunks;
  // counts this workgroup in for step 6 once its stores are complete (s_last: it is the last)
  auto arrive = [&]() {
    __builtin_amdgcn_s_waitcnt(0);   // this thread's score / logit / flag stores are complete
    __syncthreads();
    if (tid == 0)
      s_last = __hip_atomic_fetch_add(&a.counters[(size_t)b * kCounterStride + 32], 1, __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_AGENT) == n_active - 1;
  };
  if (ok) {
    // the log-sum-exp loads (wave 0) and the first merge pass's loads (waves 1-3) are in flight
    // together; the chunk is scored before the merge arithmetic, so the page scores leave
    // first, and the workgroup counts itself in for the selection as soon as they are complete
    // (the merge's loads are complete by then too; its output stores are not waited for)
    merge_outputs(c, [&]() {
      lse_heads();
      lds_barrier();   // s_M, s_L, s_lse; the merge loads stay in flight
      score_chunk(c, true);
      arrive();
    });
  } else {
    // leave the chunk to the sequence's last workgroup: its logits go to the workspace
    for (int g = 0; g < Hkv; ++g) {
      float* dst = a.logits + (((size_t)b * Hkv + g) * a.logit_pages + p0) * G * 16;
      const float* src = s_logit + (size_t)g * kC * G * 16;
      for (int i = tid; i < np * G * 16; i += kAttnThreads)
        __hip_atomic_store(dst + i, src[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (tid == 0) {
      __hip_atomic_store(deferred + c, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&a.counters[(size_t)b * kCounterStride + 48], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }

  // ---- 6. the last workgroup of the sequence finishes left chunks and selects --------------
  if (!ok) arrive();
  __syncthreads();
  if (!s_last) return;
  // every workgroup of the sequence has arrived (so every partial is stored) and has either
  // scored its chunk or left it
  __shared__ int s_flag;
  if (tid == 0) s_flag = __hip_atomic_load(&a.counters[(size_t)b * kCounterStride + 48], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  if (s_flag) {
    if (!ok) compute_lse();
    for (int cc = 0; cc < n_active; ++cc) {
      if (tid == 0) s_flag = __hip_atomic_load(deferred + cc, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __syncthreads();
      if (s_flag) {
        merge_outputs(cc, []() {});
        score_chunk(cc, false);
        if (tid == 0) __hip_atomic_store(deferred + cc, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      __syncthreads();
    }
    __builtin_amdgcn_s_waitcnt(0);   // the scores written here are complete before selecting
    __syncthreads();
  }
  select_sequence<kFusedKeysPerThread, U>(a.sel, b);
  if (tid == 0) {
    __hip_atomic_store(&a.counters[(size_t)b * kCounterStride], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&a.counters[(size_t)b * kCounterStride + 32], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&a.counters[(size_t)b * kCounterStride + 48], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

static_assert(kC * 4 == kAttnThreads, "scoring gives every thread four tokens of the chunk");

template <int G, int U>
const void* kernel_of() {
  return reinterpret_cast<const void*>(&fused_delta_kernel<128, G, U>);
}

const void* fused_kernel(int group, int unit_tokens) {
  if (unit_tokens != 16 && unit_tokens != 1) return nullptr;
  const bool pages = unit_tokens == 16;
  switch (group) {
    case 1: return pages ? kernel_of<1, 16>() : kernel_of<1, 1>();
    case 2: return pages ? kernel_of<2, 16>() : kernel_of<2, 1>();
    case 3: return pages ? kernel_of<3, 16>() : kernel_of<3, 1>();
    case 4: return pages ? kernel_of<4, 16>() : kernel_of<4, 1>();
    case 5: return pages ? kernel_of<5, 16>() : kernel_of<5, 1>();
    case 6: return pages ? kernel_of<6, 16>() : kernel_of<6, 1>();
    case 7: return pages ? kernel_of<7, 16>() : kernel_of<7, 1>();
    case 8: return pages ? kernel_of<8, 16>() : kernel_of<8, 1>();
    default: return nullptr;
  }
}

}  // namespace

int fused_delta_capacity(int head_dim, int group, int unit_tokens) {
  const void* k = head_dim == 128 ? fused_kernel(group, unit_tokens) : nullptr;
  if (!k) return 0;
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k, kAttnThreads, 0) != hipSuccess) return 0;
  return per_cu * cus;
}

hipError_t launch_fused_delta(int head_dim, int group, const FusedArgs& a, int batch,
                              hipStream_t stream) {
  const void* k = head_dim == 128 ? fused_kernel(group, a.sel.unit_tokens) : nullptr;
  if (!k) return hipErrorInvalidValue;
  switch (group) {
#define DELTA_FUSED_CASE(GG)                                                                  \
  case GG:                                                                                    \
    if (a.sel.unit_tokens == 16)                                                              \
      hipLaunchKernelGGL((fused_delta_kernel<128, GG, 16>), dim3(a.n_chunks, batch),          \
                         dim3(kAttnThreads), 0, stream, a);                                   \
    else                                                                                      \
      hipLaunchKernelGGL((fused_delta_kernel<128, GG, 1>), dim3(a.n_chunks, batch),           \
                         dim3(kAttnThreads), 0, stream, a);                                   \
    break;
    DELTA_FUSED_CASE(1) DELTA_FUSED_CASE(2) DELTA_FUSED_CASE(3) DELTA_FUSED_CASE(4)
    DELTA_FUSED_CASE(5) DELTA_FUSED_CASE(6) DELTA_FUSED_CASE(7) DELTA_FUSED_CASE(8)
#undef DELTA_FUSED_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace delta

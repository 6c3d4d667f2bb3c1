// Split-K paged decode attention for gfx950, in three row modes (full / Delta / sparse).
//
// What it computes (Sec. 2, Eq. gqa_attention; App. A, Alg. 1): for sequence b and query
// head j, out = sum_t softmax_t(scale * q_j . k_t) v_t over the rows of the sequence that the
// mode selects, with k_t, v_t read from KV head j / G.  With logits on (Delta layers) the
// scaled logits of every token (group-major: [b][kv group][page][head in group][row]) and the
// per-head log-sum-exp are also written, for the page scoring of Sec. 4 ("Selection
// mechanism", "Page-based DELTA").
//
// Work decomposition.  One workgroup (4 waves) per (split, kv head g, sequence b).  A split
// is a run of `gps` groups of 16 rows; a group is one 16-token page tile [16, D] of K and of
// V (4 KB each at D = 128, contiguous in HBM), or 16 gathered token rows in token-level
// sparse mode.  Waves take the split's groups in interleaved blocks of four and keep their
// own online-softmax state; all G query heads of the KV group share every K/V byte read.
//
// Per group and wave:
//   * QK^T on the matrix cores: v_mfma_f32_16x16x32_bf16 with A = the 16 K rows (M = rows,
//     K = head dim) and B = the G query vectors padded to 16 columns; D/32 MFMAs give the
//     16 x 16 score tile, lane l holding rows 4*(l/16)..+3 of head column l%16.
//   * online softmax in the log2 domain (exp2, scale folded with log2 e); the group's
//     probabilities and the per-head rescale factor go through a wave-private LDS slice;
//   * P.V on the vector ALUs: each lane owns 8 consecutive head-dim columns of 16/RPI rows
//     (128-bit loads, one V row per LPR consecutive lanes, fully coalesced).
//   Each wave keeps a ring of R register tiles: while one group is consumed, the K/V loads of
//   the next R - 1 groups are in flight.  With logits on, the logits of a chunk of groups are
//   staged in LDS and written by the whole workgroup between chunks.
//
// Split combine.  The 4 waves merge through LDS into one (max, sum, o) partial per split,
// written to the workspace with device-coherent stores.  The last workgroup of each (b, g) to
// arrive (device-scope atomic counter) loads every split's partial at once into registers,
// merges them in split order — a fixed order, so results do not depend on arrival order — writes bf16
// outputs (and the log-sum-exp), and re-arms the counter to zero for the next launch.  A
// sequence that fits one split skips all of this and writes its outputs directly.
#include "attn_tile.h"
#include "internal.h"
#include "wave.h"

namespace delta {
namespace {

constexpr int kWaves = kAttnThreads / 64;
constexpr float kNegInf = kNegInfF;
// Buffer-resource word 3 for raw (unformatted, stride 0) buffer access on gfx950, and the
// cache-policy operand of the buffer builtins that selects the device-coherent (sc1) policy.
constexpr int kRawBufferFlags = 0x00020000;
constexpr int kCoherent = 16;
// LDS floats for staging Delta-layer logits (128 KB: one Delta workgroup per CU; measured on
// MI355X, fewer and larger chunk flushes beat two resident workgroups with half the staging).
constexpr int kStageFloats = 32768;

template <int D, int G, int MODE, bool LOGITS>
__global__ __launch_bounds__(kAttnThreads) void attn_kernel(const AttnArgs a) {
  using Gm = Geo<D>;
  constexpr int R = Gm::R;
  const int split = blockIdx.x;
  const int g = blockIdx.y;
  const int b = blockIdx.z;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform (scalar)
  const int quad = lane >> 4;   // score-tile rows 4*quad .. 4*quad+3
  const int hcol = lane & 15;   // score-tile column = query head within the group
  const int Hq = a.n_q_heads;
  const int bg = b * a.n_kv_heads + g;

  // ---- start-up: the query operand, the sequence length / selection count and this split's
  // page (or row) list are all requested at once; the list is staged in LDS speculatively
  // (bounded by the host's group bound) and trimmed once the length is known.
  bf16x8 qb[Gm::NK];
  load_query<D, G>(qb, a.q, (size_t)b * Hq + g * G, lane);
  const int s_b = a.seq_lens[b];
  const int sel_n = (MODE == ROWS_DENSE) ? 0 : min(a.sel_cnt[b], a.sel_stride);
  const int g0 = split * a.gps;
  const int cand = max(0, min(a.gps, a.max_groups - g0));

  __shared__ int s_rows[kMaxRowSlots];
  __shared__ int s_aux[MODE == ROWS_SEL_PAGE ? kMaxRowSlots : 1];
  const int32_t* pt = a.page_table + (size_t)b * a.max_pages;
  if (MODE == ROWS_DENSE) {
    for (int i = tid; i < cand; i += kAttnThreads) s_rows[i] = pt[g0 + i];
  } else if (MODE == ROWS_SEL_PAGE) {
    // with precomputed physical pages the index and the page arrive together
    const int32_t* sel = a.sel_idx + (size_t)b * a.sel_stride;
    const int32_t* phys = a.sel_phys ? a.sel_phys + (size_t)b * a.sel_stride : nullptr;
    for (int i = tid; i < cand; i += kAttnThreads) {
      const int u = sel[g0 + i];
      const int ph = phys ? phys[g0 + i] : 0;
      const bool ok = u >= 0 && u < a.max_pages;
      s_rows[i] = ok ? (phys ? ph : pt[u]) : 0;
      s_aux[i] = ok ? u : 0;
    }
  } else {
    const int32_t* sel = a.sel_idx + (size_t)b * a.sel_stride;
    const int32_t* phys = a.sel_phys ? a.sel_phys + (size_t)b * a.sel_stride : nullptr;
    const int n_rows = min(16 * cand, a.sel_stride - 16 * g0);
    for (int i = tid; i < 16 * cand; i += kAttnThreads) {
      int packed = -1;
      if (i < n_rows) {
        const int t = sel[16 * g0 + i];
        const int ph = phys ? phys[16 * g0 + i] : 0;
        if (t >= 0 && t < 16 * a.max_pages) packed = phys ? ph : pt[t >> 4] * 16 + (t & 15);
      }
      s_rows[i] = packed;
    }
  }

  int n_groups;
  if (MODE == ROWS_DENSE) n_groups = (s_b + 15) >> 4;
  else if (MODE == ROWS_SEL_PAGE) n_groups = sel_n;
  else n_groups = (sel_n + 15) >> 4;
  // lengths beyond the host bound are clamped so that no access leaves the buffers
  n_groups = max(0, min(n_groups, a.max_groups));
  const int n_valid = (n_groups + a.gps - 1) / a.gps;

  if (n_valid == 0) {  // nothing to attend to: defined output (zeros), log-sum-exp = -inf
    if (split == 0) {
      for (int i = tid; i < G * D; i += kAttnThreads)
        a.out[((size_t)b * Hq + g * G) * D + i] = 0;
      if (LOGITS && tid < G) a.lse[(size_t)b * Hq + g * G + tid] = kNegInf;
    }
    return;
  }
  if (split >= n_valid) return;
  const int ng = min(a.gps, n_groups - g0);
  lds_barrier();   // the page / row list is in LDS; the query loads may still be in flight

  const size_t head_off = (size_t)g * 16 * D;
  // Loads tile `li` of the split.  A prefetch past the wave's last group (real == false) is
  // still issued, so that the loop's memory waits stay uniform, but with every lane at the
  // tile's first 16 bytes: one cache line per load instruction instead of a whole tile.
  auto load_tile = [&](Tile<D>& t, int li, bool real) {
    if (MODE == ROWS_SEL_TOKEN) {
      // every row is its own (page, row); rows past the selection re-read the group's first
      const int* rows = s_rows + 16 * li;
      const int base = 16 * (g0 + li);
      const int first = rows[0];
      t.kmask = 0;
#pragma unroll
      for (int r = 0; r < 16; ++r) t.kmask |= ((rows[r] >= 0 && base + r < sel_n) ? 1u : 0u) << r;
      const int kr = ((t.kmask >> hcol) & 1u) && real ? rows[hcol] : first;
      const uint16_t* kp = a.k_cache + (size_t)(kr >> 4) * a.page_stride + head_off +
                           (size_t)(kr & 15) * D + (real ? 8 * quad : 0);
#pragma unroll
      for (int ks = 0; ks < Gm::NK; ++ks) t.k[ks] = load16_stream(kp + (real ? 32 * ks : 0));
#pragma unroll
      for (int i = 0; i < Gm::NI; ++i) {
        const int r = Gm::RPI * i + lane / Gm::LPR;
        const int vr = ((t.kmask >> r) & 1u) && real ? rows[r] : first;
        t.v[i] = load16_stream(a.v_cache + (size_t)(vr >> 4) * a.page_stride + head_off +
                        (size_t)(vr & 15) * D + (real ? 8 * (lane % Gm::LPR) : 0));
      }
    } else {
      const size_t page = (size_t)s_rows[li] * a.page_stride + head_off;
      const int unit = (MODE == ROWS_DENSE) ? g0 + li : s_aux[li];
      const int nrows = min(16, s_b - 16 * unit);
      t.kmask = (nrows >= 16) ? 0xffffu : ((1u << max(nrows, 0)) - 1u);
      load_page_tile<D>(t, a.k_cache + page, a.v_cache + page, real, lane);
    }
  };

  // wave-private LDS slice: P[16 rows][8 heads] and the per-head rescale factor
  __shared__ float s_p[kWaves][16 * 8 + 8];
  float* lp = s_p[wave];

  WaveSoftmax<G> st;
  st.init();

  const int Hq_row = b * Hq + g * G;
  // Logits on: the workgroup keeps the logits of a chunk of kChunk groups in LDS ([group]
  // [head][16], the global layout) and writes the chunk out cooperatively between chunks, with
  // non-temporal (streaming) stores.  Measured on MI355X, logit stores interleaved with the
  // K/V read stream cost several times their bytes, while the same bytes written in a few large
  // streaming bursts (reads paused) cost about their share.  A chunk is a multiple of 16 groups.
  constexpr int kChunk = (kStageFloats / (G * 16)) / 16 * 16;
  __shared__ __attribute__((aligned(16))) float s_stage[LOGITS ? kChunk * G * 16 : 1];
  auto process = [&](const Tile<D>& t, int slot) {
    process_tile<D, G, LOGITS>(t, qb, a.scale_log2, st, lp, s_stage + slot * G * 16, lane);
  };

  // Waves interleave in blocks of four groups (wave w takes groups 16j + 4w .. 16j + 4w + 3),
  // so the workgroup streams about sixteen adjacent pages at a time.  A wave walks its groups
  // [kb, ke) with a ring of R register tiles: tile k lives in slot k % R, and while it is
  // consumed the loads of tiles k + 1 .. k + R - 1 are in flight.  Every load is issued
  // unconditionally (a prefetch past ke is a one-line dummy read of the range's last group)
  // and the loop has no other exits, so the compiler's wait for tile k never drains the
  // younger loads.  With logits on, the groups are walked in chunks with the ring drained at
  // each chunk end; the chunk loop is uniform over the workgroup (its barriers are reached by
  // every wave).
  {
    auto group_of = [&](int k) { return 16 * (k >> 2) + 4 * wave + (k & 3); };
    const int full_blocks = ng / 16, rem = ng - 16 * full_blocks;
    const int n_mine = 4 * full_blocks + min(4, max(0, rem - 4 * wave));
    auto walk = [&](int kb, int ke, int c0) {
      if (kb >= ke) return;
      auto fetch = [&](Tile<D>& t, int k) { load_tile(t, group_of(min(k, ke - 1)), k < ke); };
      Tile<D> t[R];
#pragma unroll
      for (int i = 0; i < R - 1; ++i) fetch(t[i], kb + i);
      for (int k = kb; k < ke; k += R) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
          fetch(t[(r + R - 1) % R], k + r + R - 1);
          if (k + r < ke) process(t[r], group_of(k + r) - c0);
        }
      }
    };
    if (!LOGITS) {
      walk(0, n_mine, 0);
    } else {
      for (int c0 = 0; c0 < ng; c0 += kChunk) {
        // this wave's groups in [c0, c0 + kChunk): a whole number of blocks of 16 except in
        // the last chunk
        const int kb = (c0 / 16) * 4;
        const int ke = min(n_mine, ((c0 + kChunk) / 16) * 4);
        walk(kb, ke, c0);
        // chunk [c0, c0 + n) goes to [b][kv group][page g0 + c0 ...][head][16], contiguous
        lds_barrier();
        const int n = min(kChunk, ng - c0) * G * 16;
        float* dst = a.logits + (((size_t)b * a.n_kv_heads + g) * a.logit_pages + g0 + c0) * G * 16;
        for (int i = 4 * tid; i < n; i += 4 * kAttnThreads)
          __builtin_nontemporal_store(*reinterpret_cast<const f32x4*>(s_stage + i),
                                      reinterpret_cast<f32x4*>(dst + i));
        lds_barrier();
      }
    }
  }

  // ---- reduce o over the lanes that share a head-dim chunk -------------------------------
  reduce_outputs<D, G>(st);

  // ---- merge the 4 waves into one split partial ------------------------------------------
  __shared__ float s_m[kWaves][kMaxGroup], s_l[kWaves][kMaxGroup];
  __shared__ __attribute__((aligned(16))) float s_o[kWaves][G][D];
  static_assert(G * D <= 4 * kAttnThreads && D % 4 == 0, "four outputs per thread cover a group");
  if (quad == 0 && hcol < G) {
    s_m[wave][hcol] = st.m_run;
    s_l[wave][hcol] = st.l_run;
  }
  if (lane < Gm::LPR) {
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) s_o[wave][h][8 * lane + e] = st.o[h][e];
  }
  lds_barrier();

  // From here on thread t owns the four consecutive outputs e0 = 4t .. 4t+3 of head h (D is a
  // multiple of 4, G * D <= 1024 = 4 * kAttnThreads), so every partial, output and merge access
  // is one 16- or 8-byte access and each thread needs the running max and sum of one head.
  const int e0 = 4 * tid;
  const bool owner = e0 < G * D;
  const int h = owner ? e0 / D : 0;
  const int dc = owner ? e0 % D : 0;
  float M = kNegInf, L = 0.f;
  f32x4 O = {0.f, 0.f, 0.f, 0.f};
  if (owner) {
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, s_m[w][h]);
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float f = (s_m[w][h] == kNegInf) ? 0.f : exp2f(s_m[w][h] - M);
      const f32x4 ow = *reinterpret_cast<const f32x4*>(&s_o[w][h][dc]);
      O += f * ow;
      L += f * s_l[w][h];
    }
  }
  auto store_out = [&](const f32x4& v, float lsum, float mx) {
    uint2 packed;
    packed.x = (uint32_t)f32_to_bf16_rne(v[0] / lsum) | ((uint32_t)f32_to_bf16_rne(v[1] / lsum) << 16);
    packed.y = (uint32_t)f32_to_bf16_rne(v[2] / lsum) | ((uint32_t)f32_to_bf16_rne(v[3] / lsum) << 16);
    *reinterpret_cast<uint2*>(a.out + (size_t)(Hq_row + h) * D + dc) = packed;
    if (LOGITS && dc == 0) a.lse[(size_t)Hq_row + h] = mx + log2f(lsum);
  };

  // A sequence with a single split needs no combine: the workgroup writes the output itself.
  if (n_valid == 1) {
    if (owner) store_out(O, L, M);
    return;
  }

  // ---- split combine --------------------------------------------------------------------
  // Partials are written and read only with device-coherent accesses (the sc1 cache policy:
  // written through to memory, and read past any stale copy in another XCD's L2), so no L2
  // write-back or invalidation is needed to publish them.  Each thread waits until its partial
  // stores are complete, the barrier makes that true for the whole workgroup, and only then
  // does one thread count the workgroup in with a device-scope atomic; the workgroup that
  // brings the count to n_valid reads every partial after the atomic has returned.  (A
  // release/acquire fence pair would instead write back and invalidate the whole L2 of the
  // XCD once per workgroup; measured on MI355X that serialises launches of many workgroups.)
  const int pair_floats = a.n_split * G * D;
  const __amdgpu_buffer_rsrc_t po = __builtin_amdgcn_make_buffer_rsrc(
      a.part_o + (size_t)bg * pair_floats, 0, pair_floats * 4, kRawBufferFlags);
  const __amdgpu_buffer_rsrc_t pml = __builtin_amdgcn_make_buffer_rsrc(
      a.part_ml + (size_t)bg * a.n_split * G * 2, 0, a.n_split * G * 8, kRawBufferFlags);
  const int o_off = (h * D + dc) * 4;   // this thread's bytes inside one split's G x D block
  if (owner) {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, O), po, o_off,
                                           split * G * D * 4, kCoherent);
    if (dc == 0)
      __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, make_float2(M, L)), pml,
                                            h * 8, split * G * 8, kCoherent);
  }
  __builtin_amdgcn_s_waitcnt(0);   // this thread's partial stores are complete
  __syncthreads();
  __shared__ int s_last;
  if (tid == 0) {
    const int prev = __hip_atomic_fetch_add(&a.counters[bg], 1, __ATOMIC_RELAXED,
                                            __HIP_MEMORY_SCOPE_AGENT);
    s_last = prev == n_valid - 1;
  }
  __syncthreads();
  if (!s_last || !owner) return;

  // Every owner thread loads its head's (max, sum) and its four outputs of kMergeBatch splits
  // at once (one wait for memory per batch, a single batch up to kMergeBatch splits) and folds
  // them into a running (max, sum, o) in split order: the result does not depend on the order
  // in which workgroups finished.
  constexpr int kMergeBatch = 16;
  M = kNegInf;
  L = 0.f;
  O = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int c0 = 0; c0 < n_valid; c0 += kMergeBatch) {
    float2 ml[kMergeBatch];
    f32x4 pv[kMergeBatch];
#pragma unroll
    for (int c = 0; c < kMergeBatch; ++c) {
      const int cc = min(c0 + c, n_valid - 1);
      ml[c] = __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(pml, h * 8, cc * G * 8, kCoherent));
      pv[c] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(po, o_off, cc * G * D * 4, kCoherent));
    }
    float bm = kNegInf;
#pragma unroll
    for (int c = 0; c < kMergeBatch; ++c)
      if (c0 + c < n_valid) bm = fmaxf(bm, ml[c].x);
    const float Mn = fmaxf(M, bm);
    const float Mu = (Mn == kNegInf) ? 0.f : Mn;
    const float rs = exp2f(M - Mu);   // 0 while nothing has been folded in (M = -inf)
    L *= rs;
    O *= rs;
#pragma unroll
    for (int c = 0; c < kMergeBatch; ++c) {
      if (c0 + c < n_valid) {
        const float f = (ml[c].x == kNegInf) ? 0.f : exp2f(ml[c].x - Mu);
        L += f * ml[c].y;
        O += f * pv[c];
      }
    }
    M = Mn;
  }
  store_out(O, L, M);
  if (tid == 0) __hip_atomic_store(&a.counters[bg], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int D, int G>
hipError_t launch_dg(int mode, const AttnArgs& a, int batch, hipStream_t stream) {
  const dim3 grid(a.n_split, a.n_kv_heads, batch), block(kAttnThreads);
  switch (mode) {
    case ROWS_DENSE:
      if (a.logits) hipLaunchKernelGGL((attn_kernel<D, G, ROWS_DENSE, true>), grid, block, 0, stream, a);
      else hipLaunchKernelGGL((attn_kernel<D, G, ROWS_DENSE, false>), grid, block, 0, stream, a);
      break;
    case ROWS_SEL_PAGE: hipLaunchKernelGGL((attn_kernel<D, G, ROWS_SEL_PAGE, false>), grid, block, 0, stream, a); break;
    case ROWS_SEL_TOKEN: hipLaunchKernelGGL((attn_kernel<D, G, ROWS_SEL_TOKEN, false>), grid, block, 0, stream, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int D>
hipError_t launch_d(int group, int mode, const AttnArgs& a, int batch, hipStream_t stream) {
  switch (group) {
    case 1: return launch_dg<D, 1>(mode, a, batch, stream);
    case 2: return launch_dg<D, 2>(mode, a, batch, stream);
    case 3: return launch_dg<D, 3>(mode, a, batch, stream);
    case 4: return launch_dg<D, 4>(mode, a, batch, stream);
    case 5: return launch_dg<D, 5>(mode, a, batch, stream);
    case 6: return launch_dg<D, 6>(mode, a, batch, stream);
    case 7: return launch_dg<D, 7>(mode, a, batch, stream);
    case 8: return launch_dg<D, 8>(mode, a, batch, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_attention(int head_dim, int group, int mode, const AttnArgs& a, int batch,
                            hipStream_t stream) {
  if (head_dim == 128) return launch_d<128>(group, mode, a, batch, stream);
  if (head_dim == 64) return launch_d<64>(group, mode, a, batch, stream);
  return hipErrorInvalidValue;
}

}  // namespace delta

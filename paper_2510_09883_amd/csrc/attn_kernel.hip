// Split-K paged decode attention for gfx950, in three row modes (full / Delta / sparse).
//
// What it computes (Sec. 2, Eq. gqa_attention; App. A, Alg. 1): for sequence b and query
// head j, out = sum_t softmax_t(scale * q_j . k_t) v_t over the rows of the sequence that the
// mode selects, with k_t, v_t read from KV head j / G.  With logits on (Delta layers) the
// scaled logits of every token (group-major: [b][kv group][page][head in group][row]) and the
// per-head log-sum-exp are also written, for the page scoring of Sec. 4 ("Selection
// mechanism", "Page-based DELTA").
//
// Work decomposition.  A group is one 16-token page tile [16, D] of K and of V (4 KB each at
// D = 128, contiguous in HBM), or 16 gathered token rows in token-level sparse mode.  The grid
// is (split, kv head g, sequence b), 4 waves per workgroup.  Statically, workgroup (split, g,
// b) takes the run of `gps` groups starting at split * gps of pair (b, g).  A dense launch
// (full / Delta layers) over a ragged batch of 2-64 sequences instead cuts the batch's actual
// groups, in (b, g, page) order, into equal runs, one per workgroup, each run possibly
// spanning pairs, so that every CU gets the same work whatever the spread of sequence
// lengths; with equal or nearly equal lengths the static cut is kept.  Waves take a piece's groups in interleaved blocks of four and keep their
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
// Combine.  The 4 waves merge through LDS into one (max, sum, o) partial per piece, written to
// the workspace with device-coherent stores.  The last workgroup of each (b, g) to arrive
// (device-scope atomic counter) loads every piece's partial at once into registers, merges
// them in piece order — a fixed order, so results do not depend on arrival order — writes bf16
// outputs (and the log-sum-exp), and re-arms the counter to zero for the next launch.  A pair
// that is one piece skips all of this and has its outputs written directly.
#include "attn_tile.h"
#include "debug_check.h"
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

template <int D, int G, int MODE, bool LOGITS, bool BAL>
__global__ __launch_bounds__(kAttnThreads) void attn_kernel(const AttnArgs a) {
  using Gm = Geo<D>;
  constexpr int R = Gm::R;
  // (not const: the piece loop below makes them opaque once per piece)
  int tid = threadIdx.x;
  int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform (scalar)
  int quad = lane >> 4;   // score-tile rows 4*quad .. 4*quad+3
  int hcol = lane & 15;   // score-tile column = query head within the group
  const int Hq = a.n_q_heads;

  // ---- staging of a piece of work: the query operand and the page (or row) list of groups
  // [g0, g0 + cand) of (sequence b, KV head g), requested at once; the list goes to LDS.
  bf16x8 qb[Gm::NK];
  __shared__ int s_rows[kMaxRowSlots];
  __shared__ int s_aux[MODE == ROWS_SEL_PAGE ? kMaxRowSlots : 1];
  // (Debug builds check every physical page and selected unit here and flag bad ones; see
  // checked_page.)
  auto stage = [&](int b, int g, int g0, int cand) {
    load_query<D, G>(qb, a.q, (size_t)b * Hq + g * G, lane);
    const int32_t* pt = a.page_table + (size_t)b * a.max_pages;
    // debug builds: the sequence's length bounds its selected units (release: unused)
    const int s_dbg = DELTA_DEBUG && MODE != ROWS_DENSE ? a.seq_lens[b] : 0;
    if (MODE == ROWS_DENSE) {
      for (int i = tid; i < cand; i += kAttnThreads)
        s_rows[i] = checked_page(pt[g0 + i], a.n_pages, a.status);
    } else if (MODE == ROWS_SEL_PAGE) {
      // with precomputed physical pages the index and the page arrive together
      const int32_t* sel = a.sel_idx + (size_t)b * a.sel_stride;
      const int32_t* phys = a.sel_phys ? a.sel_phys + (size_t)b * a.sel_stride : nullptr;
      for (int i = tid; i < cand; i += kAttnThreads) {
        const int u = sel[g0 + i];
        const int ph = phys ? phys[g0 + i] : 0;
        const bool ok = u >= 0 && u < a.max_pages;
        if (DELTA_DEBUG && u >= 0 && 16 * u >= s_dbg) debug_flag(a.status, DELTA_DEBUG_SELECTION);
        s_rows[i] = ok ? checked_page(phys ? ph : pt[u], a.n_pages, a.status) : 0;
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
          if (DELTA_DEBUG && t >= s_dbg) debug_flag(a.status, DELTA_DEBUG_SELECTION);
          if (t >= 0 && t < 16 * a.max_pages) {
            const int page = checked_page(phys ? ph >> 4 : pt[t >> 4], a.n_pages, a.status);
            packed = page * 16 + (phys ? ph & 15 : t & 15);
          }
        }
        s_rows[i] = packed;
      }
    }
  };
  // nothing to attend to (an empty sequence, or no selected unit): defined output (zeros),
  // log-sum-exp = -inf
  auto write_empty = [&](int b, int g) {
    for (int i = tid; i < G * D; i += kAttnThreads) a.out[((size_t)b * Hq + g * G) * D + i] = 0;
    if (LOGITS && tid < G) a.lse[(size_t)b * Hq + g * G + tid] = kNegInf;
  };

  // shared state of the attention of one piece
  __shared__ float s_p[kWaves][16 * 8 + 8];   // wave-private: P[16 rows][8 heads], rescale
  constexpr int kChunk = (kStageFloats / (G * 16)) / 16 * 16;
  __shared__ __attribute__((aligned(16))) float s_stage[LOGITS ? kChunk * G * 16 : 1];
  __shared__ float s_m[kWaves][kMaxGroup], s_l[kWaves][kMaxGroup];
  __shared__ __attribute__((aligned(16))) float s_o[kWaves][G][D];
  __shared__ int s_last;
#if DELTA_QK_VALU
  __shared__ __attribute__((aligned(16))) uint16_t s_qv[kWaves][G * D];
#endif
  static_assert(G * D <= 4 * kAttnThreads && D % 4 == 0, "four outputs per thread cover a group");

  // ---- attention of groups [g0, g0 + ng) of (sequence b, KV head g), staged by stage(); the
  // piece is partial `slot` of the n_valid partials of its pair (n_valid == 1: the whole pair)
  auto run = [&](int b, int g, int g0, int ng, int slot, int n_valid, int s_b, int sel_n) {
    const int bg = b * a.n_kv_heads + g;
    lds_barrier();   // the page / row list is in LDS; the query loads may still be in flight

    const size_t head_off = (size_t)g * 16 * D;
    // Loads tile `li` of the piece.  A prefetch past the wave's last group (real == false) is
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

    float* lp = s_p[wave];
    WaveSoftmax<G> st;
    st.init();
    const int Hq_row = b * Hq + g * G;
    // Logits on: the workgroup keeps the logits of a chunk of kChunk groups in LDS ([group]
    // [head][16], the global layout) and writes the chunk out cooperatively between chunks,
    // with non-temporal (streaming) stores.  Measured on MI355X, logit stores interleaved with
    // the K/V read stream cost several times their bytes, while the same bytes written in a
    // few large streaming bursts (reads paused) cost about their share.  A chunk is a multiple
    // of 16 groups.
#if DELTA_QK_VALU
    // build option: QK^T on the vector ALUs, the query vectors read from the wave's LDS copy
    stage_query_lds<D, G>(qb, s_qv[wave], lane);
    wave_lds_sync();
    auto process = [&](const Tile<D>& t, int slot_in_chunk) {
      process_tile_valu<D, G, LOGITS>(t, s_qv[wave], a.scale_log2, st, lp,
                                      s_stage + slot_in_chunk * G * 16, lane);
    };
#else
    auto process = [&](const Tile<D>& t, int slot_in_chunk) {
      process_tile<D, G, LOGITS>(t, qb, a.scale_log2, st, lp, s_stage + slot_in_chunk * G * 16, lane);
    };
#endif

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

    // ---- reduce o over the lanes that share a head-dim chunk -----------------------------
    reduce_outputs<D, G>(st);

    // ---- merge the 4 waves into one partial of the piece ---------------------------------
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

    // From here on thread t owns the four consecutive outputs e0 = 4t .. 4t+3 of head h (D is
    // a multiple of 4, G * D <= 1024 = 4 * kAttnThreads), so every partial, output and merge
    // access is one 16- or 8-byte access and each thread needs the running max and sum of one
    // head.
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

    // A pair that is one piece needs no combine: the workgroup writes the output itself.
    if (n_valid == 1) {
      if (owner) store_out(O, L, M);
      return;
    }

    // ---- combine ----------------------------------------------------------------------
    // Partials are written and read only with device-coherent accesses (the sc1 cache policy:
    // written through to memory, and read past any stale copy in another XCD's L2), so no L2
    // write-back or invalidation is needed to publish them.  Each thread waits until its
    // partial stores are complete, the barrier makes that true for the whole workgroup, and
    // only then does one thread count the workgroup in with a device-scope atomic; the
    // workgroup that brings the count to n_valid reads every partial after the atomic has
    // returned.  (A release/acquire fence pair would instead write back and invalidate the
    // whole L2 of the XCD once per workgroup; measured on MI355X that serialises launches of
    // many workgroups.)
    const int pair_floats = a.slots * G * D;
    const __amdgpu_buffer_rsrc_t po = __builtin_amdgcn_make_buffer_rsrc(
        a.part_o + (size_t)bg * pair_floats, 0, pair_floats * 4, kRawBufferFlags);
    const __amdgpu_buffer_rsrc_t pml = __builtin_amdgcn_make_buffer_rsrc(
        a.part_ml + (size_t)bg * a.slots * G * 2, 0, a.slots * G * 8, kRawBufferFlags);
    const int o_off = (h * D + dc) * 4;   // this thread's bytes inside one slot's G x D block
    if (owner) {
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, O), po, o_off,
                                             slot * G * D * 4, kCoherent);
      if (dc == 0)
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, make_float2(M, L)), pml,
                                              h * 8, slot * G * 8, kCoherent);
    }
    __builtin_amdgcn_s_waitcnt(0);   // this thread's partial stores are complete
    __syncthreads();
    if (tid == 0) {
      const int prev = __hip_atomic_fetch_add(&a.counters[(size_t)bg * kCounterStride], 1, __ATOMIC_RELAXED,
                                              __HIP_MEMORY_SCOPE_AGENT);
      s_last = prev == n_valid - 1;
    }
    __syncthreads();
    if (!s_last || !owner) return;

    // Every owner thread loads its head's (max, sum) and its four outputs of kMergeBatch
    // partials at once (one wait for memory per batch, a single batch up to kMergeBatch) and
    // folds them into a running (max, sum, o) in slot order: the result does not depend on the
    // order in which workgroups finished.  Slots past the last piece are not loaded (a uniform
    // branch; repeating the last slot's loads instead cost ≈0.3 µs per launch at two pieces).
    constexpr int kMergeBatch = 16;
    M = kNegInf;
    L = 0.f;
    O = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int c0 = 0; c0 < n_valid; c0 += kMergeBatch) {
      float2 ml[kMergeBatch];
      f32x4 pv[kMergeBatch];
#pragma unroll
      for (int c = 0; c < kMergeBatch; ++c) {
        ml[c] = make_float2(kNegInf, 0.f);
        pv[c] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (c0 + c < n_valid) {
          ml[c] = __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(pml, h * 8, (c0 + c) * G * 8, kCoherent));
          pv[c] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(po, o_off, (c0 + c) * G * D * 4, kCoherent));
        }
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
    if (tid == 0) __hip_atomic_store(&a.counters[(size_t)bg * kCounterStride], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  };

  // ---- which pieces this workgroup attends to --------------------------------------------
  // The static decomposition: workgroup (split, g, b) takes groups [split * gps, + gps) of
  // pair (b, g), as partial `split`.  Its page list and query are staged before anything else
  // (the sequence length arrives meanwhile) and kept when the balanced decomposition below
  // hands this workgroup the same piece.
  const int split = blockIdx.x;
  const int g_s = blockIdx.y;
  const int b_s = blockIdx.z;
  const int g0_s = split * a.gps;
  const int cand_s = max(0, min(a.gps, a.max_groups - g0_s));
  stage(b_s, g_s, g0_s, cand_s);
  const int s_bs = a.seq_lens[b_s];
  if (DELTA_DEBUG && (s_bs < 1 || s_bs > a.max_seq_len) && tid == 0 && blockIdx.x == 0 && blockIdx.y == 0)
    debug_flag(a.status, DELTA_DEBUG_SEQ_LEN);
  const int sel_ns = (MODE == ROWS_DENSE) ? 0 : min(a.sel_cnt[b_s], a.sel_stride);

  int bal_chunk = 0;          // > 0: this launch takes the balanced decomposition
  int bal_w = 0, bal_x = 0, bal_xe = 0;   // this workgroup's run [bal_x, bal_xe)
  // lane l of every wave: sequence l's length, groups, and groups of sequences 0 .. l - 1
  int bal_len = 0, bal_units = 0, bal_before = 0;
  if (MODE == ROWS_DENSE && BAL && gridDim.z <= 64) {   // one sequence per lane
    // Balanced decomposition of a dense launch (the work of a ragged batch spread evenly):
    // the groups of every (sequence, KV head) pair, in (b, g, page) order, are cut into runs of
    // `chunk` groups, run w for workgroup w (the launch's linear index, in dispatch order).  A
    // run may span pairs; a pair is combined from the pieces the run boundaries cut it into,
    // in order.  An empty sequence counts as one group (its piece writes the empty output).
    // Every wave derives the same cut from the sequence lengths (one per lane: B <= 64), and it
    // is taken only when no run spans more than three pairs (chunk <= 2 x the shortest pair)
    // and when it pays (below).
    const int B = gridDim.z;
    if (lane < B) {
      bal_len = a.seq_lens[lane];
      bal_units = max(1, min((max(bal_len, 0) + 15) >> 4, a.max_groups));
    }
    const int incl = wave_incl_scan(bal_units);
    bal_before = incl - bal_units;
    const int total = __builtin_amdgcn_readlane(incl, 63);
    const int shortest = (int)wave_min((uint32_t)(lane < B ? bal_units : 0x7fffffff));
    const int Hkv = a.n_kv_heads;
    // the host bounds the batch's groups (Hkv * B * max_groups) below 2^31
    const int W = Hkv * total;
    const int n_wg = gridDim.x * gridDim.y * gridDim.z;
    const int chunk = max((W + n_wg - 1) / n_wg, a.chunk_min);
    // Taken only when it shortens the longest run by a tenth or more against the static
    // pieces (gps groups); equal or nearly equal lengths keep the static split, whose pieces
    // never straddle a pair.  Otherwise, with lengths that are not a multiple of the run, the
    // run boundaries drift through successive pairs and leave slivers of a few groups, each
    // with a piece's fixed costs.
    if (chunk <= 2 * shortest && 10 * chunk <= 9 * a.gps) {   // uniform over the launch
      bal_chunk = chunk;
      bal_w = split + gridDim.x * (g_s + Hkv * b_s);
      bal_x = bal_w * chunk;
      bal_xe = min(W, bal_x + chunk);
    }
  }

  // ---- the pieces, one attention call site (the balanced runs, or the static piece) --------
  bool first = true;
  while (true) {
    // Lane-dependent values are recomputed per piece instead of being hoisted out of this loop
    // (where they would stay live, in registers, through the attention loop of every piece).
    if (BAL) asm volatile("" : "+v"(tid), "+v"(lane), "+v"(quad), "+v"(hcol));
    int b, g, g0, ng, slot, n_valid, s_b, sel_n, n_groups;
    if (bal_chunk > 0) {
      if (bal_x >= bal_xe) break;
      // sequence b: the last with Hkv * (groups before b) <= x (lanes below B, in order)
      const int Hkv = a.n_kv_heads;
      const uint64_t le = __ballot(lane < (int)gridDim.z && Hkv * bal_before <= bal_x);
      b = __builtin_amdgcn_readfirstlane(__popcll(le) - 1);
      const int pb = __builtin_amdgcn_readlane(bal_before, b);
      const int ub = __builtin_amdgcn_readlane(bal_units, b);
      const int loc = bal_x - Hkv * pb;
      g = loc / ub;
      g0 = loc - g * ub;
      const int off = Hkv * pb + g * ub;   // the pair's first group
      const int end = min(bal_xe, off + ub);
      const int first_run = off / bal_chunk;
      n_valid = (off + ub - 1) / bal_chunk - first_run + 1;
      slot = bal_w - first_run;
      ng = end - bal_x;
      s_b = __builtin_amdgcn_readlane(bal_len, b);
      sel_n = 0;
      n_groups = min((max(s_b, 0) + 15) >> 4, a.max_groups);
      bal_x = end;
      if (!(first && b == b_s && g == g_s && g0 == g0_s && ng <= cand_s)) stage(b, g, g0, ng);
    } else {
      if (!first) break;
      b = b_s;
      g = g_s;
      g0 = g0_s;
      s_b = s_bs;
      sel_n = sel_ns;
      if (MODE == ROWS_DENSE) n_groups = (s_b + 15) >> 4;
      else if (MODE == ROWS_SEL_PAGE) n_groups = sel_n;
      else n_groups = (sel_n + 15) >> 4;
      // lengths beyond the host bound are clamped so that no access leaves the buffers
      n_groups = max(0, min(n_groups, a.max_groups));
      n_valid = (n_groups + a.gps - 1) / a.gps;
      slot = split;
      ng = n_valid > 0 ? min(a.gps, n_groups - g0) : 0;
      if (n_valid > 0 && split >= n_valid) break;
      if (n_valid == 0 && split > 0) break;
    }
    first = false;
    // the piece is the same in every lane: scalar registers for the walk's bounds and addresses
    b = __builtin_amdgcn_readfirstlane(b);
    g = __builtin_amdgcn_readfirstlane(g);
    g0 = __builtin_amdgcn_readfirstlane(g0);
    ng = __builtin_amdgcn_readfirstlane(ng);
    slot = __builtin_amdgcn_readfirstlane(slot);
    n_valid = __builtin_amdgcn_readfirstlane(n_valid);
    s_b = __builtin_amdgcn_readfirstlane(s_b);
    sel_n = __builtin_amdgcn_readfirstlane(sel_n);
    n_groups = __builtin_amdgcn_readfirstlane(n_groups);
    if (n_groups == 0) write_empty(b, g);
    else run(b, g, g0, ng, slot, n_valid, s_b, sel_n);
  }
}

template <int D, int G>
hipError_t launch_dg(int mode, const AttnArgs& a, int batch, hipStream_t stream) {
  const dim3 grid(a.n_split, a.n_kv_heads, batch), block(kAttnThreads);
  switch (mode) {
    case ROWS_DENSE:
      // the balanced decomposition is a separate instantiation, so that launches which cannot
      // take it run the static kernel's code
      if (a.logits && a.balance) hipLaunchKernelGGL((attn_kernel<D, G, ROWS_DENSE, true, true>), grid, block, 0, stream, a);
      else if (a.logits) hipLaunchKernelGGL((attn_kernel<D, G, ROWS_DENSE, true, false>), grid, block, 0, stream, a);
      else if (a.balance) hipLaunchKernelGGL((attn_kernel<D, G, ROWS_DENSE, false, true>), grid, block, 0, stream, a);
      else hipLaunchKernelGGL((attn_kernel<D, G, ROWS_DENSE, false, false>), grid, block, 0, stream, a);
      break;
    case ROWS_SEL_PAGE: hipLaunchKernelGGL((attn_kernel<D, G, ROWS_SEL_PAGE, false, false>), grid, block, 0, stream, a); break;
    case ROWS_SEL_TOKEN: hipLaunchKernelGGL((attn_kernel<D, G, ROWS_SEL_TOKEN, false, false>), grid, block, 0, stream, a); break;
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

// Per-tile pieces of the gfx950 decode-attention kernels (Sec. 2, Eq. gqa_attention): loading a
// 16-row K/V tile of one KV head, and folding it into one wave's online softmax for the G query
// heads of that KV head.
//
//   * QK^T on the matrix cores: v_mfma_f32_16x16x32_bf16 with A = the 16 K rows (M = rows,
//     K = head dim) and B = the G query vectors padded to 16 columns; D/32 MFMAs give the
//     16 x 16 score tile, lane l holding rows 4*(l/16)..+3 of head column l%16.
//   * online softmax in the log2 domain (exp2, scale folded with log2 e); the tile's
//     probabilities and the per-head rescale factor go through a wave-private LDS slice;
//   * P.V on the vector ALUs: each lane owns 8 consecutive head-dim columns of 16/RPI rows
//     (128-bit loads, one V row per LPR consecutive lanes, fully coalesced).
#pragma once

#include "internal.h"
#include "wave.h"

namespace delta {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kNegInfF = -__builtin_huge_valf();

template <int D>
struct Geo {
  static constexpr int NK = D / 32;     // MFMA k-steps = 16-byte K loads per lane per tile
  static constexpr int LPR = D / 8;     // lanes per V row
  static constexpr int RPI = 64 / LPR;  // V rows per wave-wide load
  static constexpr int NI = 16 / RPI;   // V loads per lane per tile
  // register tiles per wave: loads of R - 1 tiles stay in flight while one is consumed
  static constexpr int R = D == 128 ? 3 : 4;
};

template <int D>
struct Tile {
  u32x4 k[Geo<D>::NK];
  u32x4 v[Geo<D>::NI];
  uint32_t kmask;   // bit r: row r valid (rows of the MFMA A operand and of the score tile)
};

// One wave's running softmax state for the G query heads of one KV head: running max and sum
// of head (lane & 15) (valid for lanes with lane & 15 < G), and the lane's share of the
// unnormalised outputs (8 head-dim columns of its V rows, for every head).
template <int G>
struct WaveSoftmax {
  float m_run, l_run;
  float o[G][8];
  __device__ __forceinline__ void init() {
    m_run = kNegInfF;
    l_run = 0.f;
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) o[h][e] = 0.f;
  }
};

__device__ __forceinline__ u32x4 load16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}
// K/V rows are read once per launch: non-temporal loads.  Measured on MI355X they raise the
// streaming rate of the full and sparse layers by 5-20 % over ordinary loads.
__device__ __forceinline__ u32x4 load16_stream(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;  // NaN stays NaN
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Compiler-level ordering for LDS traffic that stays inside one wave (the LDS unit executes
// one wave's requests in order; this only stops the compiler from moving them).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The query operand of the MFMA: the G query vectors of KV head g (row `qrow` = b*Hq + g*G of
// q), lane (quad, hcol) holding 8 head-dim values of head hcol; columns hcol >= G are zero.
template <int D, int G>
__device__ __forceinline__ void load_query(bf16x8 (&qb)[Geo<D>::NK], const uint16_t* q,
                                           size_t qrow, int lane) {
  const int quad = lane >> 4, hcol = lane & 15;
  const uint16_t* qp = q + (qrow + min(hcol, G - 1)) * D + 8 * quad;
#pragma unroll
  for (int ks = 0; ks < Geo<D>::NK; ++ks) {
    u32x4 w = load16(qp + 32 * ks);
    if (hcol >= G) w = u32x4{0u, 0u, 0u, 0u};
    qb[ks] = __builtin_bit_cast(bf16x8, w);
  }
}

// Loads the [16, D] K and V tile that starts at kt / vt (one page of one KV head).  With
// real == false the loads are still issued, so that a loop's memory waits stay uniform, but
// with every lane at the tile's first 16 bytes: one cache line per load instruction.
template <int D>
__device__ __forceinline__ void load_page_tile(Tile<D>& t, const uint16_t* kt, const uint16_t* vt,
                                               bool real, int lane) {
  using Gm = Geo<D>;
  const int quad = lane >> 4, hcol = lane & 15;
  const uint16_t* kp = kt + (real ? (size_t)hcol * D + 8 * quad : 0);
#pragma unroll
  for (int ks = 0; ks < Gm::NK; ++ks) t.k[ks] = load16_stream(kp + (real ? 32 * ks : 0));
  const uint16_t* vp = vt + (real ? (size_t)(lane / Gm::LPR) * D + 8 * (lane % Gm::LPR) : 0);
#pragma unroll
  for (int i = 0; i < Gm::NI; ++i) t.v[i] = load16_stream(vp + (real ? (size_t)Gm::RPI * i * D : 0));
}

// Folds one tile's score tile (acc: lane (quad, hcol) holds q_hcol . k_r for rows
// r = 4*quad .. 4*quad+3, unscaled) into the wave's softmax state.  lp: the wave's LDS slice
// (16 x 8 + 8 floats).  With LOGITS, the tile's scaled log2-domain logits go to
// logit_slot[head][16] (LDS).
template <int D, int G, bool LOGITS>
__device__ __forceinline__ void fold_tile(const f32x4 acc, const Tile<D>& t, float scale_log2,
                                          WaveSoftmax<G>& st, float* lp, float* logit_slot,
                                          int lane) {
  using Gm = Geo<D>;
  const int quad = lane >> 4, hcol = lane & 15;
  float x[4];
#pragma unroll
  for (int r = 0; r < 4; ++r)
    x[r] = ((t.kmask >> (4 * quad + r)) & 1u) ? acc[r] * scale_log2 : kNegInfF;
  if (LOGITS && hcol < G)
    *reinterpret_cast<f32x4*>(logit_slot + hcol * 16 + 4 * quad) = f32x4{x[0], x[1], x[2], x[3]};
  float mx = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
  mx = max_xor32(max_xor16(mx));
  const float m_new = fmaxf(st.m_run, mx);
  // m_new is finite whenever the tile has a valid row (always, for valid selections); the
  // guard keeps an all-masked tile from turning the running state into NaN
  const float m_use = (m_new == kNegInfF) ? 0.f : m_new;
  const float alpha = exp2f(st.m_run - m_use);
  float p[4], ps = 0.f;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    p[r] = exp2f(x[r] - m_use);
    ps += p[r];
  }
  ps = sum_xor32(sum_xor16(ps));
  st.l_run = st.l_run * alpha + ps;
  st.m_run = m_new;

  wave_lds_sync();
  if (hcol < G) {
#pragma unroll
    for (int r = 0; r < 4; ++r) lp[(4 * quad + r) * 8 + hcol] = p[r];
    if (quad == 0) lp[128 + hcol] = alpha;
  }
  wave_lds_sync();

#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float al = lp[128 + h];
#pragma unroll
    for (int e = 0; e < 8; ++e) st.o[h][e] *= al;
  }
#pragma unroll
  for (int i = 0; i < Gm::NI; ++i) {
    const int row = Gm::RPI * i + lane / Gm::LPR;
    u32x4 w = t.v[i];
    if (!((t.kmask >> row) & 1u)) w = u32x4{0u, 0u, 0u, 0u};   // rows past the end may hold NaN
    float v[8];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      v[2 * c] = __uint_as_float(w[c] << 16);
      v[2 * c + 1] = __uint_as_float(w[c] & 0xffff0000u);
    }
    const float* pr = lp + row * 8;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float ph = pr[h];
#pragma unroll
      for (int e = 0; e < 8; ++e) st.o[h][e] = fmaf(ph, v[e], st.o[h][e]);
    }
  }
}

// Folds one tile into the wave's softmax state, QK^T on the matrix cores (see the file header).
template <int D, int G, bool LOGITS>
__device__ __forceinline__ void process_tile(const Tile<D>& t, const bf16x8 (&qb)[Geo<D>::NK],
                                             float scale_log2, WaveSoftmax<G>& st, float* lp,
                                             float* logit_slot, int lane) {
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < Geo<D>::NK; ++ks)
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, t.k[ks]), qb[ks],
                                                  acc, 0, 0, 0);
  fold_tile<D, G, LOGITS>(acc, t, scale_log2, st, lp, logit_slot, lane);
}

// The same score tile with QK^T on the vector ALUs, a build option (DELTA_QK_VALU) kept for
// comparing the two engines.  Lane (quad, r) holds 32 head-dim values of K row r (the registers
// of the matrix-core operand) and forms their dot products with the same 32 values of every
// query head (sq: the wave's LDS copy of the G query vectors, bf16 [G][D]) with
// v_dot2_f32_bf16; the four quads' partial sums are added across lanes, and the tile goes
// through the wave's LDS slice into the matrix-core layout that fold_tile reads.
template <int D, int G>
__device__ __forceinline__ void stage_query_lds(const bf16x8 (&qb)[Geo<D>::NK], uint16_t* sq,
                                                int lane) {
  const int quad = lane >> 4, hcol = lane & 15;
  if (hcol < G) {
#pragma unroll
    for (int ks = 0; ks < Geo<D>::NK; ++ks)
      *reinterpret_cast<bf16x8*>(sq + hcol * D + 32 * ks + 8 * quad) = qb[ks];
  }
}

template <int D, int G, bool LOGITS>
__device__ __forceinline__ void process_tile_valu(const Tile<D>& t, const uint16_t* sq,
                                                  float scale_log2, WaveSoftmax<G>& st, float* lp,
                                                  float* logit_slot, int lane) {
  const int quad = lane >> 4, r = lane & 15;
  float part[G];
#pragma unroll
  for (int h = 0; h < G; ++h) part[h] = 0.f;
#pragma unroll
  for (int ks = 0; ks < Geo<D>::NK; ++ks) {
    const u32x4 kw = t.k[ks];
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const u32x4 qw = *reinterpret_cast<const u32x4*>(sq + h * D + 32 * ks + 8 * quad);
      // v_dot2_f32_bf16 written out: with hipcc of ROCm 7.2 at -O3 the builtin
      // (__builtin_amdgcn_fdot2_f32_bf16) compiled to the same operand pair repeated for the
      // four pairs of a 16-byte chunk (wrong sums; found with a one-tile check against the
      // matrix-core tile), the instruction itself gives the right ones
#pragma unroll
      for (int c = 0; c < 4; ++c)
        asm volatile("v_dot2_f32_bf16 %0, %1, %2, %0" : "+v"(part[h]) : "v"(kw[c]), "v"(qw[c]));
    }
  }
#pragma unroll
  for (int h = 0; h < G; ++h) part[h] = sum_xor32(sum_xor16(part[h]));
  wave_lds_sync();
  if (quad == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) lp[r * 8 + h] = part[h];
  }
  wave_lds_sync();
  f32x4 acc;
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] = r < G ? lp[(4 * quad + i) * 8 + r] : 0.f;
  fold_tile<D, G, LOGITS>(acc, t, scale_log2, st, lp, logit_slot, lane);
}

// Sums each lane's output share over the lanes that hold the same head-dim columns: afterwards
// lanes 0 .. LPR-1 hold the wave's complete outputs o[h][8*lane .. 8*lane+7].
template <int D, int G>
__device__ __forceinline__ void reduce_outputs(WaveSoftmax<G>& st) {
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float v = st.o[h][e];
      if (Geo<D>::LPR == 8) v += lane_xor8(v);
      st.o[h][e] = sum_xor32(sum_xor16(v));
    }
}

}  // namespace delta

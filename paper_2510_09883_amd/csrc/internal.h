// Internal interface between the C ABI layer (delta_api.cpp) and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/delta_attn.h"

// Debug builds (-DDELTA_DEBUG=1) check on the device the preconditions that the host cannot see
// (page-table entries, sequence lengths, selected units; see delta_build_flags in the C ABI),
// record a failure as a bit in the workspace's status word and go on with an in-range value.
#ifndef DELTA_DEBUG
#define DELTA_DEBUG 0
#endif

namespace delta {

// How the 16-row groups an attention workgroup walks are formed.
enum RowMode {
  ROWS_DENSE = 0,      // group i = logical page i of the sequence (full / Delta layers)
  ROWS_SEL_PAGE = 1,   // group i = selected page sel_idx[b, i]            (sparse, U = 16)
  ROWS_SEL_TOKEN = 2,  // group i = selected tokens sel_idx[b, 16i .. 16i+15] (sparse, U = 1)
};

// Hard limits of the attention kernel's on-chip staging.
constexpr int kAttnThreads = 256;        // 4 waves of 64
constexpr int kMaxSplits = 64;           // split partials combined by the last workgroup
constexpr int kMaxRowSlots = 1024;       // LDS slots staging a split's page / row list
constexpr int kMaxGroup = 8;             // query heads per KV head (padded to 16 MFMA columns)
constexpr int kMaxSelectKeys = 8192;     // candidate units one selection workgroup holds in registers
constexpr int kBalanceMaxBatch = 64;     // sequences of a balanced dense launch (one per lane)
// Ints between consecutive arrival counters (256 bytes): every counter that many workgroups
// update and poll sits in a memory block of its own instead of sharing one with its neighbours'.
constexpr int kCounterStride = 64;

struct AttnArgs {
  const uint16_t* k_cache;   // bf16 [pages, Hkv, 16, D]
  const uint16_t* v_cache;
  const int32_t* page_table; // [B, max_pages]
  const int32_t* seq_lens;   // [B]
  const int32_t* sel_idx;    // [B, sel_stride] (sparse modes)
  const int32_t* sel_cnt;    // [B]             (sparse modes)
  const int32_t* sel_phys;   // [B, sel_stride] physical locations of sel_idx, or null
  const uint16_t* q;         // bf16 [B, Hq, D]
  uint16_t* out;             // bf16 [B, Hq, D]
  float* part_o;             // [B*Hkv, slots, G, D]   un-normalised partial outputs
  float* part_ml;            // [B*Hkv, slots, G, 2]   partial (max, sum) in the log2 domain
  int32_t* counters;         // [B*Hkv] arrival counters (kCounterStride apart), zero between launches
  float* logits;             // [B, Hkv, logit_pages, G, 16] log2-domain logits, or null
  float* lse;                // [B, Hq] log2-domain log-sum-exp, or null
  int64_t page_stride;       // elements per physical page = Hkv * 16 * D
  int32_t n_q_heads, n_kv_heads, max_pages, sel_stride, logit_pages;
  int32_t n_split, gps;      // static decomposition: splits per (b, kv head), 16-row groups
                             // per split; the grid is (n_split, Hkv, B)
  int32_t max_groups;        // host bound on groups per sequence (n_split * gps >= it)
  int32_t slots;             // partial slots per (b, kv head), >= the pieces of any pair
  int32_t chunk_min;         // shortest run of the balanced decomposition (dense launches)
  int32_t balance;           // 1: a dense launch may take the balanced decomposition
  float scale_log2;          // sm_scale * log2(e)
  int64_t n_pages;           // physical pages of the caches (0: not stated); debug checks
  int32_t max_seq_len;       // host bound of seq_lens[b]; debug checks
  uint32_t* status;          // debug status word (workspace byte 0)
};

hipError_t launch_attention(int head_dim, int group, int mode, const AttnArgs& a, int batch,
                            hipStream_t stream);

struct ScoreArgs {
  const float* logits;       // [B, Hkv, logit_pages, G, 16]
  const float* lse;          // [B, Hq]
  const int32_t* seq_lens;   // [B]
  float* unit_scores;        // [B, nu_stride]
  int32_t n_q_heads, n_kv_heads, logit_pages, nu_stride, max_seq_len;
};

hipError_t launch_score(int agg, int unit_tokens, const ScoreArgs& a, int batch,
                        hipStream_t stream);

struct SelectArgs {
  const float* unit_scores;  // [B, nu_stride]
  const int32_t* seq_lens;   // [B]
  const int32_t* page_table; // [B, max_pages]
  int32_t* sel_idx;          // [B, budget_units]
  int32_t* sel_cnt;          // [B]
  int32_t* sel_phys;         // [B, budget_units] physical page (U = 16) or page*16 + row (U = 1)
                             // of each selected unit, -1 past the count; null: not written
  int32_t nu_stride, unit_tokens, budget_units, recent_units, max_pages;
};

hipError_t launch_select(const SelectArgs& a, int batch, hipStream_t stream);

// Fused Delta layer: attention, scoring and selection in one launch, with the logits kept in
// LDS.  One workgroup per (chunk of kFusedChunkPages pages, sequence) covers every KV head of
// the chunk, so the logits a workgroup needs for scoring are its own.
constexpr int kFusedChunkPages = 64;
constexpr int kFusedMaxQHeads = 32;      // LDS holds kFusedMaxQHeads x 64 x 16 fp32 logits
constexpr int kFusedKeysPerThread = 8;   // selection candidates held per thread (2048 units)
constexpr int kFusedMaxChunks = 32;      // chunks per sequence (2048 pages): partials load at once

struct FusedArgs {
  const uint16_t* k_cache;   // bf16 [pages, Hkv, 16, D]
  const uint16_t* v_cache;
  const int32_t* page_table; // [B, max_pages]
  const int32_t* seq_lens;   // [B]
  const uint16_t* q;         // bf16 [B, Hq, D]
  uint16_t* out;             // bf16 [B, Hq, D]
  float* part_o;             // [B, Hkv, n_chunks, G, D]  un-normalised chunk outputs
  float* part_ml;            // [B, Hkv, n_chunks, G, 2]  chunk (max, sum), log2 domain
  int32_t* counters;         // [B] x kCounterStride: arrivals after attention (int 0 of each
                             // sequence's block), arrivals after scoring (int 32), "a chunk was
                             // left to the last workgroup" (int 48); zero between launches
  int32_t* chunk_flags;      // [B, n_chunks] chunk left to the last workgroup; zero between launches
  float* logits;             // [B, Hkv, logit_pages, G, 16] logits of left chunks (workspace)
  float* unit_scores;        // [B, sel.nu_stride] page (or token) scores, written here
  int64_t page_stride;       // elements per physical page = Hkv * 16 * D
  int64_t spin_ticks;        // longest wait at the sequence barrier, 100 MHz clock ticks
  int32_t n_q_heads, n_kv_heads, max_pages, n_chunks, max_seq_len, agg, logit_pages;
  float scale_log2;
  SelectArgs sel;            // unit scores (written here), selection outputs
  int64_t n_pages;           // physical pages of the caches (0: not stated); debug checks
  uint32_t* status;          // debug status word (workspace byte 0)
};

// Largest grid (chunks x sequences) the fused kernel can have resident at once on the current
// device, or 0 when the shape has no fused kernel.
int fused_delta_capacity(int head_dim, int group, int unit_tokens);
hipError_t launch_fused_delta(int head_dim, int group, const FusedArgs& a, int batch,
                              hipStream_t stream);

// KV append (Eq. kv_update): the current token's K and V rows into the paged cache.
struct AppendArgs {
  uint16_t* k_cache;         // bf16 [pages, Hkv, 16, D]
  uint16_t* v_cache;
  const int32_t* page_table; // [B, max_pages]
  const int32_t* seq_lens;   // [B], counting the new token
  const uint16_t* k_new;     // bf16 [B, Hkv, D]
  const uint16_t* v_new;
  int64_t page_stride;       // elements per physical page = Hkv * 16 * D
  int32_t n_kv_heads, head_dim, max_pages;
  int64_t n_pages;           // physical pages of the caches (0: not stated); debug checks
};

hipError_t launch_kv_append(const AppendArgs& a, int batch, hipStream_t stream);

hipError_t launch_fill_zero(void* ptr, size_t bytes, hipStream_t stream);
hipError_t launch_fill_zero2(void* p0, size_t bytes0, void* p1, size_t bytes1, hipStream_t stream);

// Library-held scratch of the allocation-free decode step: one array of this many bytes per
// GPU (DELTA_NOALLOC_SCRATCH_BYTES of the C ABI), allocated when the step first runs there.
// *ptr gets the current device's copy.
constexpr size_t kNoallocScratchBytes = (size_t)160 << 20;
hipError_t noalloc_scratch(void** ptr);

}  // namespace delta

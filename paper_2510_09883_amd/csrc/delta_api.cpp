// C ABI of the DELTA decode-step attention hot path: argument checks, workspace layout, split
// planning, launches, and the layer-schedule driver of App. A, Alg. 1.
//
// Nothing here touches device memory directly or synchronises: every call validates on the
// host, then enqueues kernels on the caller's stream.  Grid sizes come from host-side bounds
// (max_seq_len, budget), and the kernels read the actual per-sequence lengths and selection
// counts on the device, so no step needs a device-to-host round trip.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>

#include "../../include/delta_attn.h"
#include "internal.h"

namespace {

using namespace delta;

static_assert(kNoallocScratchBytes == DELTA_NOALLOC_SCRATCH_BYTES, "scratch size of the C ABI");

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Workgroups the attention launch aims for: about one per CU (256 CUs).  Measured on MI355X,
// more and shorter workgroups (up to 4096) were slower at every workload size: each one pays a
// dependent metadata load, an LDS wave merge and a partial store before its work is counted.
// DELTA_ATTN_TARGET_WGS overrides it for tuning.
int target_workgroups() {
  static int v = [] {
    const char* e = getenv("DELTA_ATTN_TARGET_WGS");
    int x = e ? atoi(e) : 0;
    return x > 0 ? x : 256;
  }();
  return v;
}

// Minimum 16-row groups per split (per workgroup of 4 waves): two per wave.  Measured on
// MI355X, the 128-page sparse layer of one 8K sequence runs 3 % faster with 16 splits of 8
// groups than with 8 of 16, and 4 groups per split are no faster; larger launches are not
// affected (their split count is set by the workgroup target).
int min_groups_per_split() {
  static int v = [] {
    const char* e = getenv("DELTA_ATTN_MIN_GPS");
    int x = e ? atoi(e) : 0;
    return x > 0 ? x : 8;
  }();
  return v;
}

// Most splits per (sequence, kv head).  The last workgroup's merge reads every split's partial
// (one batch of loads per 16 splits) and each split adds an arrival on the same counter, so
// beyond ~16 splits the combine costs more than the shorter loop saves (measured on MI355X with
// one sequence of 8K tokens).  DELTA_ATTN_MAX_SPLITS overrides it for tuning.
int max_splits() {
  static int v = [] {
    const char* e = getenv("DELTA_ATTN_MAX_SPLITS");
    int x = e ? atoi(e) : 0;
    return x > 0 ? std::min(x, kMaxSplits) : 16;
  }();
  return v;
}

struct SplitPlan {
  int n_split = 0;
  int gps = 0;
  int max_groups = 0;
  int slots = 0;       // partial slots per (sequence, kv head)
  int chunk_min = 0;   // balanced decomposition: shortest run
  int balance = 0;     // balanced decomposition allowed (dense launches)
};

// Whether dense launches may spread a ragged batch's work evenly (the balanced decomposition
// of the attention kernel).  DELTA_ATTN_BALANCE=0 keeps the static one, for comparison.
bool balance_enabled() {
  static int v = [] {
    const char* e = getenv("DELTA_ATTN_BALANCE");
    return e && atoi(e) == 0 ? 0 : 1;
  }();
  return v != 0;
}

// Splits per (sequence, kv head) and groups per split for a launch over at most `max_groups`
// groups of 16 rows.  Deterministic in the shape, so a FULL and a DELTA call over the same
// shape use the same plan (and give bitwise-identical outputs).
bool plan_split(int pairs, int max_groups, int slot_cap, SplitPlan* p) {
  if (max_groups < 1) max_groups = 1;
  int want = std::max(1, ceil_div(target_workgroups(), pairs));
  int most = std::max(1, ceil_div(max_groups, min_groups_per_split()));
  int n_split = std::min(std::min(want, most), max_splits());
  int gps = ceil_div(max_groups, n_split);
  if (gps > slot_cap) gps = slot_cap;
  n_split = ceil_div(max_groups, gps);
  if (n_split > kMaxSplits) return false;
  p->n_split = n_split;
  p->gps = gps;
  p->max_groups = max_groups;
  p->slots = n_split;
  return true;
}

// The balanced decomposition of a dense launch over `batch` sequences, 2 to kBalanceMaxBatch
// (one sequence cannot be ragged; the kernel holds one sequence length per lane).  Runs are at
// least chunk_min groups, so no pair is cut into more than slots pieces, and at most
// kMaxRowSlots: the run of a workgroup of the static grid, ceil(work / workgroups), never
// exceeds gps.
void plan_balance(int batch, int pairs, SplitPlan* p) {
  const int cap = std::min(max_splits(), kMaxSplits - 1);
  const int chunk_min = std::max(min_groups_per_split(), ceil_div(p->max_groups, cap));
  if (!balance_enabled() || batch < 2 || batch > kBalanceMaxBatch || chunk_min > kMaxRowSlots) return;
  // the kernel does the cut's arithmetic in 32 bits
  if ((int64_t)pairs * p->max_groups >= ((int64_t)1 << 31)) return;
  p->chunk_min = chunk_min;
  p->slots = std::max(p->n_split, ceil_div(p->max_groups, chunk_min) + 1);
  p->balance = 1;
}

struct Layout {
  size_t status = 0, counters = 0, part_ml = 0, part_o = 0, logits = 0, lse = 0, uscores = 0, phys = 0;
  size_t fcnt = 0, fflag = 0;
  size_t total = 0;
  int fused_chunks = 0;   // chunks per sequence of the fused Delta kernel
  int max_split = 0;
  int logit_pages = 0;
  int nu_stride = 0;
  SplitPlan dense, sparse;
  int sparse_mode = ROWS_SEL_PAGE;
};

int check_shape(const delta_shape_t* s) {
  if (!s) return DELTA_ERR_INVALID_ARG;
  if (s->batch < 1 || s->n_q_heads < 1 || s->n_kv_heads < 1 || s->max_seq_len < 1 ||
      s->max_pages_per_seq < 1 || !(s->sm_scale >= 0.f) || isinf(s->sm_scale))
    return DELTA_ERR_INVALID_ARG;
  if (s->n_q_heads % s->n_kv_heads != 0) return DELTA_ERR_INVALID_ARG;
  if ((int64_t)s->max_seq_len > (int64_t)s->max_pages_per_seq * 16) return DELTA_ERR_INVALID_ARG;
  if (s->page_size != 16) return DELTA_ERR_UNSUPPORTED;
  if (s->head_dim != 64 && s->head_dim != 128) return DELTA_ERR_UNSUPPORTED;
  const int G = s->n_q_heads / s->n_kv_heads;
  if (G > kMaxGroup) return DELTA_ERR_UNSUPPORTED;
  if ((int64_t)s->batch * s->n_q_heads > (1 << 24) || s->batch > 65535 || s->n_kv_heads > 65535)
    return DELTA_ERR_UNSUPPORTED;
  return DELTA_OK;
}

// The recency window in units.  App. A, Alg. 1 keeps the last ceil(L / P) pages for a window
// of L tokens, so any token count is valid: the window is the last ceil(l / U) units.
int recent_units_of(const delta_select_t* sel) {
  return ceil_div(sel->recent_tokens, sel->unit_tokens);
}

int check_select(const delta_select_t* sel) {
  if (!sel) return DELTA_ERR_INVALID_ARG;
  if (sel->unit_tokens != 16 && sel->unit_tokens != 1) return DELTA_ERR_UNSUPPORTED;
  if (sel->agg != DELTA_AGG_MAX && sel->agg != DELTA_AGG_SUM) return DELTA_ERR_INVALID_ARG;
  if (sel->delta_path != DELTA_PATH_AUTO && sel->delta_path != DELTA_PATH_SPLIT &&
      sel->delta_path != DELTA_PATH_FUSED)
    return DELTA_ERR_INVALID_ARG;
  if (sel->budget_tokens < 1 || sel->recent_tokens < 0) return DELTA_ERR_INVALID_ARG;
  if (sel->budget_tokens % sel->unit_tokens) return DELTA_ERR_INVALID_ARG;
  // L < K, counted in units (a window that rounds up to the whole budget leaves no choice);
  // the token comparison comes first and keeps the rounding below from overflowing
  if (sel->recent_tokens >= sel->budget_tokens ||
      recent_units_of(sel) >= sel->budget_tokens / sel->unit_tokens)
    return DELTA_ERR_INVALID_ARG;
  return DELTA_OK;
}

int make_layout(const delta_shape_t* s, const delta_select_t* sel, Layout* L) {
  int rc = check_shape(s);
  if (rc) return rc;
  if (sel && (rc = check_select(sel))) return rc;
  const int pairs = s->batch * s->n_kv_heads;
  const int G = s->n_q_heads / s->n_kv_heads;
  if (!plan_split(pairs, ceil_div(s->max_seq_len, 16), kMaxRowSlots, &L->dense))
    return DELTA_ERR_UNSUPPORTED;
  plan_balance(s->batch, pairs, &L->dense);
  L->max_split = L->dense.slots;
  if (sel) {
    const int K = sel->budget_tokens / sel->unit_tokens;
    if (sel->unit_tokens == 16) {
      L->sparse_mode = ROWS_SEL_PAGE;
      if (!plan_split(pairs, K, kMaxRowSlots, &L->sparse)) return DELTA_ERR_UNSUPPORTED;
    } else {
      L->sparse_mode = ROWS_SEL_TOKEN;
      if (!plan_split(pairs, ceil_div(K, 16), kMaxRowSlots / 16, &L->sparse))
        return DELTA_ERR_UNSUPPORTED;
    }
    L->max_split = std::max(L->max_split, L->sparse.slots);
    // the selection holds the older units of one sequence in one workgroup's registers
    if (ceil_div(s->max_seq_len, sel->unit_tokens) - recent_units_of(sel) > kMaxSelectKeys)
      return DELTA_ERR_UNSUPPORTED;
  }
  L->logit_pages = ceil_div(s->max_seq_len, 16);
  // partial rows per (sequence, KV head): the split plan's, or the fused Delta kernel's chunks
  int part_splits = L->max_split;
  if (sel) {
    L->fused_chunks = ceil_div(L->logit_pages, kFusedChunkPages);
    part_splits = std::max(part_splits, L->fused_chunks);
  }
  size_t off = 0;
  L->status = off;    off = align_up(off + sizeof(uint32_t));   // debug builds' status word
  L->counters = off;  off = align_up(off + sizeof(int32_t) * (size_t)pairs * kCounterStride);
  L->part_ml = off;   off = align_up(off + sizeof(float) * (size_t)pairs * part_splits * G * 2);
  L->part_o = off;    off = align_up(off + sizeof(float) * (size_t)pairs * part_splits * G * s->head_dim);
  if (sel) {
    L->nu_stride = ceil_div(s->max_seq_len, sel->unit_tokens);
    L->logits = off;  off = align_up(off + sizeof(float) * (size_t)s->batch * L->logit_pages * s->n_q_heads * 16);
    L->lse = off;     off = align_up(off + sizeof(float) * (size_t)s->batch * s->n_q_heads);
    L->uscores = off; off = align_up(off + sizeof(float) * (size_t)s->batch * L->nu_stride);
    L->phys = off;    off = align_up(off + sizeof(int32_t) * (size_t)s->batch * (sel->budget_tokens / sel->unit_tokens));
    L->fcnt = off;    off = align_up(off + sizeof(int32_t) * (size_t)s->batch * kCounterStride);
    L->fflag = off;   off = align_up(off + sizeof(int32_t) * (size_t)s->batch * L->fused_chunks);
  }
  L->total = off;
  return DELTA_OK;
}

int check_kv(const delta_kv_t* kv) {
  if (!kv || !kv->k_cache || !kv->v_cache || !kv->page_table || !kv->seq_lens || kv->n_pages < 0)
    return DELTA_ERR_INVALID_ARG;
  return DELTA_OK;
}

float scale_log2(const delta_shape_t* s) {
  const float sc = s->sm_scale > 0.f ? s->sm_scale : 1.0f / sqrtf((float)s->head_dim);
  return sc * 1.4426950408889634f;
}

AttnArgs base_args(const delta_shape_t* s, const delta_kv_t* kv, const void* q, void* out,
                   const Layout& L, char* ws, const SplitPlan& plan) {
  AttnArgs a{};
  a.k_cache = static_cast<const uint16_t*>(kv->k_cache);
  a.v_cache = static_cast<const uint16_t*>(kv->v_cache);
  a.page_table = kv->page_table;
  a.seq_lens = kv->seq_lens;
  a.q = static_cast<const uint16_t*>(q);
  a.out = static_cast<uint16_t*>(out);
  a.part_o = reinterpret_cast<float*>(ws + L.part_o);
  a.part_ml = reinterpret_cast<float*>(ws + L.part_ml);
  a.counters = reinterpret_cast<int32_t*>(ws + L.counters);
  a.page_stride = (int64_t)s->n_kv_heads * 16 * s->head_dim;
  a.n_q_heads = s->n_q_heads;
  a.n_kv_heads = s->n_kv_heads;
  a.max_pages = s->max_pages_per_seq;
  a.logit_pages = L.logit_pages;
  a.n_split = plan.n_split;
  a.gps = plan.gps;
  a.max_groups = plan.max_groups;
  a.slots = plan.slots;
  a.chunk_min = plan.chunk_min;
  a.balance = plan.balance;
  a.scale_log2 = scale_log2(s);
  a.n_pages = kv->n_pages;
  a.max_seq_len = s->max_seq_len;
  a.status = reinterpret_cast<uint32_t*>(ws + L.status);
  return a;
}

int hip_rc(hipError_t e) { return e == hipSuccess ? DELTA_OK : DELTA_ERR_HIP; }

int run_full(const delta_shape_t* s, const delta_kv_t* kv, const void* q, void* out,
             const Layout& L, char* ws, hipStream_t st) {
  AttnArgs a = base_args(s, kv, q, out, L, ws, L.dense);
  return hip_rc(launch_attention(s->head_dim, s->n_q_heads / s->n_kv_heads, ROWS_DENSE, a,
                                 s->batch, st));
}

// Whether a Delta layer runs as one fused launch (logits kept in LDS) instead of attention +
// scoring + selection launches.  The fused kernel needs head_dim 128, a multiple of 4 KV
// heads, at most kFusedMaxQHeads query heads, at most 2048 selection candidates, and its grid
// of (chunks x sequences) must be resident on the device at once (otherwise its sequence
// barrier would mostly run into its time limit and fall back to the slow path).  It pays off
// only when that grid also fills the device, one workgroup per CU or more: then every CU
// streams and the fused kernel saves the logit round trip and two launches; a smaller grid
// leaves CUs idle that the split attention launch would use.  sel->delta_path picks: SPLIT
// never, FUSED wherever it can run, AUTO where it can run and fills the device.
bool use_fused_delta(const delta_shape_t* s, const delta_select_t* sel, const Layout& L) {
  if (sel->delta_path == DELTA_PATH_SPLIT) return false;
  const int G = s->n_q_heads / s->n_kv_heads;
  if (s->head_dim != 128 || s->n_kv_heads % 4 != 0 || s->n_q_heads > kFusedMaxQHeads) return false;
  const int n_c = L.nu_stride - recent_units_of(sel);
  if (n_c > kFusedKeysPerThread * 256) return false;
  if (L.fused_chunks > kFusedMaxChunks) return false;
  const int64_t grid = (int64_t)L.fused_chunks * s->batch;
  const int64_t part_bytes = (int64_t)s->batch * s->n_q_heads * L.fused_chunks * s->head_dim * 4;
  if (part_bytes > 0x7fffffff) return false;
  // resident capacity per device, group size and unit size, and the device's CU count,
  // measured once
  static std::mutex mu;
  static int cache[64][kMaxGroup + 1][2];
  static int cus[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return false;
  const int ui = sel->unit_tokens == 16 ? 0 : 1;
  int cap = 0, n_cu = 0;
  {
    std::lock_guard<std::mutex> lock(mu);
    if (!cache[dev][G][ui]) cache[dev][G][ui] = 1 + fused_delta_capacity(s->head_dim, G, sel->unit_tokens);
    if (!cus[dev] && hipDeviceGetAttribute(&cus[dev], hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      cus[dev] = 0;
    cap = cache[dev][G][ui] - 1;
    n_cu = cus[dev];
  }
  if (grid > cap) return false;
  return sel->delta_path == DELTA_PATH_FUSED || (n_cu > 0 && grid >= n_cu);
}

// Longest wait of a fused-kernel workgroup at its sequence barrier: 1 ms of the 100 MHz
// real-time clock.  A resident sequence's workgroups arrive within tens of microseconds of each
// other, and one that is not resident starts at least an attention phase (~80 us at 32K) late,
// so 1 ms tells the two apart with a wide margin while bounding the stall of a launch that
// shares the device.  DELTA_FUSED_SPIN_TICKS overrides it (0: no wait, which forces the
// fallback of every workgroup but the last to arrive; for tests).
int64_t fused_spin_ticks() {
  const char* e = getenv("DELTA_FUSED_SPIN_TICKS");
  return e ? std::max<int64_t>(0, atoll(e)) : (int64_t)100000;
}

// A Delta layer: the fused kernel, or attention (logits on), scoring and selection.  `phys`
// (nullable): where the selection also writes the physical location of every selected unit,
// read through this layer's page table.
int run_delta(const delta_shape_t* s, const delta_kv_t* kv, const void* q, void* out,
              const delta_select_t* sel, int32_t* sel_idx, int32_t* sel_cnt, float* uscores,
              int32_t* phys, const Layout& L, char* ws, hipStream_t st) {
  SelectArgs xa{};
  xa.unit_scores = uscores ? uscores : reinterpret_cast<float*>(ws + L.uscores);
  xa.seq_lens = kv->seq_lens;
  xa.page_table = kv->page_table;
  xa.sel_idx = sel_idx;
  xa.sel_cnt = sel_cnt;
  xa.sel_phys = phys;
  xa.max_pages = s->max_pages_per_seq;
  xa.nu_stride = L.nu_stride;
  xa.unit_tokens = sel->unit_tokens;
  xa.budget_units = sel->budget_tokens / sel->unit_tokens;
  xa.recent_units = recent_units_of(sel);
  if (use_fused_delta(s, sel, L)) {
    FusedArgs f{};
    f.k_cache = static_cast<const uint16_t*>(kv->k_cache);
    f.v_cache = static_cast<const uint16_t*>(kv->v_cache);
    f.page_table = kv->page_table;
    f.seq_lens = kv->seq_lens;
    f.q = static_cast<const uint16_t*>(q);
    f.out = static_cast<uint16_t*>(out);
    f.part_o = reinterpret_cast<float*>(ws + L.part_o);
    f.part_ml = reinterpret_cast<float*>(ws + L.part_ml);
    f.counters = reinterpret_cast<int32_t*>(ws + L.fcnt);
    f.chunk_flags = reinterpret_cast<int32_t*>(ws + L.fflag);
    f.logits = reinterpret_cast<float*>(ws + L.logits);
    f.logit_pages = L.logit_pages;
    f.spin_ticks = fused_spin_ticks();
    f.unit_scores = const_cast<float*>(xa.unit_scores);
    f.page_stride = (int64_t)s->n_kv_heads * 16 * s->head_dim;
    f.n_q_heads = s->n_q_heads;
    f.n_kv_heads = s->n_kv_heads;
    f.max_pages = s->max_pages_per_seq;
    f.n_chunks = L.fused_chunks;
    f.max_seq_len = s->max_seq_len;
    f.agg = sel->agg;
    f.scale_log2 = scale_log2(s);
    f.sel = xa;
    f.n_pages = kv->n_pages;
    f.status = reinterpret_cast<uint32_t*>(ws + L.status);
    return hip_rc(launch_fused_delta(s->head_dim, s->n_q_heads / s->n_kv_heads, f, s->batch, st));
  }
  AttnArgs a = base_args(s, kv, q, out, L, ws, L.dense);
  a.logits = reinterpret_cast<float*>(ws + L.logits);
  a.lse = reinterpret_cast<float*>(ws + L.lse);
  int rc = hip_rc(launch_attention(s->head_dim, s->n_q_heads / s->n_kv_heads, ROWS_DENSE, a,
                                   s->batch, st));
  if (rc) return rc;
  ScoreArgs sa{};
  sa.logits = a.logits;
  sa.lse = a.lse;
  sa.seq_lens = kv->seq_lens;
  sa.unit_scores = const_cast<float*>(xa.unit_scores);
  sa.n_q_heads = s->n_q_heads;
  sa.n_kv_heads = s->n_kv_heads;
  sa.logit_pages = L.logit_pages;
  sa.nu_stride = L.nu_stride;
  sa.max_seq_len = s->max_seq_len;
  rc = hip_rc(launch_score(sel->agg, sel->unit_tokens, sa, s->batch, st));
  if (rc) return rc;
  return hip_rc(launch_select(xa, s->batch, st));
}

// `phys` (nullable): physical locations of `sel_idx` under this layer's page table, which
// spare the kernel the page-table lookup.
int run_sparse(const delta_shape_t* s, const delta_kv_t* kv, const void* q, void* out,
               const delta_select_t* sel, const int32_t* sel_idx, const int32_t* sel_cnt,
               const int32_t* phys, const Layout& L, char* ws, hipStream_t st) {
  AttnArgs a = base_args(s, kv, q, out, L, ws, L.sparse);
  a.sel_idx = sel_idx;
  a.sel_cnt = sel_cnt;
  a.sel_phys = phys;
  a.sel_stride = sel->budget_tokens / sel->unit_tokens;
  return hip_rc(launch_attention(s->head_dim, s->n_q_heads / s->n_kv_heads, L.sparse_mode, a,
                                 s->batch, st));
}

// Argument checks of a decoding step (every layer's buffers, roles and selection slots) and
// its workspace layout.  Nothing is enqueued.
int check_step(const delta_shape_t* shape, int32_t n_layers, const int32_t* roles,
               const delta_kv_t* kv, const void* const* q, void* const* out,
               const delta_select_t* sel, int32_t* sel_idx, int32_t* sel_cnt, Layout* L) {
  if (n_layers < 0 || (n_layers > 0 && (!roles || !kv || !q || !out))) return DELTA_ERR_INVALID_ARG;
  int n_delta = 0, n_sel_users = 0;
  for (int i = 0; i < n_layers; ++i) {
    if (roles[i] < DELTA_ROLE_FULL || roles[i] > DELTA_ROLE_SPARSE) return DELTA_ERR_INVALID_ARG;
    n_delta += roles[i] == DELTA_ROLE_DELTA;
    n_sel_users += roles[i] != DELTA_ROLE_FULL;
  }
  if (n_sel_users && !sel) return DELTA_ERR_INVALID_ARG;
  if (n_delta && (!sel_idx || !sel_cnt)) return DELTA_ERR_INVALID_ARG;
  int rc = make_layout(shape, n_sel_users ? sel : nullptr, L);
  if (rc) return rc;
  for (int i = 0; i < n_layers; ++i) {
    if ((rc = check_kv(&kv[i]))) return rc;
    if (!q[i] || !out[i]) return DELTA_ERR_INVALID_ARG;
  }
  return DELTA_OK;
}

// The layer loop of App. A, Alg. 1 over a checked step, on workspace `w` laid out as `L`.
int enqueue_step(const delta_shape_t* shape, int32_t n_layers, const int32_t* roles,
                 const delta_kv_t* kv, const void* const* q, void* const* out,
                 const delta_select_t* sel, int32_t* sel_idx, int32_t* sel_cnt, const Layout& L,
                 char* w, void* stream, const delta_hooks_t* hooks) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int K = sel ? sel->budget_tokens / sel->unit_tokens : 0;
  const size_t slot = (size_t)shape->batch * K;
  int cur = -1;   // most recent Delta slot; -1 = every unit (App. A, Alg. 1 initialisation)
  // Each Delta layer also leaves the physical locations of its selection in the workspace,
  // read through its page table; later sparse layers that share that page table use them.
  int32_t* phys = sel ? reinterpret_cast<int32_t*>(w + L.phys) : nullptr;
  const int32_t* phys_pt = nullptr;
  int rc = DELTA_OK;
  for (int i = 0; i < n_layers; ++i) {
    if (hooks && hooks->before_attn && hooks->before_attn(i, hooks->user, stream))
      return DELTA_ERR_HOOK;
    if (roles[i] == DELTA_ROLE_FULL || (roles[i] == DELTA_ROLE_SPARSE && cur < 0)) {
      rc = run_full(shape, &kv[i], q[i], out[i], L, w, st);
    } else if (roles[i] == DELTA_ROLE_DELTA) {
      ++cur;
      rc = run_delta(shape, &kv[i], q[i], out[i], sel, sel_idx + cur * slot,
                     sel_cnt + (size_t)cur * shape->batch, nullptr, phys, L, w, st);
      phys_pt = kv[i].page_table;
    } else {
      rc = run_sparse(shape, &kv[i], q[i], out[i], sel, sel_idx + cur * slot,
                      sel_cnt + (size_t)cur * shape->batch,
                      kv[i].page_table == phys_pt ? phys : nullptr, L, w, st);
    }
    if (rc) return rc;
    if (hooks && hooks->after_attn && hooks->after_attn(i, hooks->user, stream))
      return DELTA_ERR_HOOK;
  }
  return DELTA_OK;
}

}  // namespace

// Only the C ABI is exported; everything else in the library has hidden visibility.
#pragma GCC visibility push(default)
extern "C" {

int delta_workspace_bytes(const delta_shape_t* shape, const delta_select_t* sel, size_t* out) {
  if (!out) return DELTA_ERR_INVALID_ARG;
  Layout L;
  int rc = make_layout(shape, sel, &L);
  if (rc) return rc;
  *out = L.total;
  return DELTA_OK;
}

int delta_delta_path(const delta_shape_t* shape, const delta_select_t* sel, int* fused) {
  if (!fused || !sel) return DELTA_ERR_INVALID_ARG;
  Layout L;
  int rc = make_layout(shape, sel, &L);
  if (rc) return rc;
  *fused = use_fused_delta(shape, sel, L) ? 1 : 0;
  return DELTA_OK;
}

int delta_workspace_init(void* ws, size_t ws_bytes, void* stream) {
  if (!ws && ws_bytes) return DELTA_ERR_INVALID_ARG;
  return hip_rc(launch_fill_zero(ws, ws_bytes, static_cast<hipStream_t>(stream)));
}

int delta_full_attn(const delta_shape_t* shape, const delta_kv_t* kv, const void* q, void* out,
                    void* ws, size_t ws_bytes, void* stream) {
  Layout L;
  int rc = make_layout(shape, nullptr, &L);
  if (rc) return rc;
  if ((rc = check_kv(kv))) return rc;
  if (!q || !out || !ws) return DELTA_ERR_INVALID_ARG;
  if (ws_bytes < L.total) return DELTA_ERR_WORKSPACE;
  return run_full(shape, kv, q, out, L, static_cast<char*>(ws), static_cast<hipStream_t>(stream));
}

int delta_delta_attn_select(const delta_shape_t* shape, const delta_kv_t* kv, const void* q,
                            void* out, const delta_select_t* sel, int32_t* sel_idx,
                            int32_t* sel_cnt, int32_t* sel_phys, float* unit_scores, void* ws,
                            size_t ws_bytes, void* stream) {
  if (!sel) return DELTA_ERR_INVALID_ARG;
  Layout L;
  int rc = make_layout(shape, sel, &L);
  if (rc) return rc;
  if ((rc = check_kv(kv))) return rc;
  if (!q || !out || !ws || !sel_idx || !sel_cnt) return DELTA_ERR_INVALID_ARG;
  if (ws_bytes < L.total) return DELTA_ERR_WORKSPACE;
  return run_delta(shape, kv, q, out, sel, sel_idx, sel_cnt, unit_scores, sel_phys, L,
                   static_cast<char*>(ws), static_cast<hipStream_t>(stream));
}

int delta_sparse_attn(const delta_shape_t* shape, const delta_kv_t* kv, const void* q,
                      void* out, const delta_select_t* sel, const int32_t* sel_idx,
                      const int32_t* sel_cnt, const int32_t* sel_phys, void* ws,
                      size_t ws_bytes, void* stream) {
  if (!sel) return DELTA_ERR_INVALID_ARG;
  Layout L;
  int rc = make_layout(shape, sel, &L);
  if (rc) return rc;
  if ((rc = check_kv(kv))) return rc;
  if (!q || !out || !ws || !sel_idx || !sel_cnt) return DELTA_ERR_INVALID_ARG;
  if (ws_bytes < L.total) return DELTA_ERR_WORKSPACE;
  return run_sparse(shape, kv, q, out, sel, sel_idx, sel_cnt, sel_phys, L,
                    static_cast<char*>(ws), static_cast<hipStream_t>(stream));
}

int delta_kv_append(const delta_shape_t* shape, void* k_cache, void* v_cache,
                    const int32_t* page_table, const int32_t* seq_lens, const void* k_new,
                    const void* v_new, void* stream) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if (!k_cache || !v_cache || !page_table || !seq_lens || !k_new || !v_new)
    return DELTA_ERR_INVALID_ARG;
  AppendArgs a{};
  a.k_cache = static_cast<uint16_t*>(k_cache);
  a.v_cache = static_cast<uint16_t*>(v_cache);
  a.page_table = page_table;
  a.seq_lens = seq_lens;
  a.k_new = static_cast<const uint16_t*>(k_new);
  a.v_new = static_cast<const uint16_t*>(v_new);
  a.page_stride = (int64_t)shape->n_kv_heads * 16 * shape->head_dim;
  a.n_kv_heads = shape->n_kv_heads;
  a.head_dim = shape->head_dim;
  a.max_pages = shape->max_pages_per_seq;
  a.n_pages = 0;   // no cache descriptor: the debug build checks the sign only
  return launch_kv_append(a, shape->batch, static_cast<hipStream_t>(stream)) == hipSuccess
             ? DELTA_OK : DELTA_ERR_HIP;
}

int delta_decode_step(const delta_shape_t* shape, int32_t n_layers, const int32_t* roles,
                      const delta_kv_t* kv, const void* const* q, void* const* out,
                      const delta_select_t* sel, int32_t* sel_idx, int32_t* sel_cnt, void* ws,
                      size_t ws_bytes, void* stream) {
  return delta_decode_step_hooked(shape, n_layers, roles, kv, q, out, sel, sel_idx, sel_cnt, ws,
                                  ws_bytes, stream, nullptr);
}

int delta_decode_step_hooked(const delta_shape_t* shape, int32_t n_layers, const int32_t* roles,
                             const delta_kv_t* kv, const void* const* q, void* const* out,
                             const delta_select_t* sel, int32_t* sel_idx, int32_t* sel_cnt,
                             void* ws, size_t ws_bytes, void* stream, const delta_hooks_t* hooks) {
  if (!ws) return DELTA_ERR_INVALID_ARG;
  Layout L;
  int rc = check_step(shape, n_layers, roles, kv, q, out, sel, sel_idx, sel_cnt, &L);
  if (rc) return rc;
  if (ws_bytes < L.total) return DELTA_ERR_WORKSPACE;
  return enqueue_step(shape, n_layers, roles, kv, q, out, sel, sel_idx, sel_cnt, L,
                      static_cast<char*>(ws), stream, hooks);
}

int delta_decode_step_noalloc(const delta_shape_t* shape, int32_t n_layers, const int32_t* roles,
                              const delta_kv_t* kv, const void* const* q, void* const* out,
                              const delta_select_t* sel, int32_t* sel_idx, int32_t* sel_cnt,
                              void* stream) {
  Layout L;
  int rc = check_step(shape, n_layers, roles, kv, q, out, sel, sel_idx, sel_cnt, &L);
  if (rc) return rc;
  if (L.total > kNoallocScratchBytes) return DELTA_ERR_WORKSPACE;   // before any device call
  void* ws = nullptr;
  if (noalloc_scratch(&ws) != hipSuccess) return DELTA_ERR_HIP;
  char* w = static_cast<char*>(ws);
  // The scratch keeps whatever the previous call on this device left, laid out for that call's
  // shape; the arrival counters of this call's layout must start at zero (every other region is
  // written before it is read, and the kernels re-arm the counters they use).
  hipStream_t st = static_cast<hipStream_t>(stream);
  const size_t fused_bytes = L.fcnt ? L.total - L.fcnt : 0;   // fused counters and chunk flags
  // (from byte 0: the debug builds' status word, then the counters)
  if (launch_fill_zero2(w, L.part_ml, w + L.fcnt, fused_bytes, st) != hipSuccess)
    return DELTA_ERR_HIP;
  return enqueue_step(shape, n_layers, roles, kv, q, out, sel, sel_idx, sel_cnt, L, w, stream,
                      nullptr);
}

int delta_build_flags(void) { return DELTA_DEBUG ? DELTA_BUILD_DEBUG : 0; }

const char* delta_status_string(int status) {
  switch (status) {
    case DELTA_OK: return "ok";
    case DELTA_ERR_INVALID_ARG: return "invalid argument";
    case DELTA_ERR_UNSUPPORTED: return "unsupported shape or parameter";
    case DELTA_ERR_WORKSPACE: return "workspace too small";
    case DELTA_ERR_HIP: return "HIP launch failed";
    case DELTA_ERR_HOOK: return "a layer hook stopped the step";
    default: return "unknown status";
  }
}

}  // extern "C"
#pragma GCC visibility pop

/*
 * delta_attn.h — C ABI of the DELTA decode-step attention hot path on MI355X (gfx950).
 *
 * DELTA (arXiv 2510.09883) keeps the whole KV cache resident and splits the layers of one
 * decoding step into three roles (App. A, Alg. 1):
 *   FULL   decode attention over every cached token (Sec. 2, Eq. gqa_attention);
 *   DELTA  the same full attention, whose softmax weights are then turned into token scores
 *          (largest weight over all query heads), summed per page, and used to keep the last
 *          L pages plus the top-(K-L) older pages (Sec. 4 "Selection mechanism" and
 *          "Page-based DELTA"; App. A, Alg. 2);
 *   SPARSE decode attention restricted to the selected pages (App. A, Alg. 1).
 *
 * Conventions shared by every entry point
 *   Memory.   Structs, the `roles` array and the per-layer pointer arrays of delta_decode_step
 *             are HOST memory.  Every other pointer is DEVICE memory owned by the caller.  The
 *             library never allocates, frees, keeps a pointer, or synchronises `stream`
 *             (a hipStream_t passed as void*; NULL = the default stream).  All work is
 *             enqueued on `stream` in order.
 *   Errors.   Every call returns a status (DELTA_OK = 0, negative on error).  All argument
 *             checks run on the host before anything is enqueued, so a call that returns an
 *             error has enqueued nothing and left every output untouched (except
 *             DELTA_ERR_HOOK: a caller's hook stopped a hooked step part way).  DELTA_ERR_HIP
 *             means a launch was rejected by the HIP runtime.
 *   Device-side preconditions (not checked): page-table entries name pages that exist;
 *             1 <= seq_lens[b] <= max_seq_len; inputs are finite; selected indices were made by
 *             delta_delta_attn_select for the same shape and selection parameters.
 *   Layouts.  bf16 = IEEE bfloat16 bits.  q, out: [batch, n_q_heads, head_dim].
 *             k_cache, v_cache: [n_phys_pages, n_kv_heads, page_size, head_dim] (one contiguous
 *             page_size x head_dim tile per page and KV head).
 *             page_table: int32 [batch, max_pages_per_seq], logical page -> physical page.
 *             Query head j reads KV head j / (n_q_heads / n_kv_heads).
 *   Numerics. bf16 inputs, fp32 accumulation and online softmax, bf16 round-to-nearest-even
 *             outputs.  Results are deterministic: the same inputs and shape give bitwise
 *             identical outputs, and a DELTA layer's attention output is bitwise identical to
 *             delta_full_attn's on the same inputs when it runs the split path (with the fused
 *             DELTA kernel, see DELTA_PATH_*, the two agree up to floating-point summation
 *             order).
 *             FULL and DELTA calls over 2 to 64 sequences split the batch's work evenly over
 *             the GPU from the actual sequence lengths, so a sequence's output bits (never
 *             its accuracy) can depend on the other sequences' lengths in the same call;
 *             DELTA_ATTN_BALANCE=0 in the environment (read once per process) keeps the
 *             per-sequence split, whose bits depend on the sequence and the shape only.
 *   Workspace. `ws` is caller-owned device memory of at least delta_workspace_bytes() bytes.
 *             It must be zero-filled once after allocation; every call leaves it ready for the
 *             next call with the same shape and selection parameters.  Calls with another
 *             shape or selection may use it after delta_workspace_init (and when it is large
 *             enough for them).  Calls that share one workspace must not run concurrently.
 */
#ifndef DELTA_ATTN_H
#define DELTA_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  DELTA_OK = 0,
  DELTA_ERR_INVALID_ARG = -1,  /* null pointer, inconsistent sizes, L >= K, ...            */
  DELTA_ERR_UNSUPPORTED = -2,  /* valid but not built: head_dim, group size, page size      */
  DELTA_ERR_WORKSPACE = -3,    /* ws_bytes smaller than delta_workspace_bytes()             */
  DELTA_ERR_HIP = -4,          /* the HIP runtime rejected a launch                          */
  DELTA_ERR_HOOK = -5          /* a delta_decode_step_hooked callback returned non-zero      */
};

enum { DELTA_ROLE_FULL = 0, DELTA_ROLE_DELTA = 1, DELTA_ROLE_SPARSE = 2 };

/* Token score aggregation over query heads.  MAX is the paper's rule (Sec. 4 "Selection
 * mechanism"; App. A, Alg. 2); SUM is offered as an alternative. */
enum { DELTA_AGG_MAX = 0, DELTA_AGG_SUM = 1 };

/* Problem shape of one layer (Sec. 2: m query heads, g KV groups, d_head). */
typedef struct {
  int32_t batch;              /* B >= 1                                                      */
  int32_t n_q_heads;          /* m, a multiple of n_kv_heads                                  */
  int32_t n_kv_heads;         /* g; supported group sizes m/g: 1..8                           */
  int32_t head_dim;           /* d_head: 64 or 128                                            */
  int32_t page_size;          /* P: must be 16 (Sec. 5 "Implementation details")             */
  int32_t max_pages_per_seq;  /* row length of page_table                                     */
  int32_t max_seq_len;        /* host upper bound of seq_lens[b]; sizes grids and workspace  */
  float sm_scale;             /* softmax scale; 0 selects 1/sqrt(head_dim) (Eq. gqa_attention) */
} delta_shape_t;

/* One layer's paged KV cache (Sec. 4 "Page-based DELTA"; never evicted, Sec. 4). */
typedef struct {
  const void* k_cache;        /* bf16 [n_phys_pages, n_kv_heads, page_size, head_dim]         */
  const void* v_cache;        /* bf16, same layout                                            */
  const int32_t* page_table;  /* int32 [batch, max_pages_per_seq]                             */
  const int32_t* seq_lens;    /* int32 [batch]: tokens cached, the current one included       */
  int64_t n_pages;            /* n_phys_pages, or 0 if not stated; read by the debug build's
                                 checks of page-table entries only                           */
} delta_kv_t;

/* Selection parameters (Sec. 4; App. A, Alg. 2).  All counts are in TOKENS.  The budget must
 * be whole units: k = K*U.  The recency window may be any token count l >= 0: it keeps the last
 * L = ceil(l / U) units (App. A, Alg. 1 rounds the window up to whole pages), and L < K is
 * required.  unit_tokens U = 16 is page-based DELTA (the paper's configuration); U = 1 is the
 * token-level rule of Sec. 4.  A sequence may have at most 8192 candidate units (units older
 * than the recency window): 131072 tokens with pages, about 8192 with single tokens; larger
 * shapes return DELTA_ERR_UNSUPPORTED. */
typedef struct {
  int32_t budget_tokens;      /* k: tokens kept per sequence, a multiple of U, > recent       */
  int32_t recent_tokens;      /* l: most recent tokens always kept (ceil(l/U) units), >= 0   */
  int32_t unit_tokens;        /* U: 16 (pages) or 1 (tokens)                                  */
  int32_t agg;                /* DELTA_AGG_MAX (paper) or DELTA_AGG_SUM                       */
  int32_t delta_path;         /* DELTA_PATH_AUTO (0), _SPLIT or _FUSED: how DELTA layers run  */
} delta_select_t;

/* How a DELTA layer is executed (same selection either way; see delta_delta_attn_select):
 *   DELTA_PATH_SPLIT  attention (logits staged through the workspace), scoring and selection
 *                     launches; the layer's attention output is bitwise delta_full_attn's.
 *   DELTA_PATH_FUSED  one kernel that keeps the logits on chip, wherever it can run: head_dim
 *                     128, a multiple of 4 KV heads, at most 32 query heads, at most 2048
 *                     candidate units and a grid of ceil(max_seq_len / 1024) x batch workgroups
 *                     that the device holds at once; elsewhere the split launches.  Its output
 *                     equals delta_full_attn's up to floating-point summation order (within the
 *                     bf16 rounding of the result), not bit for bit.
 *   DELTA_PATH_AUTO   the fused kernel where it can run and its grid also fills the device (at
 *                     least one workgroup per CU), which is where it is the faster of the two on
 *                     MI355X; the split launches elsewhere.  */
enum { DELTA_PATH_AUTO = 0, DELTA_PATH_SPLIT = 1, DELTA_PATH_FUSED = 2 };

/* Bytes of workspace needed by every call with this shape (and, if non-NULL, these selection
 * parameters; pass the same `sel` used for DELTA and SPARSE calls).  Host only. */
int delta_workspace_bytes(const delta_shape_t* shape, const delta_select_t* sel, size_t* out);

/* Zero-fills `ws_bytes` bytes of `ws` on `stream` with a kernel (safe under stream capture).
 * Equivalent to allocating the workspace zero-filled. */
int delta_workspace_init(void* ws, size_t ws_bytes, void* stream);

/* FULL role: out[b, j, :] = sum_t softmax_t(sm_scale * q[b,j].k_t) v_t over all seq_lens[b]
 * tokens of sequence b, k_t/v_t read from KV head j / G (Sec. 2, Eq. gqa_attention;
 * App. A, Alg. 1 full branch).  One kernel launch.
 *   q:   bf16 [B, m, d]   out: bf16 [B, m, d] */
int delta_full_attn(const delta_shape_t* shape, const delta_kv_t* kv, const void* q, void* out,
                    void* ws, size_t ws_bytes, void* stream);

/* DELTA role: the FULL computation (the same `out`; see DELTA_PATH_*), then RefreshPages (App. A,
 * Alg. 2): token score s_t = max over all m heads of softmax weight (Sec. 4), unit score
 * S_u = sum of s_t over the U tokens of unit u (a partial last unit sums the tokens it has),
 * and the selected set = the last L units plus the top-(K-L) of the older units by S_u,
 * equal scores taken lower index first.  When a sequence has n_u <= K units, all are kept.
 *   sel_idx:     int32 [B, K] (K = budget_tokens / U): the selected logical unit indices of
 *                each sequence in ascending order; entries at and past sel_cnt[b] are -1.
 *   sel_cnt:     int32 [B]: min(K, ceil(seq_lens[b] / U)).
 *   sel_phys:    optional int32 [B, K]: where each selected unit lives, read through
 *                kv->page_table: its physical page (U = 16) or physical page * 16 + row
 *                (U = 1); -1 where sel_idx is -1.  Handing it to delta_sparse_attn spares
 *                every sparse layer that shares this page table the page-table lookup.
 *                NULL: not written.
 *   unit_scores: optional fp32 [B, ceil(max_seq_len / U)]: S_u for u < ceil(seq_lens[b]/U);
 *                NULL keeps them in the workspace.
 * Launches, by sel->delta_path: the split path runs the attention kernel (which stages the
 * logits through the workspace), a scoring kernel and a selection kernel; the fused path one
 * kernel that keeps the logits on chip (with DELTA_PATH_AUTO, e.g. 8 sequences of 32K tokens
 * with 28 query and 4 KV heads, where its 256 workgroups fill the 256 CUs).  The fused kernel's
 * workgroups wait for the rest of their sequence for at most DELTA_FUSED_SPIN_TICKS ticks of the
 * 100 MHz clock (environment, default 1 ms) and then hand their part to the sequence's last
 * workgroup, so it never hangs when not all of them are resident, and gives the same results
 * either way. */
int delta_delta_attn_select(const delta_shape_t* shape, const delta_kv_t* kv, const void* q,
                            void* out, const delta_select_t* sel, int32_t* sel_idx,
                            int32_t* sel_cnt, int32_t* sel_phys, float* unit_scores, void* ws,
                            size_t ws_bytes, void* stream);

/* Which path delta_delta_attn_select takes for this shape and selection (sel->delta_path) on
 * the current device: *fused = 1 for the fused kernel, 0 for the attention, scoring and
 * selection launches.  Host only; it queries the current device's CU count and its occupancy
 * for the fused kernel (without a device: 0 unless the kernel cannot apply anyway).  Errors as
 * delta_workspace_bytes; `sel` and `fused` must be non-NULL. */
int delta_delta_path(const delta_shape_t* shape, const delta_select_t* sel, int* fused);

/* SPARSE role: attention of each query over the tokens of the selected units only, the
 * softmax renormalised over them (App. A, Alg. 1 sparse branch).  Unit u covers tokens
 * [u*U, min(u*U + U, seq_lens[b])).  sel_idx / sel_cnt as produced by
 * delta_delta_attn_select with the same `sel`.  sel_phys: NULL, or the sel_phys that the
 * same delta_delta_attn_select call wrote, valid only while kv->page_table is the page table
 * (pointer and contents) that call read; it then replaces the page-table lookups.  One kernel
 * launch. */
int delta_sparse_attn(const delta_shape_t* shape, const delta_kv_t* kv, const void* q,
                      void* out, const delta_select_t* sel, const int32_t* sel_idx,
                      const int32_t* sel_cnt, const int32_t* sel_phys, void* ws,
                      size_t ws_bytes, void* stream);

/* One decoding step over a layer stack (App. A, Alg. 1).  roles[i] in DELTA_ROLE_*; kv, q and
 * out are HOST arrays of n_layers entries (q[i], out[i] device pointers as above).  The
 * selected set starts as every unit; each DELTA layer writes its own slot
 * sel_idx[d] ([B, K]) and sel_cnt[d] ([B]), d counting DELTA layers from 0, and every later
 * SPARSE layer reads the most recent slot.  A SPARSE layer before the first DELTA layer
 * attends to every unit, i.e. runs FULL.  sel may be NULL only if no layer is DELTA/SPARSE.
 * The physical locations of the current selection are kept in the workspace and used by the
 * SPARSE layers whose kv[i].page_table pointer equals that of the DELTA layer that selected.
 * Enqueues only kernels, so the whole step can be captured into a HIP graph. */
int delta_decode_step(const delta_shape_t* shape, int32_t n_layers, const int32_t* roles,
                      const delta_kv_t* kv, const void* const* q, void* const* out,
                      const delta_select_t* sel, int32_t* sel_idx, int32_t* sel_cnt,
                      void* ws, size_t ws_bytes, void* stream);

/* KV append (Sec. 2, Eq. kv_update: the cache grows by the decoding token before attention
 * reads it).  For every sequence b, writes the new token's key and value rows of every KV head
 * into the paged cache of one layer.  seq_lens[b] already counts the new token, so its row is
 * s_b - 1: row (s_b - 1) % page_size of physical page page_table[b, (s_b - 1) / page_size].
 *   k_cache, v_cache: bf16 [n_phys_pages, n_kv_heads, page_size, head_dim], written in place
 *                     (only those rows);
 *   page_table, seq_lens: as in delta_kv_t (the caller has already mapped the page);
 *   k_new, v_new:     bf16 [batch, n_kv_heads, head_dim].
 * Uses batch, n_kv_heads, head_dim, page_size and max_pages_per_seq of `shape`.  A sequence
 * with seq_lens[b] < 1 or > max_pages_per_seq * page_size is skipped (nothing is written).
 * One kernel launch; no workspace; the rows are bitwise copies. */
int delta_kv_append(const delta_shape_t* shape, void* k_cache, void* v_cache,
                    const int32_t* page_table, const int32_t* seq_lens, const void* k_new,
                    const void* v_new, void* stream);

/* Host callbacks around each layer's attention in delta_decode_step_hooked.  A hook runs on
 * the calling thread while the step is being enqueued, receives the layer index, `user` and
 * the step's stream, and enqueues its own work on that stream (for example the layer's QKV
 * projection and delta_kv_append before the attention, the output projection and the FFN
 * after it), so that its work and the attention launches are ordered and a whole model step
 * can be captured into one HIP graph.  Return 0 to continue; any other value stops the step. */
typedef int (*delta_layer_hook_t)(int32_t layer, void* user, void* stream);
typedef struct {
  delta_layer_hook_t before_attn;   /* NULL: none */
  delta_layer_hook_t after_attn;    /* NULL: none */
  void* user;
} delta_hooks_t;

/* delta_decode_step with per-layer hooks (App. A, Alg. 1, with the rest of the decoder layer
 * around each attention: Sec. 2, Eq. gqa_projection, kv_update, gqa_output).  For layer
 * i = 0 .. n_layers-1: hooks->before_attn(i), the layer's attention as in delta_decode_step,
 * hooks->after_attn(i).  All arguments are checked before the first hook runs or anything is
 * enqueued; q[i] and kv[i] may point at buffers that before_attn(i) fills.  When a hook
 * returns non-zero the step stops and returns DELTA_ERR_HOOK, with the earlier layers' work
 * already enqueued.  hooks == NULL is delta_decode_step. */
int delta_decode_step_hooked(const delta_shape_t* shape, int32_t n_layers, const int32_t* roles,
                             const delta_kv_t* kv, const void* const* q, void* const* out,
                             const delta_select_t* sel, int32_t* sel_idx, int32_t* sel_cnt,
                             void* ws, size_t ws_bytes, void* stream, const delta_hooks_t* hooks);

/* Largest workspace the allocation-free step below can serve: the library's scratch array, one
 * per GPU, held from the first delta_decode_step_noalloc call on that GPU until the process
 * ends.  160 MiB covers a 32-layer step of 32 sequences of up to 32K tokens with 32 query and
 * 8 KV heads (delta_workspace_bytes: 145 MiB). */
#define DELTA_NOALLOC_SCRATCH_BYTES ((size_t)160 << 20)

/* delta_decode_step for callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops, harnesses that forbid hipMalloc): the same arguments and results
 * (bit for bit) without `ws` / `ws_bytes`; the library's own scratch array takes the
 * workspace's place.  It calls no hipMalloc, hipFree or other allocating routine (the first call
 * on a GPU looks up the array's address there, which loads it).  Each call first clears the
 * arrival counters in the scratch with a small kernel, then enqueues the step, so any sequence of
 * shapes may follow any other.  All calls on one GPU share its array: calls that may overlap on
 * one GPU (other streams, other threads) race and must be serialised by the caller.
 * Returns DELTA_ERR_WORKSPACE, before any device call, when delta_workspace_bytes() for this
 * shape and selection exceeds DELTA_NOALLOC_SCRATCH_BYTES; other errors as delta_decode_step. */
int delta_decode_step_noalloc(const delta_shape_t* shape, int32_t n_layers, const int32_t* roles,
                              const delta_kv_t* kv, const void* const* q, void* const* out,
                              const delta_select_t* sel, int32_t* sel_idx, int32_t* sel_cnt,
                              void* stream);

/* Build information: DELTA_BUILD_DEBUG is set in a library built with -DDELTA_DEBUG=1
 * (python -m paper_2510_09883_amd.build --debug: libdelta_attn_debug.so).  A debug build checks
 * on the device the preconditions that release builds only document: every page-table entry
 * and physical location it reads lies in [0, kv->n_pages) (only >= 0 when n_pages is 0), every
 * seq_lens[b] in [1, max_seq_len], every selected unit inside its sequence.  A failed check ORs
 * a DELTA_DEBUG_* bit into the 32-bit word at byte 0 of the workspace and the kernel goes on
 * with an in-range value (physical page 0, the length clamped, the unit masked), so it never
 * reads outside the caller's buffers; results are then meaningless but defined.  The word is
 * zero after delta_workspace_init; the caller reads it after synchronising the stream.  Release
 * builds never write it.  delta_kv_append has no workspace: in a debug build it skips a
 * sequence whose page-table entry fails the check. */
enum { DELTA_BUILD_DEBUG = 1 };
enum { DELTA_DEBUG_PAGE = 1, DELTA_DEBUG_SEQ_LEN = 2, DELTA_DEBUG_SELECTION = 4 };
int delta_build_flags(void);

/* Static description of a status code. */
const char* delta_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* DELTA_ATTN_H */

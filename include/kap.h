/*
 * kap.h -- C ABI of the KAP selected-KV decode / full-KV verify library for
 * AMD Instinct MI355X (gfx950).
 *
 * Paper: "KAP: Bridging the Knowledge Selection--Runtime Consumption Gap in
 * LLM Systems" (arXiv 2607.24260). The library implements the data-parallel
 * part of the GraphSpec executor:
 *
 *   kap_compile_plan     Alg. 1 (GraphSpecCompile): select evidence spans
 *                        under a token budget by prior score, resolve them to
 *                        KV pages, keep their logical positions and build the
 *                        proposal-side block table (Sec. 3.1).
 *   kap_selected_decode  one proposal step, q_prop = 1, whose attention reads
 *                        only the KV pages the plan exposes (Sec. 3.2,
 *                        "Selected-KV proposal").
 *   kap_verify           causal attention of the k+1 verify window over the
 *                        full paged KV cache (Sec. 3.2, "Full-context
 *                        verification"; Eq. (2)).
 *
 * Around them: kap_decode_schedule writes, once per view, the split map that
 * kap_selected_decode_scheduled then reads instead of computing it in every
 * proposal step (the view is fixed across the k steps of a cycle);
 * kap_selected_decode_masked takes token-granular views; kap_append_kv and
 * kap_compact_view maintain the pool; kap_fallback_update switches sequences
 * to full-context access (Sec. 3.2, "Runtime stability and fallback");
 * kap_accept_top3 scores draft windows.
 *
 * Conventions shared by every call
 * --------------------------------
 * - Every array argument is device memory owned by the caller. The library
 *   never allocates, frees or synchronises, and keeps no pointer after the
 *   call returns (kap_selected_decode_noalloc uses a scratch buffer the
 *   library holds per GPU instead of a workspace; see there). Work is enqueued on `stream` (a hipStream_t passed as
 *   void*; NULL = the default stream); the caller keeps every buffer alive
 *   until that work has completed.
 * - Scratch memory comes from the caller's `workspace`, at least the size the
 *   matching kap_*_workspace_bytes() call returns for the same arguments on
 *   the current device, 256-byte aligned. kap_selected_decode and kap_verify
 *   keep arrival counters in its first round_up(64 * batch * num_kv_heads,
 *   256) bytes: that block must be zero when the call starts, and every
 *   completed call leaves it zero again. Zero-fill a workspace once when
 *   allocating it (and again if a later call uses a larger batch *
 *   num_kv_heads); the rest of the workspace is scratch whose contents do not
 *   matter, so one workspace may serve any sequence of decode and verify calls
 *   that fit it. Calls that can run concurrently must not share a workspace.
 *   kap_compile_plan's workspace has no such block.
 * - Alignment: k_pages and v_pages, and the q and out arrays of decode and
 *   verify, must be 16-byte aligned (KAP_ERR_INVALID_ARGUMENT otherwise).
 * - Grid sizes depend only on host integers, never on device data, so the
 *   calls may be captured into a HIP graph.
 * - Host-checkable errors (null pointers, negative sizes, unsupported
 *   geometry or dtype, small workspace) return a non-zero kap_status before
 *   anything is enqueued. batch == 0 is a successful no-op. A failed launch
 *   returns KAP_ERR_HIP. kap_last_error() then describes the problem.
 * - Data-dependent problems of kap_compile_plan are reported per sequence in
 *   plan_status[] (KAP_PLAN_*); the call itself returns KAP_OK.
 * - kap_selected_decode and kap_verify never dereference a page id outside
 *   [0, num_pages): such a page contributes no keys. Results for such inputs
 *   are otherwise unspecified.
 *
 * KV cache layout (struct kap_kv_cache)
 * -------------------------------------
 *   k_pages: [num_pages][num_kv_heads][head_dim/8][page_size][8]
 *            each page's K tile grouped in 8-dim chunks: element
 *            [p][g][c][t][e] is dim 8c+e of token t
 *   v_pages: [num_pages][num_kv_heads][head_dim][page_size]  dim-major pages
 *   kv_scales (FP8 only): [num_pages][2] float, K scale then V scale; a stored
 *            E4M3FN code x of page p stands for decode(x) * scale.
 * Token t of logical page j of a sequence is its token 16*j + t; logical page j
 * lives in physical page block_table[j]. Query head h reads KV head
 * h / (num_q_heads / num_kv_heads).
 * Supported: page_size 16; head_dim 128 (64 and 256 on the generic path);
 * num_q_heads a multiple of num_kv_heads; kv_dtype F32 with q_dtype F32, or
 * kv_dtype BF16 / FP8_E4M3FN with q_dtype BF16.
 *
 * Outputs of attention are float32: out = softmax(z) V and lse = natural
 * log-sum-exp of z, with z = sm_scale * <q, k>. A row that sees no key gets
 * out = 0 and lse = -inf.
 */
#ifndef KAP_H_
#define KAP_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KAP_ABI_VERSION 1

typedef int32_t kap_status;
enum {
  KAP_OK = 0,
  KAP_ERR_INVALID_ARGUMENT = 1,
  KAP_ERR_UNSUPPORTED = 2,
  KAP_ERR_WORKSPACE_TOO_SMALL = 3,
  KAP_ERR_HIP = 4
};

typedef int32_t kap_dtype;
enum { KAP_DT_F32 = 0, KAP_DT_BF16 = 1, KAP_DT_FP8_E4M3FN = 2 };

/* What kap_compile_plan does with a span that does not fit the budget. */
typedef int32_t kap_select_policy;
enum { KAP_SELECT_SKIP = 0, KAP_SELECT_STOP = 1 };

/* Per-sequence plan status (fallback triggers, Sec. 3.2 "Runtime stability
 * and fallback"). Any value other than KAP_PLAN_OK means: the sequence's view
 * is empty (view_num_blocks = view_tokens = spans_taken = 0, its span_selected
 * flags are 0) and the executor must use full-context access. */
enum {
  KAP_PLAN_OK = 0,
  KAP_PLAN_OVER_CAPACITY = 1, /* the view needs more than view_capacity blocks */
  KAP_PLAN_BAD_SCORE = 2,     /* a prior score is NaN */
  KAP_PLAN_BAD_PAGE = 3,      /* a selected page id is outside [0, num_pages) */
  KAP_PLAN_BAD_LENGTH = 4,    /* seq_len < 1 or ceil(seq_len/16) > fbt_stride */
  KAP_PLAN_BAD_SPANS = 5      /* span_offsets[b..b+1] not within [0, num_spans] */
};

typedef struct kap_kv_cache {
  int32_t num_q_heads;  /* Hq */
  int32_t num_kv_heads; /* Hkv; Hq % Hkv == 0 */
  int32_t head_dim;     /* D */
  int32_t page_size;    /* tokens per page: 16 */
  kap_dtype kv_dtype;
  kap_dtype q_dtype;
  const void *k_pages;
  const void *v_pages;
  const float *kv_scales; /* FP8 only, else NULL */
  int64_t num_pages;
} kap_kv_cache;

/*
 * kap_compile_plan -- Alg. 1, SelectEvidenceUnderBudget through
 * EmitRuntimeAccessPlan, for `batch` sequences at once.
 *
 * Per sequence b (L = seq_lens[b], NP = ceil(L/16), valid(j) = min(16, L-16j)):
 *  1. Mandatory pages: those touched by tokens [0, min(prefix,L)) and by
 *     [max(0, L - max(suffix,1)), L); the page of the last token is always in.
 *     used = sum of valid(j) over the selected pages.
 *  2. Spans i in [span_offsets[b], span_offsets[b+1]) are clipped to [0, L)
 *     and ranked by (span_prior desc, span_start asc, i asc); -0 == +0.
 *  3. In rank order, a non-empty span whose not-yet-selected pages cost
 *     `cost` visible tokens is taken iff used + cost <= budget_tokens[b]
 *     (then used += cost). A span that does not fit is skipped
 *     (KAP_SELECT_SKIP) or ends selection (KAP_SELECT_STOP). Empty spans are
 *     ignored.
 *  4. view_logical_block[b][0..n) = selected logical pages ascending,
 *     view_block_table[b][k] = full_block_table[b][view_logical_block[b][k]],
 *     view_num_blocks[b] = n, view_tokens[b] = used (the numerator of the
 *     retained ratio s, Eq. (4)), spans_taken[b] = number of spans taken,
 *     span_selected[i] = 1 for taken spans else 0 (may be NULL).
 *
 * Arguments (device arrays unless noted):
 *   seq_lens [batch] int32; full_block_table [batch][fbt_stride] int32;
 *   span_offsets [batch+1] int32 (CSR); num_spans (host) = length of the span
 *   arrays; span_start, span_len [num_spans] int32; span_prior [num_spans]
 *   float32; prefix_tokens, suffix_tokens, budget_tokens [batch] int32;
 *   policy (host); num_pages (host) bounds valid page ids; view_capacity
 *   (host) = row stride of the view arrays and the most blocks a view may
 *   have; outputs view_block_table, view_logical_block [batch][view_capacity]
 *   int32 (entries past view_num_blocks[b] are left unchanged),
 *   view_num_blocks, view_tokens, spans_taken, plan_status [batch] int32,
 *   span_selected [num_spans] int32 or NULL.
 * Limits: fbt_stride <= 262144 pages per sequence.
 * Result is unique and bit-for-bit deterministic.
 */
kap_status kap_compile_plan(int32_t batch, const int32_t *seq_lens,
                            const int32_t *full_block_table, int32_t fbt_stride,
                            const int32_t *span_offsets, int32_t num_spans,
                            const int32_t *span_start, const int32_t *span_len,
                            const float *span_prior, const int32_t *prefix_tokens,
                            const int32_t *suffix_tokens, const int32_t *budget_tokens,
                            kap_select_policy policy, int64_t num_pages,
                            int32_t view_capacity, int32_t *view_block_table,
                            int32_t *view_logical_block, int32_t *view_num_blocks,
                            int32_t *view_tokens, int32_t *spans_taken,
                            int32_t *plan_status, int32_t *span_selected,
                            void *workspace, size_t workspace_bytes, void *stream);

size_t kap_compile_plan_workspace_bytes(int32_t batch, int32_t num_spans,
                                        int32_t fbt_stride);

/*
 * kap_compile_plan_masked -- kap_compile_plan with the visibility mask of
 * Sec. 3.1 kept at token resolution: a span is exposed as its tokens, not as
 * whole pages.
 *
 * Per sequence b, as kap_compile_plan except that selection is over token
 * sets:
 *  1. Mandatory tokens: [0, min(prefix,L)) and [max(0, L - max(suffix,1)), L).
 *     used = their number.
 *  2. Ranking as kap_compile_plan.
 *  3. A non-empty clipped span costs its tokens not yet visible; it is taken
 *     iff used + cost <= budget_tokens[b] (then its tokens become visible),
 *     else skipped or, with KAP_SELECT_STOP, selection ends.
 *  4. The view lists, ascending, every logical page holding a visible token;
 *     view_token_mask[b][k] (uint32, bits 16..31 zero) has bit t set iff token
 *     16*view_logical_block[b][k] + t is visible. view_tokens[b] = used.
 * Status codes, outputs and workspace are those of kap_compile_plan; the
 * extra output view_token_mask is [batch][view_capacity] (entries past
 * view_num_blocks[b] are left unchanged; may be NULL only if
 * view_capacity == 0).
 * Limits: fbt_stride <= 16384 pages per sequence (262144 tokens).
 * Result is unique and bit-for-bit deterministic.
 */
kap_status kap_compile_plan_masked(int32_t batch, const int32_t *seq_lens,
                                   const int32_t *full_block_table, int32_t fbt_stride,
                                   const int32_t *span_offsets, int32_t num_spans,
                                   const int32_t *span_start, const int32_t *span_len,
                                   const float *span_prior, const int32_t *prefix_tokens,
                                   const int32_t *suffix_tokens, const int32_t *budget_tokens,
                                   kap_select_policy policy, int64_t num_pages,
                                   int32_t view_capacity, int32_t *view_block_table,
                                   int32_t *view_logical_block, uint32_t *view_token_mask,
                                   int32_t *view_num_blocks, int32_t *view_tokens,
                                   int32_t *spans_taken, int32_t *plan_status,
                                   int32_t *span_selected, void *workspace,
                                   size_t workspace_bytes, void *stream);

/*
 * kap_selected_decode -- one proposal step (q_prop = 1) over the selected-KV
 * view (Sec. 3.2, "Selected-KV proposal").
 *
 * For sequence b and query head h, the visible keys are, for each
 * k < min(view_num_blocks[b], max_view_blocks), the tokens t < min(16,
 * seq_lens[b] - 16*view_logical_block[b][k]) of physical page
 * view_block_table[b][k]. The order of view blocks does not change the result.
 *   q [batch][Hq][D] (q_dtype); view arrays [batch][view_stride] int32 with
 *   view_stride >= max_view_blocks; view_num_blocks, seq_lens [batch] int32;
 *   out [batch][Hq][D] float32; lse [batch][Hq] float32.
 * num_splits (host): 0 = automatic -- the tuned path then sizes the key
 * splits of each (sequence, KV head) on the device from that sequence's
 * actual view, so ragged batches stay balanced; n > 0 forces n key splits
 * per (sequence, KV head) on the tuned path (clamped to max_view_blocks).
 * The generic path (other geometries and dtypes) splits keys into pieces of
 * at most 64 pages, finer when the call has few query rows, and takes at
 * least n pieces when n > 0. Results do not depend on the split count
 * beyond rounding.
 * Passing the full block table as the view, with view_logical_block[b][j] = j
 * and view_num_blocks[b] = ceil(seq_lens[b]/16), is full-context decode.
 */
kap_status kap_selected_decode(const kap_kv_cache *kv, int32_t batch, const void *q,
                               const int32_t *seq_lens, const int32_t *view_block_table,
                               const int32_t *view_logical_block, int32_t view_stride,
                               const int32_t *view_num_blocks, int32_t max_view_blocks,
                               float sm_scale, int32_t num_splits, float *out, float *lse,
                               void *workspace, size_t workspace_bytes, void *stream);

size_t kap_selected_decode_workspace_bytes(const kap_kv_cache *kv, int32_t batch,
                                           int32_t max_view_blocks, int32_t num_splits);

/*
 * kap_selected_decode_masked -- kap_selected_decode over a token-granular
 * view (the output of kap_compile_plan_masked): token t of view block k is
 * visible iff it is visible to kap_selected_decode AND bit t of
 * view_token_mask[b][k] is set.
 *   view_token_mask [batch][view_stride] uint32, laid out like the view
 *   tables (may be NULL only if max_view_blocks == 0). Every other argument,
 *   the workspace (kap_selected_decode_workspace_bytes) and the errors are
 *   those of kap_selected_decode.
 */
kap_status kap_selected_decode_masked(const kap_kv_cache *kv, int32_t batch, const void *q,
                                      const int32_t *seq_lens, const int32_t *view_block_table,
                                      const int32_t *view_logical_block,
                                      const uint32_t *view_token_mask, int32_t view_stride,
                                      const int32_t *view_num_blocks, int32_t max_view_blocks,
                                      float sm_scale, int32_t num_splits, float *out, float *lse,
                                      void *workspace, size_t workspace_bytes, void *stream);

/*
 * kap_selected_decode_noalloc -- kap_selected_decode for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc. It takes no workspace and allocates
 * nothing: the split partials and arrival counters live in a scratch buffer
 * the library holds on each GPU it runs on (16 MiB, kept until the process
 * ends; its address is looked up once per device, on the first call there).
 *
 * Arguments, results and every other error are those of kap_selected_decode.
 * Limits: the split partials the call needs -- what
 * kap_selected_decode_workspace_bytes() reports for the same arguments, less
 * its arrival-counter block -- at most 16 MiB - 256 KiB, else
 * KAP_ERR_WORKSPACE_TOO_SMALL; with split partials on the tuned path
 * (head_dim 128, four query heads per KV head), batch * num_kv_heads <=
 * 4096, else KAP_ERR_UNSUPPORTED. Both are reported before anything is
 * enqueued. The counters are zero when the library is loaded and every
 * completed call leaves them zero. All calls on one GPU share its scratch:
 * calls that may overlap in time on one GPU (on different streams, or from
 * different threads) race and give wrong results; keep them stream-ordered.
 */
kap_status kap_selected_decode_noalloc(const kap_kv_cache *kv, int32_t batch, const void *q,
                                       const int32_t *seq_lens, const int32_t *view_block_table,
                                       const int32_t *view_logical_block, int32_t view_stride,
                                       const int32_t *view_num_blocks, int32_t max_view_blocks,
                                       float sm_scale, int32_t num_splits, float *out, float *lse,
                                       void *stream);

/*
 * kap_decode_schedule / kap_selected_decode_scheduled -- kap_selected_decode
 * with its split assignment computed once per view. The view stays fixed over
 * the k proposal steps of a cycle (Sec. 3.2, "Selected-KV proposal"), so the
 * balanced split map that kap_selected_decode derives at the start of every
 * call from all view lengths -- before its first page loads -- can be derived
 * once by kap_decode_schedule and reused by every decode call on that view:
 * each workgroup then starts from its record (its work item and its
 * wavefronts' first view entries) and issues its first page loads at once.
 *
 * kap_decode_schedule_bytes returns the schedule size for the kv geometry,
 * batch and max_view_blocks on the current device; 0 means these calls use
 * no balanced map (one split per (sequence, KV head), or the generic path),
 * and the schedule is then neither written nor read (it may be NULL).
 * kap_decode_schedule writes the schedule -- caller-owned device memory,
 * 16-byte aligned -- from seq_lens, the view arrays (view_token_mask NULL for
 * page-granular views) and view_num_blocks, laid out as for
 * kap_selected_decode.
 *
 * kap_selected_decode_scheduled takes the arguments of kap_selected_decode
 * with num_splits = 0 (view_token_mask NULL: page-granular; otherwise as
 * kap_selected_decode_masked) plus the schedule, and returns the same results
 * bit for bit. The schedule must have been written by kap_decode_schedule on
 * this device for the same kv geometry and dtypes, batch, seq_lens, view
 * arrays, view_stride, view_num_blocks and max_view_blocks, unchanged since
 * (write it again whenever kap_compile_plan or kap_fallback_update rewrites
 * the view). With any other schedule the results, and the workspace's
 * arrival counters, are undefined; no memory outside the arrays passed is
 * accessed even then. Errors: those of kap_selected_decode; a NULL schedule
 * where kap_decode_schedule_bytes is non-zero is KAP_ERR_INVALID_ARGUMENT.
 */
size_t kap_decode_schedule_bytes(const kap_kv_cache *kv, int32_t batch,
                                 int32_t max_view_blocks);

kap_status kap_decode_schedule(const kap_kv_cache *kv, int32_t batch, const int32_t *seq_lens,
                               const int32_t *view_block_table,
                               const int32_t *view_logical_block,
                               const uint32_t *view_token_mask, int32_t view_stride,
                               const int32_t *view_num_blocks, int32_t max_view_blocks,
                               int32_t *schedule, size_t schedule_bytes, void *stream);

kap_status kap_selected_decode_scheduled(const kap_kv_cache *kv, int32_t batch, const void *q,
                                         const int32_t *seq_lens,
                                         const int32_t *view_block_table,
                                         const int32_t *view_logical_block,
                                         const uint32_t *view_token_mask, int32_t view_stride,
                                         const int32_t *view_num_blocks, int32_t max_view_blocks,
                                         const int32_t *schedule, float sm_scale, float *out,
                                         float *lse, void *workspace, size_t workspace_bytes,
                                         void *stream);

/*
 * kap_verify -- full-context verification attention of the q_len = k+1
 * window (Sec. 3.2, "Full-context verification"; Eq. (2)).
 *
 * The window's own K/V are the last q_len tokens already in the cache, so
 * seq_lens[b] counts them. Window row i of sequence b sees logical positions
 * 0 .. seq_lens[b] - q_len + i, read through full_block_table[b].
 *   q [batch][q_len][Hq][D] (q_dtype); full_block_table [batch][fbt_stride];
 *   max_seq_len (host) >= every seq_lens[b] and <= 16 * fbt_stride;
 *   out [batch][q_len][Hq][D] float32; lse [batch][q_len][Hq] float32.
 * 1 <= q_len <= 16. num_splits as for kap_selected_decode.
 */
kap_status kap_verify(const kap_kv_cache *kv, int32_t batch, int32_t q_len, const void *q,
                      const int32_t *seq_lens, const int32_t *full_block_table,
                      int32_t fbt_stride, int32_t max_seq_len, float sm_scale,
                      int32_t num_splits, float *out, float *lse, void *workspace,
                      size_t workspace_bytes, void *stream);

size_t kap_verify_workspace_bytes(const kap_kv_cache *kv, int32_t batch, int32_t q_len,
                                  int32_t max_seq_len, int32_t num_splits);

/*
 * kap_append_kv -- place newly scheduled tokens' K/V into their physical KV
 * slots (the slot mapping of Sec. 3.1, "Selected-KV view materialization"):
 * how verification advances the full-context KV state KV^{full,+} of Sec. 3.2
 * ("Full-context verification").
 *
 * Token t goes to slot slot_mapping[t] = page * 16 + offset of the pool
 * described by kv, whose k_pages / v_pages this call WRITES (the const of the
 * struct fields notwithstanding). k_new / v_new [num_tokens][Hkv][D] hold the
 * values as the pool stores them (kv_dtype: f32, bf16 bits, or E4M3FN codes
 * already quantised with the destination page's scale -- kv_scales are not
 * changed); they are copied bit for bit into the page layout (K in 8-dim
 * chunks, V dim-major). A negative slot is padding and is skipped; a slot at
 * or beyond num_pages * 16 is skipped and counted into *bad_slots (device
 * int32, may be NULL; the caller zeroes it). Two tokens with the same slot:
 * either may win. num_tokens = 0 is a no-op.
 */
kap_status kap_append_kv(const kap_kv_cache *kv, int32_t num_tokens, const void *k_new,
                         const void *v_new, const int64_t *slot_mapping, int32_t *bad_slots,
                         void *stream);

/*
 * kap_compact_view -- materialise the selected-KV view as a compact physical
 * copy (Alg. 1, AssignCompactSlots and BuildBlockTable; Sec. 3.1: the
 * selected pages are compacted in access order into a reusable compact
 * workspace whose capacity is fixed).
 *
 * For sequence b and k < min(view_num_blocks[b], view_capacity), page
 * view_block_table[b][k] of src (K, V and, for fp8, its two scales) is copied
 * to page b * view_capacity + k of dst, and compact_block_table[b][k] is set
 * to that page; entries k >= the view length are set to -1. Invalid source
 * page ids copy nothing and map to -1. dst must have the same geometry and
 * dtypes as src and at least batch * view_capacity pages. Decoding over
 * (dst, compact_block_table, the same view_logical_block and view_num_blocks)
 * gives the result of decoding over (src, view_block_table).
 *   view_block_table [batch][view_stride], compact_block_table
 *   [batch][view_capacity] int32; view_capacity <= view_stride.
 */
kap_status kap_compact_view(const kap_kv_cache *src, int32_t batch,
                            const int32_t *view_block_table, int32_t view_stride,
                            const int32_t *view_num_blocks, int32_t view_capacity,
                            const kap_kv_cache *dst, int32_t *compact_block_table,
                            void *stream);

/*
 * kap_fallback_update -- one cycle of the executor's access-mode policy, on
 * the device, so that a whole proposal / verify stream can be captured in a
 * HIP graph (Sec. 3.2 "Runtime stability and fallback"; acceptance rate
 * h = accepted / speculated, Eq. (5); margin condition h > s, Eq. (12)).
 *
 * Per sequence b, with s_b = view_tokens[b] / seq_lens[b]:
 *   reset != 0: history and cycles[b] are cleared; mode[b] = 0 (selected view)
 *     if plan_status[b] == KAP_PLAN_OK, else 1 (full context); the active
 *     view row of b is written; accepted is not read (may be NULL).
 *   reset == 0: the cycle (accepted[b], gamma) enters the last-`window`
 *     history; cycles[b] += 1; a sequence in mode 0 with cycles[b] >= 2 whose
 *     window acceptance A / S (sums over the window) satisfies A / S <= s_b
 *     -- compared exactly as A * seq_lens[b] <= view_tokens[b] * S -- switches
 *     to mode 1 for good, and its active view row is rewritten.
 * Active view row: mode 0 copies the plan's row (sel_*); mode 1 is the full
 * context: view_block_table[b][j] = full_block_table[b][j],
 * view_logical_block[b][j] = j for j < ceil(seq_lens[b] / 16), and
 * view_num_blocks[b] = that count. Entries past the row's length are left as
 * they are.
 *   history [batch][window][2] int32 (accepted, speculated); cycles, mode
 *   [batch] int32 -- caller-owned device state kept across calls.
 *   view_stride >= max(sel_stride, full_stride); 1 <= window <= 64;
 *   0 <= gamma; accepted[b] is clamped to [0, gamma].
 */
kap_status kap_fallback_update(int32_t batch, int32_t reset, int32_t window, int32_t gamma,
                               const int32_t *accepted, const int32_t *view_tokens,
                               const int32_t *seq_lens, const int32_t *plan_status,
                               int32_t *history, int32_t *cycles, int32_t *mode,
                               const int32_t *sel_block_table, const int32_t *sel_logical_block,
                               const int32_t *sel_num_blocks, int32_t sel_stride,
                               const int32_t *full_block_table, int32_t full_stride,
                               int32_t *view_block_table, int32_t *view_logical_block,
                               int32_t *view_num_blocks, int32_t view_stride, void *stream);

/*
 * kap_fallback_update_masked -- kap_fallback_update for token-granular views
 * (kap_compile_plan_masked / kap_selected_decode_masked): whenever a
 * sequence's active view row is written, its token-mask row is written too --
 * view_token_mask[b][k] = sel_token_mask[b][k] in mode 0, 0xFFFF (every token
 * of the page) in mode 1. sel_token_mask is [batch][sel_stride] and
 * view_token_mask [batch][view_stride], uint32 (NULL only with a zero
 * stride). Every other argument and error is that of kap_fallback_update.
 */
kap_status kap_fallback_update_masked(
    int32_t batch, int32_t reset, int32_t window, int32_t gamma, const int32_t *accepted,
    const int32_t *view_tokens, const int32_t *seq_lens, const int32_t *plan_status,
    int32_t *history, int32_t *cycles, int32_t *mode, const int32_t *sel_block_table,
    const int32_t *sel_logical_block, const uint32_t *sel_token_mask,
    const int32_t *sel_num_blocks, int32_t sel_stride, const int32_t *full_block_table,
    int32_t full_stride, int32_t *view_block_table, int32_t *view_logical_block,
    uint32_t *view_token_mask, int32_t *view_num_blocks, int32_t view_stride, void *stream);

/*
 * kap_accept_top3 -- target-guided tolerant acceptance of a verify window
 * (Sec. 3.2 "Full-context verification": a proposed token is accepted when it
 * lies within the full-context verifier's top candidates -- top 3 in the
 * paper; top_k here).
 *
 * The window of sequence b holds the carry token and k = window - 1 proposed
 * tokens draft_tokens[b][0..k-1]; logits[b][i] are the verifier's logits at
 * window position i (predicting the token after it). Draft i is accepted
 * when its rank in logits[b][i] is below top_k, the rank of token d being
 * the number of tokens j with logit_j > logit_d, or logit_j == logit_d and
 * j < d (a draft outside [0, vocab) is never accepted). accepted[b] = m, the
 * number of leading accepted drafts (0..k); carry_token[b] = the argmax of
 * logits[b][m] (lowest index among equal maxima): the verifier-approved next
 * token. NaN logits give unspecified results.
 *   logits [batch][window][vocab] (logits_dtype F32 or BF16, 16-byte
 *   aligned); draft_tokens [batch][window-1] int32; accepted, carry_token
 *   [batch] int32. 1 <= window <= 17, 1 <= top_k, 1 <= vocab < 2^30.
 * Workspace (kap_accept_top3_workspace_bytes): per-row counters that must be
 * zero at call start and are left zero (allocate it zero-filled once).
 */
kap_status kap_accept_top3(int32_t batch, int32_t window, int32_t vocab, const void *logits,
                           kap_dtype logits_dtype, const int32_t *draft_tokens, int32_t top_k,
                           int32_t *accepted, int32_t *carry_token, void *workspace,
                           size_t workspace_bytes, void *stream);

size_t kap_accept_top3_workspace_bytes(int32_t batch, int32_t window);

/* Static description of a status code. */
const char *kap_status_string(kap_status status);
/* Message of the last failing call on this thread ("" if none). */
const char *kap_last_error(void);
/* KAP_ABI_VERSION of the loaded library. */
int32_t kap_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* KAP_H_ */

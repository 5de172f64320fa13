// Host side of the kap.h C ABI: argument validation, split planning,
// workspace sizing and kernel dispatch. Nothing here allocates, frees or
// synchronises; every launch goes to the caller's stream.
#include "kap.h"
#include "kap_diag.h"

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>

#include "kap_internal.h"

namespace {

thread_local std::string g_last_error;

kap_status fail(kap_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

kap_status ok() {
  g_last_error.clear();
  return KAP_OK;
}

bool aligned(const void *p, size_t n) { return (reinterpret_cast<uintptr_t>(p) % n) == 0; }

size_t round_up(size_t x, size_t m) { return (x + m - 1) / m * m; }

// Compute units of the current device (cached per device).
int device_cus() {
  static std::mutex mu;
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  std::lock_guard<std::mutex> lock(mu);
  if (cache[dev] == 0) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
      v = 256;
    cache[dev] = v;
  }
  return cache[dev];
}

// ---------------------------------------------------------------------------
// KV cache / geometry checks
// ---------------------------------------------------------------------------

kap_status check_kv(const kap_kv_cache *kv) {
  if (!kv) return fail(KAP_ERR_INVALID_ARGUMENT, "kv is NULL");
  if (kv->num_q_heads <= 0 || kv->num_kv_heads <= 0 || kv->num_q_heads % kv->num_kv_heads)
    return fail(KAP_ERR_INVALID_ARGUMENT, "num_q_heads (%d) must be a positive multiple of num_kv_heads (%d)",
                kv->num_q_heads, kv->num_kv_heads);
  if (kv->page_size != 16) return fail(KAP_ERR_UNSUPPORTED, "page_size %d unsupported (16 only)", kv->page_size);
  if (kv->head_dim != 64 && kv->head_dim != 128 && kv->head_dim != 256)
    return fail(KAP_ERR_UNSUPPORTED, "head_dim %d unsupported (64, 128, 256)", kv->head_dim);
  const bool f32 = kv->kv_dtype == KAP_DT_F32 && kv->q_dtype == KAP_DT_F32;
  const bool b16 = (kv->kv_dtype == KAP_DT_BF16 || kv->kv_dtype == KAP_DT_FP8_E4M3FN) &&
                   kv->q_dtype == KAP_DT_BF16;
  if (!f32 && !b16)
    return fail(KAP_ERR_UNSUPPORTED, "dtype pair kv=%d q=%d unsupported", kv->kv_dtype, kv->q_dtype);
  if (kv->num_pages < 0) return fail(KAP_ERR_INVALID_ARGUMENT, "num_pages < 0");
  if (kv->num_pages > 0 && (!kv->k_pages || !kv->v_pages))
    return fail(KAP_ERR_INVALID_ARGUMENT, "k_pages / v_pages is NULL");
  if (!aligned(kv->k_pages, 16) || !aligned(kv->v_pages, 16))
    return fail(KAP_ERR_INVALID_ARGUMENT, "k_pages / v_pages must be 16-byte aligned");
  if (kv->kv_dtype == KAP_DT_FP8_E4M3FN && kv->num_pages > 0 && !kv->kv_scales)
    return fail(KAP_ERR_INVALID_ARGUMENT, "FP8 KV needs kv_scales");
  return KAP_OK;
}

bool fast_geometry(const kap_kv_cache *kv) {
  return kv->q_dtype == KAP_DT_BF16 &&
         (kv->kv_dtype == KAP_DT_BF16 || kv->kv_dtype == KAP_DT_FP8_E4M3FN) &&
         kv->head_dim == 128 && kv->num_q_heads == 4 * kv->num_kv_heads;
}

struct SplitPlan {
  bool fast;
  bool ragged;    // tuned kernels: split counts balanced on the device
  int n_split;    // splits per (sequence, KV head); balanced mode: workgroups launched
  int pps;        // most pages any split of the generic path can get
  int w_target;   // balanced mode: workgroups the work is spread over
  int w_uneven;   // balanced mode, uneven batch: the same, finer chunks
  int min_chunk;  // balanced mode: fewest work items per split
  long long slots;  // tuned kernels: partial slots
};

// Balanced mode sizing: the work of a call is spread over about
// kTargetPerCU workgroups per CU (decode: per KV dtype), or over kUneven*
// finer ones when the batch is uneven, and a split keeps at least kMinChunk*
// work items (decode: view pages, one per wavefront and more; verify: page
// pairs). fp8 decode takes two workgroups per CU: its widening work per
// byte is twice bf16's, and a second workgroup on each CU hides it behind
// the other's loads (full-context decode of 4 x 128K tokens on MI355X: 167.8
// vs 170.0 us per call); for bf16 the second workgroup only adds requests in
// flight. Uneven batches: 8 workgroups per CU for decode (64 ragged fp8
// sequences of 4K-128K tokens: 772 vs 795 us with 4), 4 x the target for
// verify (8 was slower for 3-token windows).
constexpr int kDecodeTargetPerCU[2] = {1, 2};   // bf16, fp8 KV
constexpr int kDecodeUnevenPerCU = 8;
constexpr int kVerifyTargetPerCU = 1;
constexpr int kVerifyUnevenFactor = 4;
constexpr int kMinChunkDecode = 16;
constexpr int kMinChunkVerify = 8;

int cdiv(long long a, long long b) { return (int)((a + b - 1) / b); }

// Resident workgroups per CU of a tuned kernel (cached per device).
// id: 0/1 = decode bf16/fp8; 2 + 8*c4 + 4*fp8 + (nt-1) = verify (c4: q_len % 4 == 1).
int blocks_per_cu(int id, int kv_type, int q_len) {
  static std::mutex mu;
  static int cache[64][18] = {{0}};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  std::lock_guard<std::mutex> lock(mu);
  int &c = cache[dev][id];
  if (c == 0) {
    const int v = id < 2 ? kap::decode_fast_blocks_per_cu(kv_type)
                         : kap::verify_mfma_blocks_per_cu(kv_type, q_len);
    c = v > 0 ? v : -1;
  }
  return c > 0 ? c : 0;
}

// Generic path (one wavefront per query row and split): splits of at most
// kGenericPagesPerSplit pages -- the keys one work item stages in LDS -- and,
// when the call has few rows, more and smaller splits (down to
// kGenericMinPagesPerSplit pages) until about kGenericTargetWaves wavefronts
// run (the 4096-token fp32 workload: 32 rows x 2 splits of 36 pages took
// 152 us per decode call). num_splits > 0 asks for at least that many.
constexpr int kGenericTargetWaves = 4096;
constexpr int kGenericMinPagesPerSplit = 4;
int generic_splits(long long rows, int max_pages, int num_splits) {
  const int lo = cdiv(max_pages, kap::kGenericPagesPerSplit);
  const int hi = std::max(lo, cdiv(max_pages, kGenericMinPagesPerSplit));
  long long want = rows > 0 ? (kGenericTargetWaves + rows - 1) / rows : 1;
  if (num_splits > want) want = num_splits;
  int n = (int)std::min<long long>(std::max<long long>(want, lo), hi);
  if (num_splits > n) n = num_splits > max_pages ? max_pages : num_splits;
  return n;
}

// Decode. Tuned path: with num_splits > 0, that many splits for every
// (sequence, KV head); otherwise the balanced mode, where the kernel sizes
// each sequence's splits from its view (about kDecodeTargetPerCU
// workgroups per CU over the whole call) -- unless there are so many
// (sequence, KV head) units that one split each already fills the device.
// Generic path: see generic_splits.
SplitPlan plan_decode(const kap_kv_cache *kv, int batch, int max_blocks, int num_splits) {
  SplitPlan p{fast_geometry(kv), false, 1, 1, 0, 0, 0, 0};
  const int mb = max_blocks > 0 ? max_blocks : 1;
  const long long units = (long long)batch * kv->num_kv_heads;
  const int target = kDecodeTargetPerCU[kv->kv_dtype == KAP_DT_FP8_E4M3FN ? 1 : 0];
  if (p.fast) {
    if (num_splits > 0) {
      // uniform: the same split count for every (sequence, KV head)
      p.n_split = num_splits > mb ? mb : num_splits;
      p.slots = units * p.n_split;
    } else if (units >= 4LL * target * device_cus()) {
      p.n_split = 1;
      p.slots = units;
    } else {
      // balanced: split counts follow each sequence's actual view
      p.ragged = true;
      p.w_target = target * device_cus();
      p.w_uneven = kDecodeUnevenPerCU * device_cus();
      p.min_chunk = kMinChunkDecode;
      p.n_split = (int)((long long)std::max(p.w_target, p.w_uneven) + units);
      p.slots = p.n_split;
    }
    p.pps = cdiv(mb, p.n_split);
  } else {
    const int n = generic_splits((long long)batch * kv->num_q_heads, mb, num_splits);
    p.pps = cdiv(mb, n);
    p.n_split = cdiv(mb, p.pps);
  }
  return p;
}

// Verify (tuned path): as decode, with page pairs as the work items.
SplitPlan plan_verify(const kap_kv_cache *kv, int batch, int q_len, int max_pages, int num_splits) {
  SplitPlan p{fast_geometry(kv) && q_len * 4 <= 64, false, 1, 1, 0, 0, 0, 0};
  const int mp = max_pages > 0 ? max_pages : 1;
  const long long units = (long long)batch * kv->num_kv_heads;
  if (p.fast) {
    const int pairs = cdiv(mp, 2);
    if (num_splits > 0) {
      p.n_split = num_splits > pairs ? pairs : num_splits;
      p.slots = units * p.n_split;
    } else {
      const int fp8 = kv->kv_dtype == KAP_DT_FP8_E4M3FN;
      const int nt = (q_len * 4 + 15) / 16;
      int bpc = blocks_per_cu(2 + 8 * (q_len % 4 == 1) + 4 * fp8 + (nt - 1),
                              fp8 ? kap::kFP8 : kap::kBF16, q_len);
      if (bpc <= 0) bpc = 1;
      if (units >= 4LL * kVerifyTargetPerCU * bpc * device_cus()) {
        p.n_split = 1;
        p.slots = units;
        p.pps = 2 * pairs;
        return p;
      }
      p.ragged = true;
      p.w_target = kVerifyTargetPerCU * bpc * device_cus();
      p.w_uneven = kVerifyUnevenFactor * p.w_target;
      p.min_chunk = kMinChunkVerify;
      p.n_split = (int)((long long)p.w_uneven + units);
      p.slots = p.n_split;
    }
    p.pps = 2 * cdiv(pairs, p.n_split);
  } else {
    const int n = generic_splits((long long)batch * q_len * kv->num_q_heads, mp, num_splits);
    p.pps = cdiv(mp, n);
    p.n_split = cdiv(mp, p.pps);
  }
  return p;
}

// Workspace: [arrival counters, batch*Hkv int32][partial o][partial lse],
// each part 256-byte aligned. Generic path: nothing for a single split;
// partials [rows][n_split]. Tuned kernels: partials by slot, [slot][q_len*4],
// nothing when every (sequence, KV head) has a single uniform split.
struct WsLayout {
  size_t tickets, part_o, part_lse, total;
};

WsLayout ws_layout(const kap_kv_cache *kv, int batch, int q_len, const SplitPlan &p) {
  WsLayout w{0, 0, 0, 0};
  if (batch <= 0) return w;
  size_t prow;   // partial rows (one per split and output row)
  if (p.fast) {
    if (!p.ragged && p.n_split <= 1) return w;
    prow = (size_t)p.slots * q_len * 4;
  } else {
    if (p.n_split <= 1) return w;
    prow = (size_t)batch * q_len * kv->num_q_heads * p.n_split;
  }
  const size_t t = round_up(
      (size_t)batch * kv->num_kv_heads * sizeof(int32_t) * kap::kTicketStride, 256);
  const size_t o = round_up(prow * kv->head_dim * sizeof(float), 256);
  const size_t l = round_up(prow * sizeof(float), 256);
  w.tickets = 0;
  w.part_o = t;
  w.part_lse = t + o;
  w.total = t + o + l;
  return w;
}

size_t partial_bytes(const kap_kv_cache *kv, int batch, int q_len, const SplitPlan &p) {
  return ws_layout(kv, batch, q_len, p).total;
}

// Device scratch of kap_selected_decode_noalloc: one copy per GPU, zero when
// the library's code object is loaded there. Fixed layout: the arrival
// counters of the fused split merge in the first kScratchTicketBytes (the
// kernels leave every counter they use at zero), the split partials after
// them, so that no call's partials overlap another call's counters. In host
// code `scratch` only names the variable; its device address comes from
// scratch_base().
constexpr size_t kScratchBytes = size_t(16) << 20;
constexpr size_t kScratchTicketBytes = size_t(256) << 10;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// Device address of `scratch` on the current device, looked up once per
// device (with that device current); nullptr if the lookup fails.
void *scratch_base(hipError_t *err) {
  static std::mutex mu;
  static void *cache[64] = {nullptr};
  int dev = 0;
  *err = hipGetDevice(&dev);
  if (*err != hipSuccess) return nullptr;
  if (dev < 0 || dev >= 64) {
    *err = hipErrorInvalidDevice;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (!cache[dev]) {
    void *ptr = nullptr;
    *err = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (*err != hipSuccess) return nullptr;
    cache[dev] = ptr;
  }
  return cache[dev];
}

// The static scratch layout for a call whose workspace layout is w (its
// partial o and lse blocks, moved behind the fixed counter block).
WsLayout scratch_layout(const WsLayout &w) {
  WsLayout f{0, 0, 0, 0};
  if (w.total == 0) return f;
  f.part_o = kScratchTicketBytes;
  f.part_lse = f.part_o + (w.part_lse - w.part_o);
  f.total = f.part_lse + (w.total - w.part_lse);
  return f;
}

kap_status launch_attention(kap::AttnArgs &a, const kap_kv_cache *kv, const SplitPlan &p,
                            bool decode, void *ws, const WsLayout &w, hipStream_t s) {
  a.n_split = p.n_split;
  a.pages_per_split = p.pps;
  a.ragged = p.ragged ? 1 : 0;
  a.w_target = p.w_target;
  a.w_uneven = p.w_uneven;
  a.min_chunk = p.min_chunk;
  a.rcp_w_target = p.w_target > 0 ? 1.0 / p.w_target : 0.0;
  a.rcp_w_uneven = p.w_uneven > 0 ? 1.0 / p.w_uneven : 0.0;
  {
    const long long units = (long long)a.batch * a.Hkv;
    const long long ng = units > 0 ? p.w_target / units : 1;
    a.guess_splits = ng > 1 ? (int)ng : 1;
  }
  (void)kv;
  if (p.fast && w.total > 0x7fffffffULL)
    return fail(KAP_ERR_UNSUPPORTED, "split partials need %zu bytes (> 2 GiB); pass fewer splits",
                w.total);
  char *base = static_cast<char *>(ws);
  a.tickets = w.total ? reinterpret_cast<int32_t *>(base + w.tickets) : nullptr;
  a.part_o = w.total ? reinterpret_cast<float *>(base + w.part_o) : nullptr;
  a.part_lse = w.total ? reinterpret_cast<float *>(base + w.part_lse) : nullptr;
  (void)hipGetLastError();  // clear a stale error so a launch failure is ours
  hipError_t e;
  if (p.fast) {
    // the tuned kernels merge their splits themselves
    e = decode ? kap::launch_decode_fast(a, s) : kap::launch_verify_mfma(a, s);
  } else {
    e = kap::launch_attn_generic(a, s);
    if (e == hipSuccess && p.n_split > 1) e = kap::launch_merge(a, s);
  }
  if (e != hipSuccess) return fail(KAP_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

}  // namespace

extern "C" {

const char *kap_status_string(kap_status s) {
  switch (s) {
    case KAP_OK: return "KAP_OK";
    case KAP_ERR_INVALID_ARGUMENT: return "KAP_ERR_INVALID_ARGUMENT";
    case KAP_ERR_UNSUPPORTED: return "KAP_ERR_UNSUPPORTED";
    case KAP_ERR_WORKSPACE_TOO_SMALL: return "KAP_ERR_WORKSPACE_TOO_SMALL";
    case KAP_ERR_HIP: return "KAP_ERR_HIP";
    default: return "KAP_UNKNOWN_STATUS";
  }
}

const char *kap_last_error(void) { return g_last_error.c_str(); }

int32_t kap_abi_version(void) { return KAP_ABI_VERSION; }

// ---------------------------------------------------------------------------
// kap_compile_plan
// ---------------------------------------------------------------------------

size_t kap_compile_plan_workspace_bytes(int32_t batch, int32_t num_spans, int32_t fbt_stride) {
  (void)batch;
  (void)fbt_stride;
  return num_spans > 0 ? round_up((size_t)num_spans * sizeof(int32_t), 256) : 0;
}

static kap_status compile_plan(int32_t batch, const int32_t *seq_lens,
                               const int32_t *full_block_table, int32_t fbt_stride,
                               const int32_t *span_offsets, int32_t num_spans,
                               const int32_t *span_start, const int32_t *span_len,
                               const float *span_prior, const int32_t *prefix_tokens,
                               const int32_t *suffix_tokens, const int32_t *budget_tokens,
                               kap_select_policy policy, int64_t num_pages, int32_t view_capacity,
                               int32_t *view_block_table, int32_t *view_logical_block,
                               uint32_t *view_token_mask, bool token_mode,
                               int32_t *view_num_blocks, int32_t *view_tokens,
                               int32_t *spans_taken, int32_t *plan_status, int32_t *span_selected,
                               void *workspace, size_t workspace_bytes, void *stream) {
  if (batch < 0) return fail(KAP_ERR_INVALID_ARGUMENT, "batch < 0");
  if (num_spans < 0) return fail(KAP_ERR_INVALID_ARGUMENT, "num_spans < 0");
  if (view_capacity < 0) return fail(KAP_ERR_INVALID_ARGUMENT, "view_capacity < 0");
  if (num_pages < 0) return fail(KAP_ERR_INVALID_ARGUMENT, "num_pages < 0");
  if (policy != KAP_SELECT_SKIP && policy != KAP_SELECT_STOP)
    return fail(KAP_ERR_INVALID_ARGUMENT, "unknown selection policy %d", policy);
  if (fbt_stride < 1) return fail(KAP_ERR_INVALID_ARGUMENT, "fbt_stride < 1");
  const int max_pages = token_mode ? kap::kMaxTokenPlanPages : kap::kMaxPlanPages;
  if (fbt_stride > max_pages)
    return fail(KAP_ERR_UNSUPPORTED, "fbt_stride %d exceeds %d pages", fbt_stride, max_pages);
  if (batch == 0) return ok();
  if (!seq_lens || !full_block_table || !span_offsets || !prefix_tokens || !suffix_tokens ||
      !budget_tokens || !view_num_blocks || !view_tokens || !spans_taken || !plan_status)
    return fail(KAP_ERR_INVALID_ARGUMENT, "a required pointer is NULL");
  if (num_spans > 0 && (!span_start || !span_len || !span_prior))
    return fail(KAP_ERR_INVALID_ARGUMENT, "span arrays are NULL");
  if (view_capacity > 0 && (!view_block_table || !view_logical_block))
    return fail(KAP_ERR_INVALID_ARGUMENT, "view tables are NULL");
  if (token_mode && view_capacity > 0 && !view_token_mask)
    return fail(KAP_ERR_INVALID_ARGUMENT, "view_token_mask is NULL");
  const size_t need = kap_compile_plan_workspace_bytes(batch, num_spans, fbt_stride);
  if (need > 0 && (!workspace || workspace_bytes < need))
    return fail(KAP_ERR_WORKSPACE_TOO_SMALL, "workspace needs %zu bytes, got %zu", need, workspace_bytes);

  kap::PlanArgs a;
  a.batch = batch;
  a.seq_lens = seq_lens;
  a.fbt = full_block_table;
  a.fbt_stride = fbt_stride;
  a.span_offsets = span_offsets;
  a.num_spans = num_spans;
  a.span_start = span_start;
  a.span_len = span_len;
  a.span_prior = span_prior;
  a.prefix = prefix_tokens;
  a.suffix = suffix_tokens;
  a.budget = budget_tokens;
  a.policy = policy;
  a.num_pages = num_pages;
  a.capacity = view_capacity;
  a.view_bt = view_block_table;
  a.view_lblk = view_logical_block;
  a.view_nblk = view_num_blocks;
  a.view_tokens = view_tokens;
  a.spans_taken = spans_taken;
  a.status = plan_status;
  a.span_selected = span_selected;
  a.perm = static_cast<int32_t *>(workspace);
  a.token_mode = token_mode ? 1 : 0;
  a.view_mask = token_mode ? view_token_mask : nullptr;
  (void)hipGetLastError();
  const hipError_t e = kap::launch_compile_plan(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(KAP_ERR_HIP, "compile_plan launch failed: %s", hipGetErrorString(e));
  return ok();
}

kap_status kap_compile_plan(int32_t batch, const int32_t *seq_lens, const int32_t *full_block_table,
                            int32_t fbt_stride, const int32_t *span_offsets, int32_t num_spans,
                            const int32_t *span_start, const int32_t *span_len,
                            const float *span_prior, const int32_t *prefix_tokens,
                            const int32_t *suffix_tokens, const int32_t *budget_tokens,
                            kap_select_policy policy, int64_t num_pages, int32_t view_capacity,
                            int32_t *view_block_table, int32_t *view_logical_block,
                            int32_t *view_num_blocks, int32_t *view_tokens, int32_t *spans_taken,
                            int32_t *plan_status, int32_t *span_selected, void *workspace,
                            size_t workspace_bytes, void *stream) {
  return compile_plan(batch, seq_lens, full_block_table, fbt_stride, span_offsets, num_spans,
                      span_start, span_len, span_prior, prefix_tokens, suffix_tokens,
                      budget_tokens, policy, num_pages, view_capacity, view_block_table,
                      view_logical_block, nullptr, false, view_num_blocks, view_tokens,
                      spans_taken, plan_status, span_selected, workspace, workspace_bytes,
                      stream);
}

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
                                   size_t workspace_bytes, void *stream) {
  return compile_plan(batch, seq_lens, full_block_table, fbt_stride, span_offsets, num_spans,
                      span_start, span_len, span_prior, prefix_tokens, suffix_tokens,
                      budget_tokens, policy, num_pages, view_capacity, view_block_table,
                      view_logical_block, view_token_mask, true, view_num_blocks, view_tokens,
                      spans_taken, plan_status, span_selected, workspace, workspace_bytes,
                      stream);
}

// ---------------------------------------------------------------------------
// kap_selected_decode
// ---------------------------------------------------------------------------

size_t kap_selected_decode_workspace_bytes(const kap_kv_cache *kv, int32_t batch,
                                           int32_t max_view_blocks, int32_t num_splits) {
  if (check_kv(kv) != KAP_OK || batch <= 0 || max_view_blocks < 0) return 0;
  const SplitPlan p = plan_decode(kv, batch, max_view_blocks, num_splits);
  return partial_bytes(kv, batch, 1, p);
}

static kap_status selected_decode(const kap_kv_cache *kv, int32_t batch, const void *q,
                                  const int32_t *seq_lens, const int32_t *view_block_table,
                                  const int32_t *view_logical_block,
                                  const uint32_t *view_token_mask, bool masked,
                                  int32_t view_stride, const int32_t *view_num_blocks,
                                  int32_t max_view_blocks, float sm_scale, int32_t num_splits,
                                  float *out, float *lse, void *workspace,
                                  size_t workspace_bytes, void *stream, bool noalloc = false,
                                  const int32_t *schedule = nullptr, bool scheduled = false) {
  kap_status st = check_kv(kv);
  if (st != KAP_OK) return st;
  if (batch < 0) return fail(KAP_ERR_INVALID_ARGUMENT, "batch < 0");
  if (batch > 65535) return fail(KAP_ERR_UNSUPPORTED, "batch %d > 65535", batch);
  if (max_view_blocks < 0 || view_stride < max_view_blocks)
    return fail(KAP_ERR_INVALID_ARGUMENT, "need 0 <= max_view_blocks (%d) <= view_stride (%d)",
                max_view_blocks, view_stride);
  if (num_splits < 0) return fail(KAP_ERR_INVALID_ARGUMENT, "num_splits < 0");
  if (!(sm_scale == sm_scale) || sm_scale > 3.0e38f || sm_scale < -3.0e38f)
    return fail(KAP_ERR_INVALID_ARGUMENT, "sm_scale must be finite");
  if (kv->num_q_heads > 65535) return fail(KAP_ERR_UNSUPPORTED, "too many query heads");
  if (batch == 0) return ok();
  if (kv->num_pages < 1) return fail(KAP_ERR_INVALID_ARGUMENT, "KV pool has no pages");
  if (!q || !seq_lens || !view_num_blocks || !out || !lse)
    return fail(KAP_ERR_INVALID_ARGUMENT, "a required pointer is NULL");
  if (max_view_blocks > 0 && (!view_block_table || !view_logical_block))
    return fail(KAP_ERR_INVALID_ARGUMENT, "view tables are NULL");
  if (masked && max_view_blocks > 0 && !view_token_mask)
    return fail(KAP_ERR_INVALID_ARGUMENT, "view_token_mask is NULL");
  if (!aligned(q, 16) || !aligned(out, 16))
    return fail(KAP_ERR_INVALID_ARGUMENT, "q and out must be 16-byte aligned");
  const SplitPlan p = plan_decode(kv, batch, max_view_blocks, num_splits);
  if (scheduled && p.fast && p.ragged && !schedule)
    return fail(KAP_ERR_INVALID_ARGUMENT,
                "schedule is NULL (kap_decode_schedule_bytes is %zu for these arguments)",
                (size_t)p.n_split * kap::kSchedInts * sizeof(int32_t));
  WsLayout layout = ws_layout(kv, batch, 1, p);
  if (noalloc) {
    // the library's own scratch instead of a workspace
    layout = scratch_layout(layout);
    if (p.fast && layout.total > 0 &&
        (size_t)batch * kv->num_kv_heads * sizeof(int32_t) * kap::kTicketStride >
            kScratchTicketBytes)
      return fail(KAP_ERR_UNSUPPORTED,
                  "batch * num_kv_heads = %lld exceeds the %zu arrival counters of the "
                  "allocation-free call's scratch", (long long)batch * kv->num_kv_heads,
                  kScratchTicketBytes / (sizeof(int32_t) * kap::kTicketStride));
    if (layout.total > kScratchBytes)
      return fail(KAP_ERR_WORKSPACE_TOO_SMALL,
                  "the call's split partials need %zu bytes; the allocation-free call's scratch "
                  "holds %zu (use kap_selected_decode with a workspace)",
                  layout.total - kScratchTicketBytes, kScratchBytes - kScratchTicketBytes);
    hipError_t e = hipSuccess;
    workspace = scratch_base(&e);
    if (!workspace)
      return fail(KAP_ERR_HIP, "device address of the scratch buffer: %s", hipGetErrorString(e));
  } else {
    const size_t need = layout.total;
    if (need > 0 && (!workspace || workspace_bytes < need))
      return fail(KAP_ERR_WORKSPACE_TOO_SMALL, "workspace needs %zu bytes, got %zu", need,
                  workspace_bytes);
    if (need > 0 && !aligned(workspace, 256))
      return fail(KAP_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
  }

  kap::AttnArgs a;
  a.batch = batch;
  a.Hq = kv->num_q_heads;
  a.Hkv = kv->num_kv_heads;
  a.G = kv->num_q_heads / kv->num_kv_heads;
  a.D = kv->head_dim;
  a.kv_type = kv->kv_dtype;
  a.k_pages = kv->k_pages;
  a.v_pages = kv->v_pages;
  a.kv_scales = kv->kv_scales;
  a.num_pages = kv->num_pages;
  a.q = q;
  a.q_f32 = kv->q_dtype == KAP_DT_F32;
  a.q_len = 1;
  a.seq_lens = seq_lens;
  // An empty view may come with NULL tables: point them at seq_lens (row
  // stride 0) so kernels may read entry 0 of a row without a guard; no entry
  // is used, since every view is then empty.
  const bool no_table = max_view_blocks == 0;
  a.block_table = no_table ? seq_lens : view_block_table;
  a.bt_stride = no_table ? 0 : view_stride;
  a.logical_block = no_table ? seq_lens : view_logical_block;
  if (masked)
    a.token_mask = no_table ? reinterpret_cast<const uint32_t *>(seq_lens) : view_token_mask;
  a.num_blocks = view_num_blocks;
  a.max_blocks = max_view_blocks;
  a.causal = 0;
  a.scale_log2 = sm_scale * kap::kLog2e;
  a.out = out;
  a.lse = lse;
  a.schedule = scheduled && p.fast && p.ragged ? schedule : nullptr;
  return launch_attention(a, kv, p, true, workspace, layout, static_cast<hipStream_t>(stream));
}

kap_status kap_selected_decode(const kap_kv_cache *kv, int32_t batch, const void *q,
                               const int32_t *seq_lens, const int32_t *view_block_table,
                               const int32_t *view_logical_block, int32_t view_stride,
                               const int32_t *view_num_blocks, int32_t max_view_blocks,
                               float sm_scale, int32_t num_splits, float *out, float *lse,
                               void *workspace, size_t workspace_bytes, void *stream) {
  return selected_decode(kv, batch, q, seq_lens, view_block_table, view_logical_block, nullptr,
                         false, view_stride, view_num_blocks, max_view_blocks, sm_scale,
                         num_splits, out, lse, workspace, workspace_bytes, stream);
}

kap_status kap_selected_decode_masked(const kap_kv_cache *kv, int32_t batch, const void *q,
                                      const int32_t *seq_lens, const int32_t *view_block_table,
                                      const int32_t *view_logical_block,
                                      const uint32_t *view_token_mask, int32_t view_stride,
                                      const int32_t *view_num_blocks, int32_t max_view_blocks,
                                      float sm_scale, int32_t num_splits, float *out, float *lse,
                                      void *workspace, size_t workspace_bytes, void *stream) {
  return selected_decode(kv, batch, q, seq_lens, view_block_table, view_logical_block,
                         view_token_mask, true, view_stride, view_num_blocks, max_view_blocks,
                         sm_scale, num_splits, out, lse, workspace, workspace_bytes, stream);
}

size_t kap_decode_schedule_bytes(const kap_kv_cache *kv, int32_t batch,
                                 int32_t max_view_blocks) {
  if (check_kv(kv) != KAP_OK || batch <= 0 || max_view_blocks < 0) return 0;
  const SplitPlan p = plan_decode(kv, batch, max_view_blocks, 0);
  return p.fast && p.ragged ? (size_t)p.n_split * kap::kSchedInts * sizeof(int32_t) : 0;
}

kap_status kap_decode_schedule(const kap_kv_cache *kv, int32_t batch, const int32_t *seq_lens,
                               const int32_t *view_block_table,
                               const int32_t *view_logical_block,
                               const uint32_t *view_token_mask, int32_t view_stride,
                               const int32_t *view_num_blocks, int32_t max_view_blocks,
                               int32_t *schedule, size_t schedule_bytes, void *stream) {
  kap_status st = check_kv(kv);
  if (st != KAP_OK) return st;
  if (batch < 0) return fail(KAP_ERR_INVALID_ARGUMENT, "batch < 0");
  if (batch > 65535) return fail(KAP_ERR_UNSUPPORTED, "batch %d > 65535", batch);
  if (max_view_blocks < 0 || view_stride < max_view_blocks)
    return fail(KAP_ERR_INVALID_ARGUMENT, "need 0 <= max_view_blocks (%d) <= view_stride (%d)",
                max_view_blocks, view_stride);
  const size_t need = kap_decode_schedule_bytes(kv, batch, max_view_blocks);
  if (need == 0) return ok();   // no balanced split map for these arguments: nothing to record
  if (!seq_lens || !view_num_blocks)
    return fail(KAP_ERR_INVALID_ARGUMENT, "a required pointer is NULL");
  if (max_view_blocks > 0 && (!view_block_table || !view_logical_block))
    return fail(KAP_ERR_INVALID_ARGUMENT, "view tables are NULL");
  if (!schedule || schedule_bytes < need)
    return fail(KAP_ERR_WORKSPACE_TOO_SMALL, "schedule needs %zu bytes, got %zu", need,
                schedule_bytes);
  if (!aligned(schedule, 16)) return fail(KAP_ERR_INVALID_ARGUMENT, "schedule must be 16-byte aligned");
  const SplitPlan p = plan_decode(kv, batch, max_view_blocks, 0);
  kap::AttnArgs a;
  a.batch = batch;
  a.Hq = kv->num_q_heads;
  a.Hkv = kv->num_kv_heads;
  a.G = kv->num_q_heads / kv->num_kv_heads;
  a.D = kv->head_dim;
  a.kv_type = kv->kv_dtype;
  a.num_pages = kv->num_pages;
  a.q_len = 1;
  a.seq_lens = seq_lens;
  const bool no_table = max_view_blocks == 0;
  a.block_table = no_table ? seq_lens : view_block_table;
  a.bt_stride = no_table ? 0 : view_stride;
  a.logical_block = no_table ? seq_lens : view_logical_block;
  a.token_mask = view_token_mask && !no_table ? view_token_mask : nullptr;
  a.num_blocks = view_num_blocks;
  a.max_blocks = max_view_blocks;
  a.n_split = p.n_split;
  a.ragged = 1;
  a.w_target = p.w_target;
  a.w_uneven = p.w_uneven;
  a.min_chunk = p.min_chunk;
  a.rcp_w_target = p.w_target > 0 ? 1.0 / p.w_target : 0.0;
  a.rcp_w_uneven = p.w_uneven > 0 ? 1.0 / p.w_uneven : 0.0;
  a.schedule_out = schedule;
  (void)hipGetLastError();
  const hipError_t e = kap::launch_decode_schedule(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess)
    return fail(KAP_ERR_HIP, "decode_schedule launch failed: %s", hipGetErrorString(e));
  return ok();
}

kap_status kap_selected_decode_scheduled(const kap_kv_cache *kv, int32_t batch, const void *q,
                                         const int32_t *seq_lens,
                                         const int32_t *view_block_table,
                                         const int32_t *view_logical_block,
                                         const uint32_t *view_token_mask, int32_t view_stride,
                                         const int32_t *view_num_blocks, int32_t max_view_blocks,
                                         const int32_t *schedule, float sm_scale, float *out,
                                         float *lse, void *workspace, size_t workspace_bytes,
                                         void *stream) {
  return selected_decode(kv, batch, q, seq_lens, view_block_table, view_logical_block,
                         view_token_mask, view_token_mask != nullptr, view_stride,
                         view_num_blocks, max_view_blocks, sm_scale, 0, out, lse, workspace,
                         workspace_bytes, stream, false, schedule, true);
}

kap_status kap_selected_decode_noalloc(const kap_kv_cache *kv, int32_t batch, const void *q,
                                       const int32_t *seq_lens, const int32_t *view_block_table,
                                       const int32_t *view_logical_block, int32_t view_stride,
                                       const int32_t *view_num_blocks, int32_t max_view_blocks,
                                       float sm_scale, int32_t num_splits, float *out, float *lse,
                                       void *stream) {
  return selected_decode(kv, batch, q, seq_lens, view_block_table, view_logical_block, nullptr,
                         false, view_stride, view_num_blocks, max_view_blocks, sm_scale,
                         num_splits, out, lse, nullptr, 0, stream, true);
}

// ---------------------------------------------------------------------------
// kap_verify
// ---------------------------------------------------------------------------

size_t kap_verify_workspace_bytes(const kap_kv_cache *kv, int32_t batch, int32_t q_len,
                                  int32_t max_seq_len, int32_t num_splits) {
  if (check_kv(kv) != KAP_OK || batch <= 0 || q_len < 1 || q_len > 16 || max_seq_len < 0) return 0;
  const int max_pages = cdiv(max_seq_len, 16);
  const SplitPlan p = plan_verify(kv, batch, q_len, max_pages, num_splits);
  return partial_bytes(kv, batch, q_len, p);
}

kap_status kap_verify(const kap_kv_cache *kv, int32_t batch, int32_t q_len, const void *q,
                      const int32_t *seq_lens, const int32_t *full_block_table,
                      int32_t fbt_stride, int32_t max_seq_len, float sm_scale,
                      int32_t num_splits, float *out, float *lse, void *workspace,
                      size_t workspace_bytes, void *stream) {
  kap_status st = check_kv(kv);
  if (st != KAP_OK) return st;
  if (batch < 0) return fail(KAP_ERR_INVALID_ARGUMENT, "batch < 0");
  if (batch > 65535) return fail(KAP_ERR_UNSUPPORTED, "batch %d > 65535", batch);
  if (q_len < 1 || q_len > 16) return fail(KAP_ERR_INVALID_ARGUMENT, "q_len %d outside [1, 16]", q_len);
  if (max_seq_len < 0) return fail(KAP_ERR_INVALID_ARGUMENT, "max_seq_len < 0");
  const int max_pages = cdiv(max_seq_len, 16);
  if (fbt_stride < max_pages)
    return fail(KAP_ERR_INVALID_ARGUMENT, "fbt_stride %d < ceil(max_seq_len/16) = %d", fbt_stride, max_pages);
  if (num_splits < 0) return fail(KAP_ERR_INVALID_ARGUMENT, "num_splits < 0");
  if (!(sm_scale == sm_scale) || sm_scale > 3.0e38f || sm_scale < -3.0e38f)
    return fail(KAP_ERR_INVALID_ARGUMENT, "sm_scale must be finite");
  if ((long long)q_len * kv->num_q_heads > 65535) return fail(KAP_ERR_UNSUPPORTED, "too many rows");
  if (batch == 0) return ok();
  if (kv->num_pages < 1) return fail(KAP_ERR_INVALID_ARGUMENT, "KV pool has no pages");
  if (!q || !seq_lens || !out || !lse) return fail(KAP_ERR_INVALID_ARGUMENT, "a required pointer is NULL");
  if (max_pages > 0 && !full_block_table)
    return fail(KAP_ERR_INVALID_ARGUMENT, "full_block_table is NULL");
  if (!aligned(q, 16) || !aligned(out, 16))
    return fail(KAP_ERR_INVALID_ARGUMENT, "q and out must be 16-byte aligned");
  const SplitPlan p = plan_verify(kv, batch, q_len, max_pages, num_splits);
  const size_t need = partial_bytes(kv, batch, q_len, p);
  if (need > 0 && (!workspace || workspace_bytes < need))
    return fail(KAP_ERR_WORKSPACE_TOO_SMALL, "workspace needs %zu bytes, got %zu", need, workspace_bytes);
  if (need > 0 && !aligned(workspace, 256))
    return fail(KAP_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");

  kap::AttnArgs a;
  a.batch = batch;
  a.Hq = kv->num_q_heads;
  a.Hkv = kv->num_kv_heads;
  a.G = kv->num_q_heads / kv->num_kv_heads;
  a.D = kv->head_dim;
  a.kv_type = kv->kv_dtype;
  a.k_pages = kv->k_pages;
  a.v_pages = kv->v_pages;
  a.kv_scales = kv->kv_scales;
  a.num_pages = kv->num_pages;
  a.q = q;
  a.q_f32 = kv->q_dtype == KAP_DT_F32;
  a.q_len = q_len;
  a.seq_lens = seq_lens;
  a.block_table = full_block_table;
  a.bt_stride = fbt_stride;
  a.logical_block = nullptr;
  a.num_blocks = nullptr;
  a.max_blocks = max_pages;
  a.causal = 1;
  a.scale_log2 = sm_scale * kap::kLog2e;
  a.out = out;
  a.lse = lse;
  return launch_attention(a, kv, p, false, workspace, ws_layout(kv, batch, q_len, p),
                          static_cast<hipStream_t>(stream));
}

// ---------------------------------------------------------------------------
// kap_append_kv / kap_compact_view
// ---------------------------------------------------------------------------

static int elem_bytes(kap_dtype t) {
  return t == KAP_DT_F32 ? 4 : (t == KAP_DT_BF16 ? 2 : 1);
}

kap_status kap_append_kv(const kap_kv_cache *kv, int32_t num_tokens, const void *k_new,
                         const void *v_new, const int64_t *slot_mapping, int32_t *bad_slots,
                         void *stream) {
  kap_status st = check_kv(kv);
  if (st != KAP_OK) return st;
  if (num_tokens < 0) return fail(KAP_ERR_INVALID_ARGUMENT, "num_tokens < 0");
  if (num_tokens == 0) return ok();
  if (num_tokens > 0x7fffffff / 2) return fail(KAP_ERR_UNSUPPORTED, "too many tokens");
  if (!k_new || !v_new || !slot_mapping)
    return fail(KAP_ERR_INVALID_ARGUMENT, "k_new, v_new and slot_mapping are required");
  if (kv->num_pages < 1) return fail(KAP_ERR_INVALID_ARGUMENT, "KV pool has no pages");
  kap::AppendArgs a;
  a.num_tokens = num_tokens;
  a.Hkv = kv->num_kv_heads;
  a.D = kv->head_dim;
  a.elem_bytes = elem_bytes(kv->kv_dtype);
  if (!aligned(k_new, a.elem_bytes) || !aligned(v_new, a.elem_bytes) || !aligned(slot_mapping, 8))
    return fail(KAP_ERR_INVALID_ARGUMENT, "k_new / v_new / slot_mapping misaligned");
  a.k_new = k_new;
  a.v_new = v_new;
  a.slots = slot_mapping;
  a.k_pages = const_cast<void *>(kv->k_pages);
  a.v_pages = const_cast<void *>(kv->v_pages);
  a.num_pages = kv->num_pages;
  a.bad_slots = bad_slots;
  (void)hipGetLastError();
  const hipError_t e = kap::launch_append_kv(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(KAP_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

kap_status kap_compact_view(const kap_kv_cache *src, int32_t batch,
                            const int32_t *view_block_table, int32_t view_stride,
                            const int32_t *view_num_blocks, int32_t view_capacity,
                            const kap_kv_cache *dst, int32_t *compact_block_table,
                            void *stream) {
  kap_status st = check_kv(src);
  if (st != KAP_OK) return st;
  st = check_kv(dst);
  if (st != KAP_OK) return st;
  if (batch < 0) return fail(KAP_ERR_INVALID_ARGUMENT, "batch < 0");
  if (view_capacity < 0 || view_stride < view_capacity)
    return fail(KAP_ERR_INVALID_ARGUMENT, "need 0 <= view_capacity (%d) <= view_stride (%d)",
                view_capacity, view_stride);
  if (batch == 0 || view_capacity == 0) return ok();
  if (src->num_kv_heads != dst->num_kv_heads || src->num_q_heads != dst->num_q_heads ||
      src->head_dim != dst->head_dim || src->kv_dtype != dst->kv_dtype ||
      src->q_dtype != dst->q_dtype)
    return fail(KAP_ERR_INVALID_ARGUMENT, "src and dst caches differ in geometry or dtype");
  const long long need = (long long)batch * view_capacity;
  if (dst->num_pages < need)
    return fail(KAP_ERR_INVALID_ARGUMENT, "dst holds %lld pages, needs batch * view_capacity = %lld",
                (long long)dst->num_pages, need);
  if (need > 0x7fffffffLL) return fail(KAP_ERR_UNSUPPORTED, "compact workspace too large");
  if (!view_block_table || !view_num_blocks || !compact_block_table)
    return fail(KAP_ERR_INVALID_ARGUMENT, "a required pointer is NULL");
  if (!aligned(dst->k_pages, 16) || !aligned(dst->v_pages, 16))
    return fail(KAP_ERR_INVALID_ARGUMENT, "dst pages must be 16-byte aligned");
  kap::CompactArgs a;
  a.batch = batch;
  a.capacity = view_capacity;
  a.view_stride = view_stride;
  a.Hkv = src->num_kv_heads;
  a.D = src->head_dim;
  a.elem_bytes = elem_bytes(src->kv_dtype);
  a.view_bt = view_block_table;
  a.view_num_blocks = view_num_blocks;
  a.src_k = src->k_pages;
  a.src_v = src->v_pages;
  a.src_scales = src->kv_dtype == KAP_DT_FP8_E4M3FN ? src->kv_scales : nullptr;
  a.src_pages = src->num_pages;
  a.dst_k = const_cast<void *>(dst->k_pages);
  a.dst_v = const_cast<void *>(dst->v_pages);
  a.dst_scales = const_cast<float *>(dst->kv_scales);
  a.compact_bt = compact_block_table;
  // enough workgroups to stream at full bandwidth; each strides over entries
  const long long grid = need < 4LL * device_cus() ? need : 4LL * device_cus();
  (void)hipGetLastError();
  const hipError_t e = kap::launch_compact_view(a, (int)grid, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(KAP_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

static kap_status fallback_update(int32_t batch, int32_t reset, int32_t window, int32_t gamma,
                                  const int32_t *accepted, const int32_t *view_tokens,
                                  const int32_t *seq_lens, const int32_t *plan_status,
                                  int32_t *history, int32_t *cycles, int32_t *mode,
                                  const int32_t *sel_block_table,
                                  const int32_t *sel_logical_block,
                                  const uint32_t *sel_token_mask, const int32_t *sel_num_blocks,
                                  int32_t sel_stride, const int32_t *full_block_table,
                                  int32_t full_stride, int32_t *view_block_table,
                                  int32_t *view_logical_block, uint32_t *view_token_mask,
                                  bool masked, int32_t *view_num_blocks, int32_t view_stride,
                                  void *stream) {
  if (batch < 0) return fail(KAP_ERR_INVALID_ARGUMENT, "batch < 0");
  if (batch > 0x7fffffff / 2) return fail(KAP_ERR_UNSUPPORTED, "batch too large");
  if (window < 1 || window > 64) return fail(KAP_ERR_INVALID_ARGUMENT, "window %d outside [1, 64]", window);
  if (gamma < 0) return fail(KAP_ERR_INVALID_ARGUMENT, "gamma < 0");
  if (sel_stride < 0 || full_stride < 0 || view_stride < sel_stride || view_stride < full_stride)
    return fail(KAP_ERR_INVALID_ARGUMENT,
                "need view_stride (%d) >= sel_stride (%d) and full_stride (%d) >= 0", view_stride,
                sel_stride, full_stride);
  if (batch == 0) return ok();
  if ((!reset && !accepted) || !view_tokens || !seq_lens || !plan_status || !history || !cycles ||
      !mode || !sel_num_blocks || !view_num_blocks)
    return fail(KAP_ERR_INVALID_ARGUMENT, "a required pointer is NULL");
  if ((sel_stride > 0 && (!sel_block_table || !sel_logical_block)) ||
      (full_stride > 0 && !full_block_table) ||
      (view_stride > 0 && (!view_block_table || !view_logical_block)))
    return fail(KAP_ERR_INVALID_ARGUMENT, "a table is NULL");
  if (masked && ((sel_stride > 0 && !sel_token_mask) || (view_stride > 0 && !view_token_mask)))
    return fail(KAP_ERR_INVALID_ARGUMENT, "a token-mask table is NULL");
  kap::FallbackArgs a;
  a.batch = batch;
  a.reset = reset != 0;
  a.window = window;
  a.gamma = gamma;
  a.accepted = accepted;
  a.view_tokens = view_tokens;
  a.seq_lens = seq_lens;
  a.plan_status = plan_status;
  a.history = history;
  a.cycles = cycles;
  a.mode = mode;
  a.sel_bt = sel_block_table;
  a.sel_lb = sel_logical_block;
  a.sel_nb = sel_num_blocks;
  a.sel_stride = sel_stride;
  a.full_bt = full_block_table;
  a.full_stride = full_stride;
  a.view_bt = view_block_table;
  a.view_lb = view_logical_block;
  a.view_nb = view_num_blocks;
  a.view_stride = view_stride;
  if (masked && view_stride > 0) {
    a.sel_mask = sel_token_mask;
    a.view_mask = view_token_mask;
  }
  (void)hipGetLastError();
  const hipError_t e = kap::launch_fallback_update(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(KAP_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

kap_status kap_fallback_update(int32_t batch, int32_t reset, int32_t window, int32_t gamma,
                               const int32_t *accepted, const int32_t *view_tokens,
                               const int32_t *seq_lens, const int32_t *plan_status,
                               int32_t *history, int32_t *cycles, int32_t *mode,
                               const int32_t *sel_block_table, const int32_t *sel_logical_block,
                               const int32_t *sel_num_blocks, int32_t sel_stride,
                               const int32_t *full_block_table, int32_t full_stride,
                               int32_t *view_block_table, int32_t *view_logical_block,
                               int32_t *view_num_blocks, int32_t view_stride, void *stream) {
  return fallback_update(batch, reset, window, gamma, accepted, view_tokens, seq_lens,
                         plan_status, history, cycles, mode, sel_block_table, sel_logical_block,
                         nullptr, sel_num_blocks, sel_stride, full_block_table, full_stride,
                         view_block_table, view_logical_block, nullptr, false, view_num_blocks,
                         view_stride, stream);
}

kap_status kap_fallback_update_masked(
    int32_t batch, int32_t reset, int32_t window, int32_t gamma, const int32_t *accepted,
    const int32_t *view_tokens, const int32_t *seq_lens, const int32_t *plan_status,
    int32_t *history, int32_t *cycles, int32_t *mode, const int32_t *sel_block_table,
    const int32_t *sel_logical_block, const uint32_t *sel_token_mask,
    const int32_t *sel_num_blocks, int32_t sel_stride, const int32_t *full_block_table,
    int32_t full_stride, int32_t *view_block_table, int32_t *view_logical_block,
    uint32_t *view_token_mask, int32_t *view_num_blocks, int32_t view_stride, void *stream) {
  return fallback_update(batch, reset, window, gamma, accepted, view_tokens, seq_lens,
                         plan_status, history, cycles, mode, sel_block_table, sel_logical_block,
                         sel_token_mask, sel_num_blocks, sel_stride, full_block_table,
                         full_stride, view_block_table, view_logical_block, view_token_mask, true,
                         view_num_blocks, view_stride, stream);
}

// Workspace of kap_accept_top3: [row_best u64 x rows][row_count i32 x rows].
static size_t accept_ws(int batch, int window, size_t *count_off) {
  const size_t rows = (size_t)batch * window;
  const size_t best = round_up(rows * sizeof(unsigned long long), 256);
  if (count_off) *count_off = best;
  return best + round_up(rows * sizeof(int32_t), 256);
}

size_t kap_accept_top3_workspace_bytes(int32_t batch, int32_t window) {
  if (batch <= 0 || window < 1 || window > 17) return 0;
  return accept_ws(batch, window, nullptr);
}

kap_status kap_accept_top3(int32_t batch, int32_t window, int32_t vocab, const void *logits,
                           kap_dtype logits_dtype, const int32_t *draft_tokens, int32_t top_k,
                           int32_t *accepted, int32_t *carry_token, void *workspace,
                           size_t workspace_bytes, void *stream) {
  if (batch < 0) return fail(KAP_ERR_INVALID_ARGUMENT, "batch < 0");
  if (window < 1 || window > 17) return fail(KAP_ERR_INVALID_ARGUMENT, "window %d outside [1, 17]", window);
  if (vocab < 1 || vocab >= (1 << 30)) return fail(KAP_ERR_INVALID_ARGUMENT, "vocab %d outside [1, 2^30)", vocab);
  if (top_k < 1) return fail(KAP_ERR_INVALID_ARGUMENT, "top_k < 1");
  if (logits_dtype != KAP_DT_F32 && logits_dtype != KAP_DT_BF16)
    return fail(KAP_ERR_UNSUPPORTED, "logits must be F32 or BF16");
  if (batch == 0) return ok();
  if ((long long)batch * window > 65535)
    return fail(KAP_ERR_UNSUPPORTED, "batch * window > 65535");
  if (!logits || !accepted || !carry_token || (window > 1 && !draft_tokens))
    return fail(KAP_ERR_INVALID_ARGUMENT, "a required pointer is NULL");
  if (!aligned(logits, 16)) return fail(KAP_ERR_INVALID_ARGUMENT, "logits must be 16-byte aligned");
  size_t count_off = 0;
  const size_t need = accept_ws(batch, window, &count_off);
  if (!workspace || workspace_bytes < need)
    return fail(KAP_ERR_WORKSPACE_TOO_SMALL, "workspace needs %zu bytes, got %zu", need, workspace_bytes);
  if (!aligned(workspace, 256)) return fail(KAP_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
  kap::AcceptArgs a;
  a.batch = batch;
  a.window = window;
  a.vocab = vocab;
  a.top_k = top_k;
  a.f32 = logits_dtype == KAP_DT_F32;
  a.logits = logits;
  a.drafts = draft_tokens;
  a.accepted = accepted;
  a.carry = carry_token;
  a.row_best = static_cast<unsigned long long *>(workspace);
  a.row_count = reinterpret_cast<int32_t *>(static_cast<char *>(workspace) + count_off);
  (void)hipGetLastError();
  const hipError_t e = kap::launch_accept_top3(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(KAP_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

// ---------------------------------------------------------------------------
// kap_stream_read (measurement helper)
// ---------------------------------------------------------------------------

kap_status kap_stream_read(const void *src, size_t bytes, uint32_t *sink, void *stream) {
  if (bytes == 0) return ok();
  if (!src || !sink) return fail(KAP_ERR_INVALID_ARGUMENT, "a required pointer is NULL");
  if (!aligned(src, 16) || bytes % 16 != 0)
    return fail(KAP_ERR_INVALID_ARGUMENT, "src must be 16-byte aligned and bytes a multiple of 16");
  (void)hipGetLastError();
  const hipError_t e = kap::launch_stream_read(src, bytes, sink, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(KAP_ERR_HIP, "stream_read launch failed: %s", hipGetErrorString(e));
  return ok();
}

}  // extern "C"


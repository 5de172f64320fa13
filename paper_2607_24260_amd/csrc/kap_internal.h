// Internal declarations shared by the HIP sources of libkap (not installed).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace kap {

constexpr int kPage = 16;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kPlanThreads = 256;
constexpr int kGenericPagesPerSplit = 64;   // 1024 keys staged per generic work item
constexpr int kMaxPlanPages = 262144;       // pages per sequence the plan bitmap covers
constexpr int kMaxTokenPlanPages = 16384;   // the same with a bit per token (32 KB of LDS)
// Arrival counters of the fused split merge are kTicketStride int32 apart (a
// 64-byte block each): packed into one line, the device-coherent atomics of
// all (sequence, KV head) pairs met at a single memory channel (128K
// workload: 23.45 vs 23.62 us per decode call; 256-byte and 4-KB blocks
// measured the same as 64-byte ones).
constexpr int kTicketStride = 16;

enum KvType { kF32 = 0, kBF16 = 1, kFP8 = 2 };

// Arguments of kap_compile_plan after host validation.
struct PlanArgs {
  int batch;
  const int32_t *seq_lens;
  const int32_t *fbt;
  int fbt_stride;
  const int32_t *span_offsets;
  int num_spans;
  const int32_t *span_start;
  const int32_t *span_len;
  const float *span_prior;
  const int32_t *prefix;
  const int32_t *suffix;
  const int32_t *budget;
  int policy;
  int64_t num_pages;
  int capacity;
  int32_t *view_bt;
  int32_t *view_lblk;
  int32_t *view_nblk;
  int32_t *view_tokens;
  int32_t *spans_taken;
  int32_t *status;
  int32_t *span_selected;
  int32_t *perm;  // workspace: [num_spans] rank -> local span index
  int token_mode = 0;             // 1: a bit per token (the plan also writes view_mask)
  uint32_t *view_mask = nullptr;  // token mode: [batch][capacity] 16-bit token masks
};

// One attention call (decode or verify) after host validation.
// Rows per sequence: R = q_len * Hq; row r is window token r / Hq, head r % Hq.
struct AttnArgs {
  int batch, Hq, Hkv, G, D;
  int kv_type;
  const void *k_pages;
  const void *v_pages;
  const float *kv_scales;
  int64_t num_pages;
  const void *q;          // [batch][q_len][Hq][D], bf16 or f32
  int q_f32;              // 1 if q is float32
  int q_len;
  const int32_t *seq_lens;
  const int32_t *block_table;    // decode: view table; verify: full table
  int bt_stride;
  const int32_t *logical_block;  // decode: view logical pages; verify: NULL (identity)
  const int32_t *num_blocks;     // decode: view_num_blocks; verify: NULL (ceil(L/16))
  int max_blocks;                // host bound on pages read per sequence
  int causal;                    // verify: row i sees positions < L - q_len + i + 1
  float scale_log2;              // sm_scale * log2(e)
  int n_split;                   // splits per (sequence, KV head); balanced mode: workgroups
  int pages_per_split;
  // Tuned kernels, balanced mode (ragged != 0): split counts per sequence
  // come from its actual work on the device (see ragged_map); blockIdx.x is
  // the partial slot. Otherwise the grid is (n_split, Hkv, batch).
  int ragged;
  int w_target;                  // balanced mode: workgroups the work is spread over
  int w_uneven;                  // balanced mode, uneven batch: the same, finer
  int min_chunk;                 // balanced mode: fewest work items per split
  int guess_splits;              // balanced mode: max(1, w_target / (batch * Hkv))
  double rcp_w_target;           // balanced mode: 1 / w_target and 1 / w_uneven (host-rounded)
  double rcp_w_uneven;
  // Partials. Generic path: [batch * R][n_split][D] and [batch * R][n_split].
  // Tuned kernels: by slot, [slot][R_loc][D] and [slot][R_loc], R_loc =
  // q_len * 4 local rows; (sequence, KV head) owns slots slot0 .. slot0 + n - 1.
  float *part_o;    // normalised partial outputs
  float *part_lse;  // log2-domain partial LSE
  int32_t *tickets; // [batch][Hkv][kTicketStride] arrival counters of the fused merge
                    // (element 0 of each block; zero between calls)
  // decode over a token-granular view: [batch][bt_stride] masks, bit t = token
  // t of the view page is visible; NULL: every token below seq_len is
  const uint32_t *token_mask = nullptr;
  // decode, balanced mode with a precomputed schedule (kap_decode_schedule):
  // one kSchedInts record per workgroup; NULL: the kernel computes the map
  const int32_t *schedule = nullptr;
  int32_t *schedule_out = nullptr;   // kap_decode_schedule: the records written
  float *out;       // [batch * R][D]
  float *lse;       // [batch * R]
};

// Decode schedule record of workgroup w (int32 fields): the work item the
// balanced map gives w -- sequence, KV head, split, split count (0: no work),
// first slot -- the sequence's length and view blocks, and the first two view
// entries of each of the four wavefronts (page id, logical block, token mask)
// that start its page ring.
constexpr int kSchedInts = 32;
enum SchedField { kSchedB, kSchedG, kSchedSplit, kSchedNSplit, kSchedSlot0, kSchedL, kSchedNb,
                  kSchedEntries = 8 };   // + 3 * (2 * wave + ring slot) + {page, lblk, mask}

// kap_append_kv after host validation.
struct AppendArgs {
  int num_tokens, Hkv, D, elem_bytes;
  const void *k_new, *v_new;     // [num_tokens][Hkv][D]
  const int64_t *slots;          // [num_tokens]
  void *k_pages, *v_pages;       // the pool written into
  int64_t num_pages;
  int32_t *bad_slots;            // may be NULL
};

// kap_compact_view after host validation.
struct CompactArgs {
  int batch, capacity, view_stride, Hkv, D, elem_bytes;
  const int32_t *view_bt, *view_num_blocks;
  const void *src_k, *src_v;
  const float *src_scales;       // fp8 only, else NULL
  int64_t src_pages;
  void *dst_k, *dst_v;
  float *dst_scales;
  int32_t *compact_bt;           // [batch][capacity]
};

// kap_fallback_update after host validation.
struct FallbackArgs {
  int batch, reset, window, gamma;
  const int32_t *accepted, *view_tokens, *seq_lens, *plan_status;
  int32_t *history, *cycles, *mode;
  const int32_t *sel_bt, *sel_lb, *sel_nb;
  int sel_stride;
  const int32_t *full_bt;
  int full_stride;
  int32_t *view_bt, *view_lb, *view_nb;
  int view_stride;
  // token-granular views: the plan's and the active row's token masks, laid
  // out like the tables (NULL: page-granular)
  const uint32_t *sel_mask = nullptr;
  uint32_t *view_mask = nullptr;
};

// kap_accept_top3 after host validation.
constexpr int kAcceptChunk = 16384;  // vocabulary tokens per row workgroup
struct AcceptArgs {
  int batch, window, vocab, top_k, f32;
  const void *logits;            // [batch][window][vocab]
  const int32_t *drafts;         // [batch][window - 1]
  int32_t *accepted, *carry;     // [batch]
  int32_t *row_count;            // workspace [batch * window], zero between calls
  unsigned long long *row_best;  // workspace [batch * window], zero between calls
};

hipError_t launch_compile_plan(const PlanArgs &a, hipStream_t s);
hipError_t launch_accept_top3(const AcceptArgs &a, hipStream_t s);
hipError_t launch_fallback_update(const FallbackArgs &a, hipStream_t s);
hipError_t launch_append_kv(const AppendArgs &a, hipStream_t s);
hipError_t launch_compact_view(const CompactArgs &a, int grid, hipStream_t s);
hipError_t launch_attn_generic(const AttnArgs &a, hipStream_t s);
hipError_t launch_decode_fast(const AttnArgs &a, hipStream_t s);
hipError_t launch_decode_schedule(const AttnArgs &a, hipStream_t s);
hipError_t launch_verify_mfma(const AttnArgs &a, hipStream_t s);
hipError_t launch_merge(const AttnArgs &a, hipStream_t s);
hipError_t launch_stream_read(const void *src, size_t bytes, uint32_t *sink, hipStream_t s);

// Workgroups of the tuned kernels that fit on one compute unit at once
// (0 if the runtime cannot tell).
int decode_fast_blocks_per_cu(int kv_type);
int verify_mfma_blocks_per_cu(int kv_type, int q_len);

// ---------------------------------------------------------------------------
// device helpers
// ---------------------------------------------------------------------------

// Streaming load of KV data: every KV byte is read once per call, so the
// loads are nontemporal (they measurably raise achieved HBM read bandwidth).
template <typename T>
__device__ __forceinline__ T load_stream(const T *p) {
  return __builtin_nontemporal_load(p);
}

// Buffer descriptor of one (page, KV head) tile of `bytes` bytes at
// base + byte_off (wave-uniform). Loads through it take a per-lane byte
// offset, are bounds-checked by the hardware (reads past `bytes` return 0) and
// need no per-page vector address arithmetic.
typedef uint32_t kv_u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t kv_u32x2 __attribute__((ext_vector_type(2)));
constexpr int kBufDword3 = 0x00020000;   // raw 32-bit buffer, gfx9 family
constexpr int kNonTemporal = 2;          // cache-policy bit: no temporal reuse

__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const void *base, size_t byte_off,
                                                            int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(
      const_cast<char *>(static_cast<const char *>(base) + byte_off), 0, bytes, kBufDword3);
}
__device__ __forceinline__ kv_u32x4 tile_load16(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(kv_u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kNonTemporal));
}
__device__ __forceinline__ kv_u32x2 tile_load8(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(kv_u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kNonTemporal));
}
__device__ __forceinline__ uint32_t tile_load4(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kNonTemporal);
}

// Block-table entries read ahead through the vector memory pipe. A scalar
// load of the next entry, waited for right before the page load that needs
// it, stalls the wavefront for a full cache round trip on every page; a
// vector load travels in order with the KV loads, so it can be issued a ring
// round before its use and waited for with the page data. `opaque_zero` is a
// VGPR the compiler cannot see through (so the load stays a vector load);
// lane l reads element idx + (l & 1) of the table row, so lanes 0 and 1 hold
// two consecutive entries. Reads past the row's `bytes` return 0.
__device__ __forceinline__ int opaque_zero() {
  int z;
  asm volatile("v_mov_b32 %0, 0" : "=v"(z));
  return z;
}
__device__ __forceinline__ __amdgpu_buffer_rsrc_t table_rsrc(const int32_t *row, int entries) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t *>(row), 0, entries * 4, kBufDword3);
}
__device__ __forceinline__ int table_ahead(__amdgpu_buffer_rsrc_t r, int vzero_or_4, int idx) {
  return (int)__builtin_amdgcn_raw_buffer_load_b32(r, vzero_or_4, idx * 4, 0);
}
__device__ __forceinline__ int lane_value(int v, int lane) {
  return __builtin_amdgcn_readlane(v, lane);
}

// The (K, V) fp8 scales of a page, loaded with the page's KV data (in the
// same in-order vector-memory stream, so they arrive with it); a dead page
// reads nothing and gets (0, 0). Every KV head reads them, so they are
// cached normally.
__device__ __forceinline__ float2 page_scales(const float *kv_scales, int page, bool live) {
  const auto r = tile_rsrc(kv_scales, (size_t)page * 8, live ? 8 : 0);
  return __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(r, 0, 0, 0));
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Round-to-nearest-even float -> bfloat16 bits (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

// Two OCP E4M3FN codes (bytes 0,1 or 2,3 of w) -> two floats, exact.
template <bool HIGH>
__device__ __forceinline__ float2 fp8x2_to_f32(uint32_t w) {
  auto v = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(w), HIGH);
  return make_float2(v[0], v[1]);
}

// Four E4M3FN codes (one dword) -> two dwords of bf16 pairs, exact (every
// E4M3FN value, subnormals included, is a bf16 value); unit scale.
typedef __bf16 kv_bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ kv_u32x2 fp8x4_to_bf16x4(uint32_t w) {
  const kv_bf16x2 lo = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, false);
  const kv_bf16x2 hi = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, true);
  return kv_u32x2{__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi)};
}

// 2^x on the hardware unit, without the range reduction that keeps
// denormal results: results below 2^-126 may come out as 0. Used for softmax
// weights, whose sum is at least 1.
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// max(x, y) as the hardware maximum: unlike fmaxf it does not quiet signalling
// NaNs first (one instruction per operand whose origin the compiler cannot
// vouch for), and a NaN operand gives NaN -- which the softmax turns into NaN
// outputs either way. Equal for all other inputs (+0 above -0).
__device__ __forceinline__ float max_f(float x, float y) {
  return __builtin_elementwise_maximum(x, y);
}

// One E4M3FN code -> float (generic path).
__device__ __forceinline__ float fp8_to_f32(uint8_t b) {
  return __builtin_amdgcn_cvt_f32_fp8(static_cast<int>(b), 0);
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}
__device__ __forceinline__ int wave_sum_i(int x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// ---------------------------------------------------------------------------
// balanced work map of the tuned kernels
// ---------------------------------------------------------------------------

// One (sequence b, KV head g, split) work unit; the splits of (b, g) own
// partial slots slot0 .. slot0 + n_split - 1.
struct WorkItem {
  int b, g, split, n_split, slot0;
};

// Wavefront-wide inclusive prefix sum / running maximum through DPP row
// shifts and row broadcasts (no LDS round trips); lane 63 holds the total.
template <int CTRL, int ROWS>
__device__ __forceinline__ int dpp_or_zero(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, ROWS, 0xF, false);
}
__device__ __forceinline__ int wave_scan_add(int x) {
  x += dpp_or_zero<0x111, 0xF>(x);   // row_shr:1
  x += dpp_or_zero<0x112, 0xF>(x);   // row_shr:2
  x += dpp_or_zero<0x114, 0xF>(x);   // row_shr:4
  x += dpp_or_zero<0x118, 0xF>(x);   // row_shr:8
  x += dpp_or_zero<0x142, 0xA>(x);   // row_bcast:15 into rows 1, 3
  x += dpp_or_zero<0x143, 0xC>(x);   // row_bcast:31 into rows 2, 3
  return x;
}
__device__ __forceinline__ int wave_scan_max(int x) {   // x >= 0
  x = max(x, dpp_or_zero<0x111, 0xF>(x));
  x = max(x, dpp_or_zero<0x112, 0xF>(x));
  x = max(x, dpp_or_zero<0x114, 0xF>(x));
  x = max(x, dpp_or_zero<0x118, 0xF>(x));
  x = max(x, dpp_or_zero<0x142, 0xA>(x));
  x = max(x, dpp_or_zero<0x143, 0xC>(x));
  return x;
}
__device__ __forceinline__ int lane63(int x) { return __builtin_amdgcn_readlane(x, 63); }

// floor(n / d) for 0 <= n < 2^31 and d >= 1. The quotient of two doubles is
// correctly rounded, and for n < 2^53 rounding never reaches the next
// integer, so truncating it is exact (shorter than the integer division
// sequence).
__device__ __forceinline__ int div_small(int n, int d) {
  return (int)((double)n / (double)d);
}

// floor(n / d) for 0 <= n < 2^21 and d >= 1 through the hardware reciprocal:
// the float estimate n * rcp(d) is off by less than n/d * 2^-22 < 1/2, so
// its truncation is within one of the quotient, and one correction step each
// way makes it exact. (A handful of single-precision instructions where a
// double division is a dependent chain of about ten.)
__device__ __forceinline__ int div_u21(int n, int d) {
  int q = (int)((float)n * __builtin_amdgcn_rcpf((float)d));
  const int r = n - q * d;
  q += (r >= d) ? 1 : 0;
  q -= (r < 0) ? 1 : 0;
  return q;
}

// floor(n / d) for 0 <= n < 2^52 and d >= 1, given rcp = 1/d rounded to a
// double: n * rcp is within n * 2^-52 * (1/d) of n/d, less than the distance
// 1/d from a non-integer quotient to the next integer, so truncation is exact
// except below an integer quotient, which the correction step catches.
__device__ __forceinline__ long long div_rcp(long long n, long long d, double rcp) {
  long long q = (long long)((double)n * rcp);
  const long long r = n - q * d;
  q += (r >= d) ? 1 : 0;
  q -= (r < 0) ? 1 : 0;
  return q;
}

// Balanced mode: sequence b holds load(b).items work items per KV head (decode:
// view pages; verify: page pairs), counted up to 2^24 for sizing. With
// T = Hkv * sum_b items_b, the chunk is C = max(min_chunk, T / w_target)
// items when the sequences are even (the largest holds at most 5/4 of the
// mean: one split per workgroup slot is then balanced), else T / w_uneven --
// finer chunks, which the hardware dispatcher spreads over the CUs as they
// free up. Every (b, g) gets n_b = max(1, round(items_b / C)) splits when
// the batch is even -- for equal views exactly w_target / (batch * Hkv), one
// workgroup per slot -- and max(1, ceil(items_b / C)) when it is uneven, so
// that no split holds more than C items (rounding to nearest there left
// splits of up to 1.5 C, and the call waited for them at its end). Slots are
// numbered sequence-major, then KV head, then split. Workgroup w takes slot w
// and returns false past the last slot. The result is the same in every
// wavefront, which computes it alone (two passes over the batch, 64
// sequences per pass). Since C >= T / W, the slots number at most
// W + batch * Hkv, W = max(w_target, w_uneven): the grid the host launches.
constexpr int kMapItemCap = 1 << 24;

// What the map reads per sequence: its work items and one more value the
// caller wants for the sequence it is given (returned through aux_b).
struct SeqLoad {
  int items, aux;
};

// The loads of sequences 0..63 (one per lane), issued early by the caller so
// that their wait does not cover loads issued after them.
template <class Load>
__device__ __forceinline__ SeqLoad map_first_loads(const AttnArgs &a, Load load) {
  const int lane = threadIdx.x & 63;
  SeqLoad first = load(min(lane, a.batch - 1));   // branch-free; batch >= 1
  if (lane >= a.batch) first.items = 0;
  return first;
}

template <class Load>
__device__ __forceinline__ bool ragged_map(const AttnArgs &a, Load load, const SeqLoad &first,
                                           int w, WorkItem &wi, int &items_b, int &aux_b) {
  const int lane = threadIdx.x & 63;
  int v0 = min(first.items, kMapItemCap);
  long long tot = lane63(wave_scan_add(v0));
  int mx = lane63(wave_scan_max(v0));
  for (int b0 = 64; b0 < a.batch; b0 += 64) {
    const int v = b0 + lane < a.batch ? min(load(b0 + lane).items, kMapItemCap) : 0;
    tot += lane63(wave_scan_add(v));
    mx = max(mx, lane63(wave_scan_max(v)));
  }
  const long long T = tot * a.Hkv;
  const bool even = 4LL * mx * a.batch <= 5 * tot;
  const int W = even ? a.w_target : a.w_uneven;
  // C = ceil(T / W), exactly (T < 2^52: at most 2^24 items per sequence)
  long long C = div_rcp(T + W - 1, W, even ? a.rcp_w_target : a.rcp_w_uneven);
  if (C < a.min_chunk) C = a.min_chunk;
  const int Ci = (int)(C < kMapItemCap ? C : kMapItemCap);
  const double rcp_c = 1.0 / (double)Ci;   // the one device division of the map
  int base = 0;
  for (int b0 = 0; b0 < a.batch; b0 += 64) {
    const int b = b0 + lane;
    const bool in = b < a.batch;
    SeqLoad m = first;
    if (b0 > 0) m = in ? load(b) : SeqLoad{0, 0};
    const int v = min(m.items, kMapItemCap);
    const int nb =
        in ? max(1, (int)div_rcp(v + (even ? Ci / 2 : Ci - 1), Ci, rcp_c)) : 0;
    const int cnt = nb * a.Hkv;
    const int incl = wave_scan_add(cnt);
    const int excl = incl - cnt;
    const unsigned long long hit = __ballot(in && w >= base + excl && w < base + incl);
    if (hit) {
      const int l = __builtin_amdgcn_readfirstlane(__ffsll((long long)hit) - 1);
      const int e = base + __builtin_amdgcn_readlane(excl, l);
      wi.n_split = __builtin_amdgcn_readlane(nb, l);
      wi.b = b0 + l;
      const int off = w - e;
      wi.g = div_u21(off, wi.n_split);   // off < slots <= W + batch * Hkv < 2^21
      wi.split = off - wi.g * wi.n_split;
      wi.slot0 = w - wi.split;
      items_b = __builtin_amdgcn_readlane(m.items, l);
      aux_b = __builtin_amdgcn_readlane(m.aux, l);
      return true;
    }
    base += lane63(incl);
  }
  return false;
}

// ---------------------------------------------------------------------------
// fused split merge for the tuned kernels (four query heads per KV head)
// ---------------------------------------------------------------------------

// Row index (in out / lse) of local row r = 4 * window_token + head_in_group.
__device__ __forceinline__ size_t out_row(const AttnArgs &a, int b, int g, int r) {
  return ((size_t)b * a.q_len + (r >> 2)) * a.Hq + g * 4 + (r & 3);
}

// Partial results travel between workgroups with stores and loads that carry
// the agent-scope coherence bit (sc1): the bit the AMDGPU memory model uses
// for agent-scope atomic stores and loads. Such stores are written through to
// the device-coherent level and such loads bypass non-coherent cached copies,
// so no L2 write-back or invalidate (whose cost grows with the number of
// workgroups) is needed; a vmcnt(0) wait orders the partial stores before the
// arrival ticket.
constexpr int kCoherent = 16;   // sc1

__device__ __forceinline__ __amdgpu_buffer_rsrc_t partial_rsrc(const float *base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(base), 0, 0x7fffffff, kBufDword3);
}
__device__ __forceinline__ void partial_store4(__amdgpu_buffer_rsrc_t r, size_t byte_off,
                                               float4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(kv_u32x4, v), r, (int)byte_off, 0,
                                         kCoherent);
}
__device__ __forceinline__ void partial_store1(__amdgpu_buffer_rsrc_t r, size_t byte_off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, (int)byte_off, 0, kCoherent);
}
__device__ __forceinline__ float4 partial_load4(__amdgpu_buffer_rsrc_t r, size_t byte_off) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)byte_off, 0,
                                                                          kCoherent));
}
__device__ __forceinline__ float partial_load1(__amdgpu_buffer_rsrc_t r, size_t byte_off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)byte_off, 0, kCoherent));
}

// True in every thread of the workgroup that completes the last of the
// n_split partials of (b, g). Only wavefront 0 may have written this
// workgroup's partial (with partial_store*): it waits until those stores are
// complete, then takes a ticket. The last workgroup resets the counter.
__device__ __forceinline__ bool last_arrival(const AttnArgs &a, int b, int g, int n_split,
                                             int *flag) {
  if (threadIdx.x < 64) {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): this wave's stores are complete
    asm volatile("" ::: "memory");
    if (threadIdx.x == 0) {
      int32_t *ctr = a.tickets + ((size_t)b * a.Hkv + g) * kTicketStride;
      const int prev = __hip_atomic_fetch_add(ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const int last = (prev == n_split - 1) ? 1 : 0;
      if (last) __hip_atomic_store(ctr, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      *flag = last;
    }
  }
  __syncthreads();
  return *flag != 0;
}

// last_arrival for a workgroup whose wavefronts may all have written part of
// its partial: each waits until its own stores are complete, the workgroup
// meets at a barrier, and one thread takes the ticket.
__device__ __forceinline__ bool last_arrival_all(const AttnArgs &a, int b, int g, int n_split,
                                                 int *flag) {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): this wave's stores are complete
  asm volatile("" ::: "memory");
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t *ctr = a.tickets + ((size_t)b * a.Hkv + g) * kTicketStride;
    const int prev = __hip_atomic_fetch_add(ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int last = (prev == n_split - 1) ? 1 : 0;
    if (last) __hip_atomic_store(ctr, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *flag = last;
  }
  __syncthreads();
  return *flag != 0;
}

// LSE merge of the ns partials (slots slot0 .. slot0 + ns - 1) of the R_loc
// local rows of (b, g), D = 128:
// lse = log2 sum_s 2^lse_s, o = sum_s 2^(lse_s - lse) o_s (empty splits drop out).
// Every thread takes up to kMergeItems (row, 4-dim) items at once -- one for
// decode's 4 rows (128 items), 3 for verify's up to 64 (one pass over 640
// items at 20 rows instead of three) -- and reads their partials eight splits
// at a time with independent loads (one memory round trip per eight splits
// for all its items), folding them in with a running maximum.
template <int kMergeItems>
__device__ __forceinline__ void merge_rows(const AttnArgs &a, int b, int g, int R_loc, int slot0,
                                           int ns) {
  constexpr int kBatch = 8;
  const auto ro = partial_rsrc(a.part_o);
  const auto rl = partial_rsrc(a.part_lse);
  const int n_items = R_loc * 32;
  for (int e0 = threadIdx.x; e0 < n_items; e0 += kMergeItems * blockDim.x) {
    bool ok[kMergeItems];
    int r[kMergeItems], d4[kMergeItems];
    float M[kMergeItems], tot[kMergeItems];
    float4 o[kMergeItems];
#pragma unroll
    for (int it = 0; it < kMergeItems; ++it) {
      const int e = e0 + it * blockDim.x;
      ok[it] = e < n_items;
      r[it] = ok[it] ? e >> 5 : 0;
      d4[it] = (e & 31) * 4;
      M[it] = -INFINITY;
      tot[it] = 0.f;
      o[it] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
    for (int s0 = 0; s0 < ns; s0 += kBatch) {
      float ls[kMergeItems][kBatch];
      float4 vs[kMergeItems][kBatch];
#pragma unroll
      for (int it = 0; it < kMergeItems; ++it) {
        if (!ok[it]) continue;
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
          const size_t pr = (size_t)(slot0 + min(s0 + j, ns - 1)) * R_loc + r[it];
          ls[it][j] = partial_load1(rl, pr * 4);
          vs[it][j] = partial_load4(ro, (pr * 128 + d4[it]) * 4);
        }
      }
#pragma unroll
      for (int it = 0; it < kMergeItems; ++it) {
        if (!ok[it]) continue;
        float mc = M[it];
#pragma unroll
        for (int j = 0; j < kBatch; ++j)
          if (s0 + j < ns) mc = fmaxf(mc, ls[it][j]);
        if (mc == -INFINITY) continue;               // every split so far is empty
        const float sc = exp2f(M[it] - mc);          // 0 while M is still -inf
        tot[it] *= sc;
        o[it].x *= sc; o[it].y *= sc; o[it].z *= sc; o[it].w *= sc;
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
          if (s0 + j >= ns) continue;
          const float w = exp2f(ls[it][j] - mc);
          tot[it] += w;
          o[it].x = fmaf(w, vs[it][j].x, o[it].x);
          o[it].y = fmaf(w, vs[it][j].y, o[it].y);
          o[it].z = fmaf(w, vs[it][j].z, o[it].z);
          o[it].w = fmaf(w, vs[it][j].w, o[it].w);
        }
        M[it] = mc;
      }
    }
#pragma unroll
    for (int it = 0; it < kMergeItems; ++it) {
      if (!ok[it]) continue;
      const size_t row = out_row(a, b, g, r[it]);
      float lse = -INFINITY;
      float4 v = o[it];
      if (M[it] != -INFINITY) {
        const float inv = 1.f / tot[it];
        v.x *= inv; v.y *= inv; v.z *= inv; v.w *= inv;
        lse = (M[it] + log2f(tot[it])) * kLn2;
      }
      *reinterpret_cast<float4 *>(a.out + row * 128 + d4[it]) = v;
      if (d4[it] == 0) a.lse[row] = lse;
    }
  }
}

}  // namespace kap

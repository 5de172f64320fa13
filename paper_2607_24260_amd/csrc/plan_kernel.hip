// kap_compile_plan on the GPU: Alg. 1 of the paper, SelectEvidenceUnderBudget
// through BuildBlockTable, one workgroup per sequence.
//
// Per sequence the workgroup
//   1. checks the CSR bounds, the length and the scores (status codes),
//   2. marks the mandatory prefix / suffix in an LDS bitmap,
//   3. ranks the spans by (prior desc, start asc, index asc) -- for every
//      span, 1 to 8 threads (as many as the span count leaves) count how many
//      spans precede it, and the inverse permutation goes to LDS (to the
//      workspace when the spans exceed one LDS chunk),
//   4. walks the spans in rank order with one wavefront, 64 at a time: each
//      lane prices its span against the bitmap (its cost in visible tokens),
//      a ballot finds the first span that fits, and only a taken span changes
//      the state -- one round per taken span, not per span,
//   5. compacts the bitmap into the ascending logical-page list (staged in
//      LDS) and maps it through the full block table.
// Page mode keeps one bit per page; token mode (the visibility mask of
// Sec. 3.1 at token resolution) one bit per token, and also emits each view
// page's 16-bit mask of visible tokens.
// Selection uses integer arithmetic only (float priors are only compared), so
// the plan is bit-for-bit deterministic.
#include "kap_internal.h"

namespace kap {
namespace {

constexpr int kRankChunk = 2048;   // ranking keys staged per pass; also the LDS view list

// The ranking order without the index, as one unsigned integer: the prior,
// descending (-0 ranks as +0; NaN never gets here), above the start,
// ascending. Span j ranks before span i iff key_j < key_i, or the keys are
// equal and j < i. No span's key is ~0 (the padding key).
__device__ __forceinline__ uint64_t rank_key(float prior, int start) {
  uint32_t u = __float_as_uint(prior == 0.f ? 0.f : prior);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);   // monotone in the float's value
  return ((uint64_t)~u << 32) | (uint32_t)(start ^ 0x80000000);
}
constexpr uint64_t kPadKey = ~0ull;

// Exclusive prefix sum of v over the workgroup (kPlanThreads threads, in
// thread order); *total receives the sum. s_tmp holds kPlanThreads/64 ints.
__device__ __forceinline__ int block_exclusive_scan(int v, int *s_tmp, int *total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int x = wave_scan_add(v);                      // inclusive, within the wavefront
  if (lane == 63) s_tmp[w] = x;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int i = 0; i < kPlanThreads / 64; ++i) {
    before += (i < w) ? s_tmp[i] : 0;
    all += s_tmp[i];
  }
  __syncthreads();
  *total = all;
  return before + x - v;
}

// Bits of bitmap word w (bits 32w .. 32w + 31) that lie in [x, e).
__device__ __forceinline__ uint32_t range_bits(int w, int x, int e) {
  const int lo = min(max(x - 32 * w, 0), 32);
  const int hi = min(max(e - 32 * w, 0), 32);
  return (uint32_t)(((1ull << hi) - 1ull) ^ ((1ull << lo) - 1ull));
}

// Spare words past the last bitmap word: count_clear reads up to 7 of them.
constexpr int kBitmapPadWords = 8;

// Number of clear bits of the bitmap in [x, e), x < e.
// Page bitmap: a span covers one to three words, counted one at a time.
// Token bitmap: a span covers tens of words. The count is the length of the
// range less its set bits, which are summed over the whole words w0 .. w1 (a
// popcount with accumulate per word) and corrected by the set bits of the two
// end words that lie outside [x, e). The words are read eight at a time before
// they are counted, so that their LDS latencies overlap; a batch may read up
// to seven words past w1 (into the spare words at the end) and counts nothing
// there.
template <bool TOK>
__device__ __forceinline__ int count_clear(const uint32_t* bitmap, int x, int e) {
  if constexpr (!TOK) {
    int c = 0;
    for (int w = x >> 5; w <= (e - 1) >> 5; ++w) c += __popc(range_bits(w, x, e) & ~bitmap[w]);
    return c;
  } else {
    constexpr int kW = 8;
    static_assert(kW <= kBitmapPadWords, "batch reads past the spare words");
    const int w0 = x >> 5, w1 = (e - 1) >> 5;
    const uint32_t below = (1u << (x & 31)) - 1u;            // bits of w0 before x
    const uint32_t above = ~((2u << ((e - 1) & 31)) - 1u);   // bits of w1 from e on
    int set = -(int)(__popc(bitmap[w0] & below) + __popc(bitmap[w1] & above));
    for (int w = w0; w <= w1; w += kW) {
      uint32_t v[kW];
#pragma unroll
      for (int k = 0; k < kW; ++k) v[k] = bitmap[w + k];
      const int last = w1 - w;
#pragma unroll
      for (int k = 0; k < kW; ++k) set += __popc(k <= last ? v[k] : 0u);
    }
    return (e - x) - set;
  }
}

template <bool TOK>
__global__ __launch_bounds__(kPlanThreads) void compile_plan_kernel(PlanArgs a) {
  extern __shared__ uint32_t bitmap[];   // page mode: bit per page; token mode: bit per token
  __shared__ int s_flag;
  __shared__ int s_scan[kPlanThreads / 64];
  __shared__ long long s_used;
  __shared__ int s_taken;
  // ranking keys; after the ranking (one chunk) each span's (length, start);
  // at the end the view list (and its token masks)
  __shared__ __align__(16) union {
    uint64_t key[kRankChunk];
    struct {
      int page[kRankChunk];
      uint32_t mask[kRankChunk];
    } view;
  } s_u;
  uint64_t *const s_key = s_u.key;
  __shared__ int s_perm[kRankChunk];   // one chunk: rank -> local span index

  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;

  const int lo = a.span_offsets[b];
  const int hi = a.span_offsets[b + 1];

  auto write_fail = [&](int status, bool zero_flags) {
    if (zero_flags && a.span_selected) {
      for (int i = lo + tid; i < hi; i += kPlanThreads) a.span_selected[i] = 0;
    }
    if (tid == 0) {
      a.view_nblk[b] = 0;
      a.view_tokens[b] = 0;
      a.spans_taken[b] = 0;
      a.status[b] = status;
    }
  };

  if (lo < 0 || hi < lo || hi > a.num_spans) {
    write_fail(5 /*KAP_PLAN_BAD_SPANS*/, false);
    return;
  }
  const int L = a.seq_lens[b];
  const int NP = (L >= 1) ? (int)(((long long)L + kPage - 1) / kPage) : 0;
  if (L < 1 || NP > a.fbt_stride) {
    write_fail(4 /*KAP_PLAN_BAD_LENGTH*/, true);
    return;
  }

  // -- scores, and the first chunk of ranking keys -----------------------------
  // Keys are staged in LDS padded to a multiple of four with the padding key,
  // which no span's key equals or exceeds.
  const int n = hi - lo;
  const bool one_chunk = n <= kRankChunk;
  if (tid == 0) s_flag = 0;
  __syncthreads();
  {
    const int jn4 = (min(n, kRankChunk) + 3) & ~3;
    const int lim = max(n, jn4);
    for (int t = tid; t < lim; t += kPlanThreads) {
      if (t < n) {
        const float pr = a.span_prior[lo + t];
        if (__builtin_isnan(pr)) s_flag = 1;
        if (t < kRankChunk) s_key[t] = rank_key(pr, a.span_start[lo + t]);
      } else {
        s_key[t] = kPadKey;
      }
    }
  }
  __syncthreads();
  if (s_flag) {
    write_fail(2 /*KAP_PLAN_BAD_SCORE*/, true);
    return;
  }
  // one chunk: the span lengths the greedy walk needs, loaded now and stored
  // to LDS (beside the starts) once the ranking is done
  constexpr int kLenRegs = kRankChunk / kPlanThreads;
  int len_r[kLenRegs];
#pragma unroll
  for (int q = 0; q < kLenRegs; ++q) {
    const int t = tid + q * kPlanThreads;
    len_r[q] = (one_chunk && t < n) ? a.span_len[lo + t] : 0;
  }

  // -- mandatory prefix / suffix ----------------------------------------------
  const int pre = min(max(a.prefix[b], 0), L);
  const int suf_start = max(0, L - max(a.suffix[b], 1));
  const int W = TOK ? (L + 31) / 32 : (NP + 31) / 32;  // bitmap words
  if constexpr (TOK) {
    // tokens [0, pre) and [suf_start, L); no bit at or past L is ever set
    for (int w = tid; w < W; w += kPlanThreads)
      bitmap[w] = range_bits(w, 0, pre) | range_bits(w, suf_start, L);
  } else {
    for (int w = tid; w < W; w += kPlanThreads) bitmap[w] = 0u;
    __syncthreads();
    const int pre_pages = (pre + kPage - 1) / kPage;     // pages [0, pre_pages)
    const int suf_page0 = suf_start / kPage;             // pages [suf_page0, NP)
    for (int p = tid; p < pre_pages; p += kPlanThreads) atomicOr(&bitmap[p >> 5], 1u << (p & 31));
    for (int p = suf_page0 + tid; p < NP; p += kPlanThreads)
      atomicOr(&bitmap[p >> 5], 1u << (p & 31));
  }

  // -- rank the spans ---------------------------------------------------------
  // rank(i) = number of spans ordered before span i = #{j : key_j < key_i}
  // + #{j < i : key_j = key_i}. Keys are read from LDS in chunks of
  // kRankChunk (a single chunk, staged above, in the common case), four per
  // two broadcast reads. One pass counts the keys below and equal to key_i;
  // only when some span shares its key with another (equal prior and start)
  // does a second pass count the equal keys of lower index. With few spans,
  // TS = 2, 4 or 8 neighbouring threads share span i, thread s counting over
  // keys 4 s, 4 s + 4 TS, ..., and their counts are summed with lane swaps.
  const int TS = n <= kPlanThreads / 8 ? 8 : n <= kPlanThreads / 4 ? 4 : n <= kPlanThreads / 2 ? 2 : 1;
  const int sub = tid & (TS - 1);
  typedef uint64_t u64x2 __attribute__((ext_vector_type(2)));
  // counts over all chunks: below (ties == false) or equal with lower index
  // (ties == true); every thread takes part (chunk staging has barriers)
  auto count = [&](bool act, int i, uint64_t ki, bool ties, int &c_lt, int &c_eq) {
    for (int jb = 0; jb < n; jb += kRankChunk) {
      const int jn = min(kRankChunk, n - jb);
      const int jn4 = (jn + 3) & ~3;
      if (!one_chunk) {
        __syncthreads();
        for (int t = tid; t < jn4; t += kPlanThreads)
          s_key[t] = t < jn ? rank_key(a.span_prior[lo + jb + t], a.span_start[lo + jb + t]) : kPadKey;
        __syncthreads();
      }
      if (act) {
#pragma unroll 2
        for (int t = 4 * sub; t < jn4; t += 4 * TS) {
          const u64x2 k01 = *reinterpret_cast<const u64x2 *>(&s_key[t]);
          const u64x2 k23 = *reinterpret_cast<const u64x2 *>(&s_key[t + 2]);
          if (!ties) {
            c_lt += (k01.x < ki) + (k01.y < ki) + (k23.x < ki) + (k23.y < ki);
            c_eq += (k01.x == ki) + (k01.y == ki) + (k23.x == ki) + (k23.y == ki);
          } else {
            const int j = jb + t;
            c_eq += ((k01.x == ki) & (j < i)) + ((k01.y == ki) & (j + 1 < i)) +
                    ((k23.x == ki) & (j + 2 < i)) + ((k23.y == ki) & (j + 3 < i));
          }
        }
      }
    }
    // the TS threads of span i are lanes l .. l + TS - 1 of one wavefront
    for (int m = 1; m < TS; m <<= 1) {
      c_lt += __shfl_xor(c_lt, m);
      c_eq += __shfl_xor(c_eq, m);
    }
  };
  for (int ib = 0; ib < n; ib += kPlanThreads / TS) {
    const int i = ib + tid / TS;
    const bool act = i < n;
    uint64_t ki = kPadKey;
    if (act) ki = one_chunk ? s_key[i] : rank_key(a.span_prior[lo + i], a.span_start[lo + i]);
    int below = 0, equal = 0;
    count(act, i, ki, false, below, equal);   // equal counts span i itself
    int rank = below;
    if (__syncthreads_or(act && equal > 1)) {
      int unused = 0, tied = 0;
      count(act, i, ki, true, unused, tied);
      rank += tied;
    }
    if (act && sub == 0) {
      if (one_chunk) s_perm[rank] = i;
      else a.perm[lo + rank] = i;
      if (a.span_selected) a.span_selected[lo + i] = 0;
    }
  }
  __syncthreads();
  if (one_chunk) {
    // (length, start) of every span for the greedy walk, over its key
#pragma unroll
    for (int q = 0; q < kLenRegs; ++q) {
      const int t = tid + q * kPlanThreads;
      if (t < n) s_key[t] = ((uint64_t)(uint32_t)len_r[q] << 32) | (uint32_t)(s_key[t] & 0xffffffffu);
    }
  }
  __syncthreads();

  // -- visible tokens of the mandatory part -----------------------------------
  {
    int c = 0;
    for (int w = tid; w < W; w += kPlanThreads) c += __popc(bitmap[w]);
    int total = 0;
    block_exclusive_scan(c, s_scan, &total);
    if (tid == 0) {
      if constexpr (TOK) {
        s_used = total;
      } else {
        // the last page is always selected (suffix >= 1 token)
        const int last_valid = L - kPage * (NP - 1);    // 1..16
        s_used = (long long)kPage * total - (kPage - last_valid);
      }
      s_taken = 0;
    }
  }
  __syncthreads();

  // -- greedy selection in rank order (one wavefront) -------------------------
  // The spans are walked 64 ranks at a time, lane l holding the span of rank
  // r0 + l as a bit range [u0, u1) of the bitmap (pages; tokens in token mode)
  // and its count of bits not yet set. The state changes only when a span is
  // taken, so every span between two taken ones is decided against the same
  // state: a ballot finds the first span (in rank order) that fits, the ones
  // before it are rejected (SKIP) or, if one of them fails, selection ends
  // (STOP). When span j is taken, each later lane whose range meets j's
  // subtracts the bits j newly covers (read before j's bits are set), so a
  // batch costs one round per taken span instead of one per span. Page mode:
  // every page but the last (always selected) holds 16 tokens, so a span costs
  // 16 per new page. The budget state is wavefront-uniform.
  if (tid < 64) {
    int used = __builtin_amdgcn_readfirstlane((int)s_used);
    int taken = 0;
    const int T = a.budget[b];
    bool stop = false;
    for (int r0 = 0; r0 < n && !stop; r0 += 64) {
      int my_i = -1, x = 0, e = 0;
      if (r0 + lane < n) {
        // (two separate paths: merged into one load from a selected address,
        // the LDS and the global read would both become generic loads)
        int li;
        if (one_chunk) {
          li = s_perm[r0 + lane];
        } else {
          li = a.perm[lo + r0 + lane];
          asm volatile("" ::: "memory");
        }
        my_i = lo + li;
        int st32, len32;
        if (one_chunk) {
          const uint64_t v = s_key[li];
          st32 = (int)((uint32_t)v ^ 0x80000000u);
          len32 = (int)(uint32_t)(v >> 32);
        } else {
          st32 = a.span_start[my_i];
          len32 = a.span_len[my_i];
        }
        const long long st = st32;
        const long long x64 = st > 0 ? st : 0;
        long long e64 = st + (long long)len32;
        if (e64 > L) e64 = L;
        x = (int)x64;
        e = (int)(e64 > x64 ? e64 : x64);               // e <= x: empty after clipping
      }
      const bool valid = e > x;                         // empty spans are ignored
      const int u0 = TOK ? x : x / kPage;
      const int u1 = TOK ? e : (e + kPage - 1) / kPage;
      int fresh = valid ? count_clear<TOK>(bitmap, u0, u1) : 0;
      bool my_taken = false;
      int pos = 0;                                      // lanes below pos are decided
      while (true) {
        const int cost = TOK ? fresh : kPage * fresh;
        const bool open = valid && lane >= pos;
        const bool fits = used + cost <= T;
        const unsigned long long mf = __ballot(open && fits);
        const unsigned long long mx = __ballot(open && !fits);
        const int j = mf ? __builtin_ctzll(mf) : 64;
        const int jx = mx ? __builtin_ctzll(mx) : 64;
        if (a.policy == 1 /*KAP_SELECT_STOP*/ && jx < j) {
          stop = true;
          break;
        }
        if (j == 64) break;
        // take span j
        const int ju0 = __builtin_amdgcn_readlane(u0, j);
        const int ju1 = __builtin_amdgcn_readlane(u1, j);
        used += __builtin_amdgcn_readlane(cost, j);
        ++taken;
        my_taken |= lane == j;
        pos = j + 1;
        const int c0 = max(u0, ju0), c1 = min(u1, ju1);
        if (valid && lane > j && c0 < c1) fresh -= count_clear<TOK>(bitmap, c0, c1);
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        const int jw0 = ju0 >> 5, jw1 = (ju1 - 1) >> 5;
        for (int wb = jw0; wb <= jw1; wb += 64) {
          const int w = wb + lane;
          const bool in = w <= jw1;
          atomicOr(&bitmap[in ? w : jw1], in ? range_bits(w, ju0, ju1) : 0u);
        }
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      }
      if (a.span_selected && my_taken) a.span_selected[my_i] = 1;
    }
    if (lane == 0) {
      s_used = used;
      s_taken = taken;
    }
  }
  __syncthreads();

  // -- compaction: ascending logical pages -> block table ---------------------
  // Token mode: page p is the half p & 1 of token word p >> 1 and is in the
  // view when any of its 16 bits is set; that half is its token mask.
  const int chunk = (W + kPlanThreads - 1) / kPlanThreads;
  const int w0 = min(W, tid * chunk);
  const int w1 = min(W, w0 + chunk);
  int mine = 0;
  for (int w = w0; w < w1; ++w) {
    const uint32_t x = bitmap[w];
    mine += TOK ? ((x & 0xFFFFu) != 0u) + ((x >> 16) != 0u) : __popc(x);
  }
  if (tid == 0) s_flag = 0;
  int nblk = 0;
  const int first = block_exclusive_scan(mine, s_scan, &nblk);
  if (nblk > a.capacity) {
    write_fail(1 /*KAP_PLAN_OVER_CAPACITY*/, true);
    return;
  }
  int out = first;
  const int32_t *fbt_row = a.fbt + (size_t)b * a.fbt_stride;
  int32_t *vbt = a.view_bt + (size_t)b * a.capacity;
  int32_t *vlb = a.view_lblk + (size_t)b * a.capacity;
  uint32_t *vmk = TOK ? a.view_mask + (size_t)b * a.capacity : nullptr;
  bool bad = false;
  // Views of up to kRankChunk pages: the logical pages (and masks) go to LDS
  // at their output index first, then every thread maps entries k, k + 256,
  // ... through the full block table, so the table reads are all in flight
  // at once. Longer views map each page where it is found.
  const bool staged = nblk <= kRankChunk;
  auto emit = [&](int p, uint32_t mask) {
    if (staged) {
      s_u.view.page[out] = p;
      if constexpr (TOK) s_u.view.mask[out] = mask;
    } else {
      const int page = fbt_row[p];
      bad |= (page < 0) || ((int64_t)page >= a.num_pages);
      vlb[out] = p;
      vbt[out] = page;
      if constexpr (TOK) vmk[out] = mask;
    }
    ++out;
  };
  for (int w = w0; w < w1; ++w) {
    const uint32_t x = bitmap[w];
    if constexpr (TOK) {
      if (x & 0xFFFFu) emit(2 * w, x & 0xFFFFu);
      if (x >> 16) emit(2 * w + 1, x >> 16);
    } else {
      uint32_t bits = x;
      while (bits) {
        const int bit = __ffs(bits) - 1;
        bits &= bits - 1u;
        emit(w * 32 + bit, 0u);
      }
    }
  }
  if (staged) {
    __syncthreads();
    for (int k = tid; k < nblk; k += kPlanThreads) {
      const int p = s_u.view.page[k];
      const int page = fbt_row[p];
      bad |= (page < 0) || ((int64_t)page >= a.num_pages);
      vlb[k] = p;
      vbt[k] = page;
      if constexpr (TOK) vmk[k] = s_u.view.mask[k];
    }
  }
  if (bad) s_flag = 1;
  __syncthreads();
  if (s_flag) {
    write_fail(3 /*KAP_PLAN_BAD_PAGE*/, true);
    return;
  }
  if (tid == 0) {
    a.view_nblk[b] = nblk;
    a.view_tokens[b] = (int)s_used;
    a.spans_taken[b] = s_taken;
    a.status[b] = 0;
  }
}

size_t plan_lds_bytes(int fbt_stride, bool token_mode) {
  // page mode: a bit per page; token mode: a bit per token (16 per page)
  const size_t words = token_mode ? ((size_t)fbt_stride * kPage + 31) / 32
                                  : ((size_t)fbt_stride + 31) / 32;
  return (words + kBitmapPadWords) * sizeof(uint32_t);
}

}  // namespace

hipError_t launch_compile_plan(const PlanArgs &a, hipStream_t s) {
  const bool tok = a.token_mode != 0;
  const size_t lds = plan_lds_bytes(a.fbt_stride, tok);
  if (tok)
    hipLaunchKernelGGL(compile_plan_kernel<true>, dim3(a.batch), dim3(kPlanThreads), lds, s, a);
  else
    hipLaunchKernelGGL(compile_plan_kernel<false>, dim3(a.batch), dim3(kPlanThreads), lds, s, a);
  return hipGetLastError();
}

}  // namespace kap

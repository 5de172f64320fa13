// kap_compile_plan on the GPU: Alg. 1 of the paper, SelectEvidenceUnderBudget
// through BuildBlockTable, one workgroup per sequence.
//
// Per sequence the workgroup
//   1. checks the CSR bounds, the length and the scores (status codes),
//   2. marks the mandatory prefix / suffix in an LDS bitmap,
//   3. ranks the spans by (prior desc, start asc, index asc) -- every thread
//      counts, for its spans, how many spans precede them, and writes the
//      inverse permutation to the workspace,
//   4. walks the spans in rank order with one wavefront: the 64 lanes test the
//      span against the bitmap, a wavefront reduction counts what is new (its
//      cost in visible tokens), and the span is taken when it fits the budget,
//   5. compacts the bitmap into the ascending logical-page list and maps it
//      through the full block table.
// Page mode keeps one bit per page; token mode (the visibility mask of
// Sec. 3.1 at token resolution) one bit per token, and also emits each view
// page's 16-bit mask of visible tokens.
// Selection uses integer arithmetic only (float priors are only compared), so
// the plan is bit-for-bit deterministic.
#include "kap_internal.h"

namespace kap {
namespace {

constexpr int kRankChunk = 1024;

__device__ __forceinline__ bool ranks_before(float pj, int sj, int j, float pi, int si, int i) {
  if (pj > pi) return true;
  if (pj < pi) return false;           // equal values (including -0 == +0) fall through
  if (sj != si) return sj < si;
  return j < i;
}

// Exclusive prefix sum of v over the workgroup (kPlanThreads threads, in
// thread order); *total receives the sum. s_tmp holds kPlanThreads/64 ints.
__device__ __forceinline__ int block_exclusive_scan(int v, int *s_tmp, int *total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
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

// Bits of token word w (tokens 32w .. 32w + 31) that lie in [x, e).
__device__ __forceinline__ uint32_t range_bits(int w, int x, int e) {
  const int lo = min(max(x - 32 * w, 0), 32);
  const int hi = min(max(e - 32 * w, 0), 32);
  return (uint32_t)(((1ull << hi) - 1ull) ^ ((1ull << lo) - 1ull));
}

// Sum over the wavefront of a per-lane count in [0, 63]: one ballot per bit.
__device__ __forceinline__ int wave_count_sum(int c) {
  int s = 0;
#pragma unroll
  for (int k = 0; k < 6; ++k) s += __popcll(__ballot((c >> k) & 1)) << k;
  return s;
}

template <bool TOK>
__global__ __launch_bounds__(kPlanThreads) void compile_plan_kernel(PlanArgs a) {
  extern __shared__ uint32_t bitmap[];   // page mode: bit per page; token mode: bit per token
  __shared__ int s_flag;
  __shared__ int s_scan[kPlanThreads / 64];
  __shared__ long long s_used;
  __shared__ int s_taken;
  __shared__ float s_prior[kRankChunk];
  __shared__ int s_start[kRankChunk];

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

  // -- scores ---------------------------------------------------------------
  if (tid == 0) s_flag = 0;
  __syncthreads();
  for (int i = lo + tid; i < hi; i += kPlanThreads)
    if (__builtin_isnan(a.span_prior[i])) s_flag = 1;
  __syncthreads();
  if (s_flag) {
    write_fail(2 /*KAP_PLAN_BAD_SCORE*/, true);
    return;
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
  // rank(i) = number of spans ordered before span i; keys are staged through
  // LDS in chunks of kRankChunk so the all-pairs count reads LDS broadcasts.
  const int n = hi - lo;
  for (int ib = 0; ib < n; ib += kPlanThreads) {
    const int i = ib + tid;
    const bool act = i < n;
    const float pi = act ? a.span_prior[lo + i] : 0.f;
    const int si = act ? a.span_start[lo + i] : 0;
    int rank = 0;
    for (int jb = 0; jb < n; jb += kRankChunk) {
      __syncthreads();
      const int jn = min(kRankChunk, n - jb);
      for (int t = tid; t < jn; t += kPlanThreads) {
        s_prior[t] = a.span_prior[lo + jb + t];
        s_start[t] = a.span_start[lo + jb + t];
      }
      __syncthreads();
      if (act)
        for (int t = 0; t < jn; ++t) rank += ranks_before(s_prior[t], s_start[t], jb + t, pi, si, i);
    }
    if (act) {
      a.perm[lo + rank] = i;
      if (a.span_selected) a.span_selected[lo + i] = 0;
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
  // Lane l holds the clipped span of rank r0 + l, so one global round trip
  // serves 64 decisions. Page mode: every page except the last (always
  // selected) holds 16 tokens, so a span costs 16 x (its pages not yet
  // selected), counted with a ballot over 64 pages at a time. Token mode: a
  // span costs its tokens not yet visible, 64 bitmap words at a time.
  if (tid < 64) {
    long long used = s_used;
    int taken = 0;
    const long long T = a.budget[b];
    bool stop = false;
    for (int r0 = 0; r0 < n && !stop; r0 += 64) {
      int my_i = -1, my_x = 0, my_e = 0;
      if (r0 + lane < n) {
        my_i = lo + a.perm[lo + r0 + lane];
        const long long st = a.span_start[my_i];
        const long long x = st > 0 ? st : 0;
        long long e = st + (long long)a.span_len[my_i];
        if (e > L) e = L;
        my_x = (int)x;
        my_e = (int)(e > x ? e : x);                    // e <= x: empty after clipping
      }
      const int cnt = min(64, n - r0);
      for (int j = 0; j < cnt; ++j) {
        const int i = __builtin_amdgcn_readlane(my_i, j);
        const int x = __builtin_amdgcn_readlane(my_x, j);
        const int e = __builtin_amdgcn_readlane(my_e, j);
        if (e <= x) continue;                           // ignored
        long long cost = 0;
        int u0, u1;                                     // bitmap units (pages / words) touched
        if constexpr (TOK) {
          u0 = x >> 5;
          u1 = ((e - 1) >> 5) + 1;
          for (int w = u0 + lane; w - lane < u1; w += 64) {
            const int c = w < u1 ? __popc(range_bits(w, x, e) & ~bitmap[w]) : 0;
            cost += wave_count_sum(c);
          }
        } else {
          u0 = x / kPage;
          u1 = (e + kPage - 1) / kPage;
          int new_pages = 0;
          for (int p = u0; p < u1; p += 64) {
            const int pp = p + lane;
            const bool fresh = pp < u1 && !((bitmap[pp >> 5] >> (pp & 31)) & 1u);
            new_pages += __popcll(__ballot(fresh));
          }
          cost = (long long)kPage * new_pages;
        }
        if (used + cost <= T) {
          if constexpr (TOK) {
            for (int w = u0 + lane; w < u1; w += 64) bitmap[w] |= range_bits(w, x, e);
          } else {
            for (int p = u0 + lane; p < u1; p += 64) atomicOr(&bitmap[p >> 5], 1u << (p & 31));
          }
          used += cost;
          ++taken;
          if (lane == 0 && a.span_selected) a.span_selected[i] = 1;
        } else if (a.policy == 1 /*KAP_SELECT_STOP*/) {
          stop = true;
          break;
        }
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      }
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
  bool bad = false;
  auto emit = [&](int p, uint32_t mask) {
    const int page = fbt_row[p];
    bad |= (page < 0) || ((int64_t)page >= a.num_pages);
    vlb[out] = p;
    vbt[out] = page;
    if constexpr (TOK) a.view_mask[(size_t)b * a.capacity + out] = mask;
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
  return (words + 1) * sizeof(uint32_t);   // + a spare word
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

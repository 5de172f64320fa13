// kap_compile_plan on the GPU: Alg. 1 of the paper, SelectEvidenceUnderBudget
// through BuildBlockTable, one workgroup per sequence.
//
// Per sequence the workgroup
//   1. checks the CSR bounds, the length and the scores (status codes),
//   2. marks the mandatory prefix / suffix pages in an LDS page bitmap,
//   3. ranks the spans by (prior desc, start asc, index asc) -- every thread
//      counts, for its spans, how many spans precede them, and writes the
//      inverse permutation to the workspace,
//   4. walks the spans in rank order with one wavefront: the 64 lanes test the
//      span's pages against the bitmap, a wavefront ballot counts the new
//      pages (their cost in visible tokens), and the span is taken when it fits
//      the budget,
//   5. compacts the bitmap into the ascending logical-page list and maps it
//      through the full block table.
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

__global__ __launch_bounds__(kPlanThreads) void compile_plan_kernel(PlanArgs a) {
  extern __shared__ uint32_t bitmap[];
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

  // -- mandatory pages --------------------------------------------------------
  const int W = (NP + 31) / 32;
  for (int w = tid; w < W; w += kPlanThreads) bitmap[w] = 0u;
  __syncthreads();
  const int pre = min(max(a.prefix[b], 0), L);
  const int suf_start = max(0, L - max(a.suffix[b], 1));
  const int pre_pages = (pre + kPage - 1) / kPage;     // pages [0, pre_pages)
  const int suf_page0 = suf_start / kPage;             // pages [suf_page0, NP)
  for (int p = tid; p < pre_pages; p += kPlanThreads) atomicOr(&bitmap[p >> 5], 1u << (p & 31));
  for (int p = suf_page0 + tid; p < NP; p += kPlanThreads)
    atomicOr(&bitmap[p >> 5], 1u << (p & 31));

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

  // -- visible tokens of the mandatory pages ---------------------------------
  const int last_valid = L - kPage * (NP - 1);          // 1..16
  {
    int c = 0;
    for (int w = tid; w < W; w += kPlanThreads) c += __popc(bitmap[w]);
    int total = 0;
    block_exclusive_scan(c, s_scan, &total);
    if (tid == 0) {
      // the last page is always selected (suffix >= 1 token)
      s_used = (long long)kPage * total - (kPage - last_valid);
      s_taken = 0;
    }
  }
  __syncthreads();

  // -- greedy selection in rank order (one wavefront) -------------------------
  // Lane l holds the clipped span of rank r0 + l, so one global round trip
  // serves 64 decisions. Every page except the last (always selected) holds 16
  // tokens, so a span's cost is 16 x (its pages not yet selected), counted with
  // a wavefront ballot over 64 pages at a time.
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
        const int p0 = x / kPage;
        const int p1 = (e + kPage - 1) / kPage;
        int new_pages = 0;
        for (int p = p0; p < p1; p += 64) {
          const int pp = p + lane;
          const bool fresh = pp < p1 && !((bitmap[pp >> 5] >> (pp & 31)) & 1u);
          new_pages += __popcll(__ballot(fresh));
        }
        const long long cost = (long long)kPage * new_pages;
        if (used + cost <= T) {
          for (int p = p0 + lane; p < p1; p += 64) atomicOr(&bitmap[p >> 5], 1u << (p & 31));
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
  const int chunk = (W + kPlanThreads - 1) / kPlanThreads;
  const int w0 = min(W, tid * chunk);
  const int w1 = min(W, w0 + chunk);
  int mine = 0;
  for (int w = w0; w < w1; ++w) mine += __popc(bitmap[w]);
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
  for (int w = w0; w < w1; ++w) {
    uint32_t bits = bitmap[w];
    while (bits) {
      const int bit = __ffs(bits) - 1;
      bits &= bits - 1u;
      const int p = w * 32 + bit;
      const int page = fbt_row[p];
      bad |= (page < 0) || ((int64_t)page >= a.num_pages);
      vlb[out] = p;
      vbt[out] = page;
      ++out;
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

}  // namespace

hipError_t launch_compile_plan(const PlanArgs &a, hipStream_t s) {
  const size_t words = (size_t)(a.fbt_stride + 31) / 32 + 1;   // + spare count word
  hipLaunchKernelGGL(compile_plan_kernel, dim3(a.batch), dim3(kPlanThreads),
                     words * sizeof(uint32_t), s, a);
  return hipGetLastError();
}

}  // namespace kap

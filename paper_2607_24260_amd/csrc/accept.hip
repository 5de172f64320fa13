// Target-guided tolerant acceptance of a verify window (Sec. 3.2 of the
// paper, "Full-context verification": a proposed token is accepted when it is
// among the verifier's top candidates; top 3 in the paper).
//
// Two launches. The row kernel streams the verifier's logits: a grid of
// (vocabulary chunk, window row) workgroups, each counting the tokens of its
// chunk that rank before the row's draft token and taking the chunk's argmax;
// both are combined per row with device-scope vector atomics (integer add, and
// 64-bit max of (orderable value, inverted index), so the largest value and
// then the lowest index win). The finalize kernel walks each window, sets the
// accepted count m and the carry token argmax(row m), and zeroes the row
// counters for the next call. Integer results: exact.
#include "kap_internal.h"

namespace kap {
namespace {

constexpr int kThreads = 256;

// Monotone map of a float to an unsigned key (-0 folded into +0).
__device__ __forceinline__ uint32_t order_key(float x) {
  if (x == 0.f) x = 0.f;
  const uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// 8 logits at j (16-byte aligned): the raw 16-byte words, then the values.
template <int F32> struct Raw8;
template <> struct Raw8<1> { kv_u32x4 a, b; };
template <> struct Raw8<0> { kv_u32x4 a; };

template <int F32>
__device__ __forceinline__ Raw8<F32> load8(const void *row, int j) {
  Raw8<F32> r;
  if constexpr (F32) {
    const kv_u32x4 *p = reinterpret_cast<const kv_u32x4 *>(static_cast<const float *>(row) + j);
    r.a = __builtin_nontemporal_load(p);
    r.b = __builtin_nontemporal_load(p + 1);
  } else {
    r.a = __builtin_nontemporal_load(
        reinterpret_cast<const kv_u32x4 *>(static_cast<const uint16_t *>(row) + j));
  }
  return r;
}

template <int F32>
__device__ __forceinline__ void values8(const Raw8<F32> &r, float v[8]) {
  if constexpr (F32) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[e] = __uint_as_float(r.a[e]);
      v[4 + e] = __uint_as_float(r.b[e]);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[2 * e] = bf16_lo(r.a[e]);
      v[2 * e + 1] = bf16_hi(r.a[e]);
    }
  }
}

template <int F32>
__device__ __forceinline__ float load1(const void *row, int j) {
  if constexpr (F32) return static_cast<const float *>(row)[j];
  return __uint_as_float((uint32_t)static_cast<const uint16_t *>(row)[j] << 16);
}

template <int F32>
__global__ __launch_bounds__(kThreads) void accept_rows_kernel(AcceptArgs a) {
  __shared__ int s_cnt[kThreads / 64];
  __shared__ unsigned long long s_best[kThreads / 64];
  const int row = blockIdx.y;                          // b * window + i
  const int b = row / a.window, i = row - b * a.window;
  const int j0 = blockIdx.x * kAcceptChunk;
  const int j1 = min(a.vocab, j0 + kAcceptChunk);
  const void *lrow = static_cast<const char *>(a.logits) +
                     (size_t)row * a.vocab * (F32 ? 4 : 2);
  // the draft of this position (none for the last one, or out of range)
  const int d = i < a.window - 1 ? a.drafts[(size_t)b * (a.window - 1) + i] : -1;
  const bool has_d = d >= 0 && d < a.vocab;
  const float xd = has_d ? load1<F32>(lrow, d) : 0.f;
  // Each thread visits its tokens in increasing index order, so a strict >
  // keeps the lowest index among equal maxima; the packed key is formed once.
  int cnt = 0;
  float bv = -INFINITY;
  int bi = -1;
  auto visit = [&](float x, int j) {
    cnt += (x > xd) | ((x == xd) & (j < d));
    if (bi < 0 || x > bv) {
      bv = x;
      bi = j;
    }
  };
  // 8 tokens per load, four loads in flight per step; the vocabulary tail
  // one by one (rows are 16-byte aligned only when vocab * size % 16 == 0,
  // otherwise the whole row goes one by one)
  const bool vec = ((size_t)a.vocab * (F32 ? 4 : 2)) % 16 == 0;
  int j = j0 + threadIdx.x * 8;
  if (vec) {
    constexpr int kStep = kThreads * 8;
    for (; j + 3 * kStep + 8 <= j1; j += 4 * kStep) {
      Raw8<F32> r[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) r[u] = load8<F32>(lrow, j + u * kStep);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        float v[8];
        values8<F32>(r[u], v);
#pragma unroll
        for (int e = 0; e < 8; ++e) visit(v[e], j + u * kStep + e);
      }
    }
    for (; j + 8 <= j1; j += kStep) {
      float v[8];
      values8<F32>(load8<F32>(lrow, j), v);
#pragma unroll
      for (int e = 0; e < 8; ++e) visit(v[e], j + e);
    }
    for (; j < j1; j += kThreads * 8)
      for (int e = j; e < min(j + 8, j1); ++e) visit(load1<F32>(lrow, e), e);
  } else {
    for (int e = j0 + threadIdx.x; e < j1; e += kThreads) visit(load1<F32>(lrow, e), e);
  }
  if (!has_d) cnt = 0;
  unsigned long long best =
      bi < 0 ? 0ull : ((unsigned long long)order_key(bv) << 32) | (0xFFFFFFFFu - (uint32_t)bi);
  // workgroup reduction, then one atomic each per workgroup
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    cnt += __shfl_xor(cnt, o, 64);
    const unsigned long long y = __shfl_xor(best, o, 64);
    best = y > best ? y : best;
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    s_cnt[w] = cnt;
    s_best[w] = best;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int c = 0;
    unsigned long long m = 0;
    for (int k = 0; k < kThreads / 64; ++k) {
      c += s_cnt[k];
      m = s_best[k] > m ? s_best[k] : m;
    }
    if (c) atomicAdd(a.row_count + row, c);
    atomicMax(a.row_best + row, m);
  }
}

__global__ __launch_bounds__(kThreads) void accept_finalize_kernel(AcceptArgs a) {
  const int b = blockIdx.x * kThreads + threadIdx.x;
  if (b >= a.batch) return;
  const int k = a.window - 1;
  int m = 0;
  while (m < k) {
    const int d = a.drafts[(size_t)b * k + m];
    if (d < 0 || d >= a.vocab || a.row_count[b * a.window + m] >= a.top_k) break;
    ++m;
  }
  const unsigned long long best = a.row_best[b * a.window + m];
  a.accepted[b] = m;
  a.carry[b] = (int)(0xFFFFFFFFu - (uint32_t)(best & 0xFFFFFFFFull));
  for (int i = 0; i < a.window; ++i) {
    a.row_count[b * a.window + i] = 0;
    a.row_best[b * a.window + i] = 0;
  }
}

}  // namespace

hipError_t launch_accept_top3(const AcceptArgs &a, hipStream_t s) {
  const dim3 grid((a.vocab + kAcceptChunk - 1) / kAcceptChunk, a.batch * a.window);
  if (a.f32)
    hipLaunchKernelGGL(accept_rows_kernel<1>, grid, dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL(accept_rows_kernel<0>, grid, dim3(kThreads), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(accept_finalize_kernel, dim3((a.batch + kThreads - 1) / kThreads),
                     dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace kap

// Log-sum-exp merge of split-KV partial attention.
//
// Split s of a row holds the normalised attention o_s over its keys and
// lse_s = log2 sum exp2(z) (log2 units). Over the union of keys,
//   lse = log2 sum_s 2^lse_s,   o = sum_s 2^(lse_s - lse) o_s;
// splits without keys (lse_s = -inf) drop out. The final LSE is written in
// natural-log units. One wavefront per row; lanes cover the head dims.
#include "kap_internal.h"

namespace kap {
namespace {

__global__ __launch_bounds__(64) void merge_kernel(const float *__restrict__ part_o,
                                                    const float *__restrict__ part_lse,
                                                    float *__restrict__ out,
                                                    float *__restrict__ lse, int n_split, int D) {
  const size_t row = blockIdx.x;
  const int lane = threadIdx.x;
  const float *pl = part_lse + row * n_split;
  float m = -INFINITY;
  for (int s = lane; s < n_split; s += 64) m = fmaxf(m, pl[s]);
  m = wave_max(m);
  if (m == -INFINITY) {
    for (int d = lane; d < D; d += 64) out[row * D + d] = 0.f;
    if (lane == 0) lse[row] = -INFINITY;
    return;
  }
  float tot = 0.f;
  for (int s = lane; s < n_split; s += 64) tot += exp2f(pl[s] - m);
  tot = wave_sum(tot);
  const float inv = 1.f / tot;
  const float *po = part_o + row * (size_t)n_split * D;
  for (int d = lane; d < D; d += 64) {
    float acc = 0.f;
    for (int s = 0; s < n_split; ++s) {
      const float w = exp2f(pl[s] - m);
      if (w != 0.f) acc = fmaf(w, po[(size_t)s * D + d], acc);
    }
    out[row * D + d] = acc * inv;
  }
  if (lane == 0) lse[row] = (m + log2f(tot)) * kLn2;
}

}  // namespace

hipError_t launch_merge(const AttnArgs &a, hipStream_t s) {
  const unsigned rows = (unsigned)(a.batch * a.q_len * a.Hq);
  hipLaunchKernelGGL(merge_kernel, dim3(rows), dim3(64), 0, s, a.part_o, a.part_lse, a.out,
                     a.lse, a.n_split, a.D);
  return hipGetLastError();
}

}  // namespace kap

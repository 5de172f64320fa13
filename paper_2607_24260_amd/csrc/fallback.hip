// The executor's access-mode policy for one cycle, on the device (Sec. 3.2
// "Runtime stability and fallback"; h = accepted / speculated, Eq. (5); the
// margin condition h > s, Eq. (12)), together with the switch of the active
// view rows: with it, a whole proposal / verify stream runs without host
// round trips and can be captured in a HIP graph.
//
// One workgroup per sequence: thread 0 updates the sequence's history and
// mode; then the workgroup rewrites the sequence's active view row if its
// mode was (re)set (with token-granular views, also its token-mask row: the
// plan's masks, or all 16 tokens of every page on full context). h <= s is
// compared exactly, in integers: A * seq_len <= view_tokens * S.
#include "kap_internal.h"

namespace kap {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void fallback_update_kernel(FallbackArgs a) {
  __shared__ int s_write;   // 0: nothing, 1: the plan's row, 2: the full-context row
  const int b = blockIdx.x;
  if (threadIdx.x == 0) {
    int write = 0;
    int32_t *h = a.history + (size_t)b * a.window * 2;
    if (a.reset) {
      for (int i = 0; i < 2 * a.window; ++i) h[i] = 0;
      a.cycles[b] = 0;
      const int m = a.plan_status[b] == 0 ? 0 : 1;
      a.mode[b] = m;
      write = m == 0 ? 1 : 2;
    } else {
      const int c = a.cycles[b];
      const int acc = min(max(a.accepted[b], 0), a.gamma);
      const int slot = c % a.window;
      h[2 * slot] = acc;
      h[2 * slot + 1] = a.gamma;
      a.cycles[b] = c + 1;
      if (a.mode[b] == 0 && c + 1 >= 2) {
        long long A = 0, S = 0;   // slots never written are zero since the reset
        for (int i = 0; i < a.window; ++i) {
          A += h[2 * i];
          S += h[2 * i + 1];
        }
        const long long L = a.seq_lens[b], V = a.view_tokens[b];
        if (S > 0 && A * L <= V * S) {
          a.mode[b] = 1;
          write = 2;
        }
      }
    }
    s_write = write;
  }
  __syncthreads();
  const int write = s_write;
  if (write == 0) return;
  int32_t *vbt = a.view_bt + (size_t)b * a.view_stride;
  int32_t *vlb = a.view_lb + (size_t)b * a.view_stride;
  if (write == 1) {
    const int nb = a.sel_nb[b];
    const int n = max(0, min(nb, a.sel_stride));
    const int32_t *sbt = a.sel_bt + (size_t)b * a.sel_stride;
    const int32_t *slb = a.sel_lb + (size_t)b * a.sel_stride;
    for (int j = threadIdx.x; j < n; j += kThreads) {
      vbt[j] = sbt[j];
      vlb[j] = slb[j];
    }
    if (a.view_mask) {
      const uint32_t *smk = a.sel_mask + (size_t)b * a.sel_stride;
      uint32_t *vmk = a.view_mask + (size_t)b * a.view_stride;
      for (int j = threadIdx.x; j < n; j += kThreads) vmk[j] = smk[j];
    }
    if (threadIdx.x == 0) a.view_nb[b] = nb;
  } else {
    const int L = a.seq_lens[b];
    const int np = L > 0 ? (int)(((long long)L + kPage - 1) / kPage) : 0;
    const int n = min(np, a.full_stride);
    const int32_t *fbt = a.full_bt + (size_t)b * a.full_stride;
    for (int j = threadIdx.x; j < n; j += kThreads) {
      vbt[j] = fbt[j];
      vlb[j] = j;
    }
    if (a.view_mask) {
      uint32_t *vmk = a.view_mask + (size_t)b * a.view_stride;
      for (int j = threadIdx.x; j < n; j += kThreads) vmk[j] = 0xFFFFu;
    }
    if (threadIdx.x == 0) a.view_nb[b] = n;
  }
}

}  // namespace

hipError_t launch_fallback_update(const FallbackArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(fallback_update_kernel, dim3(a.batch), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace kap

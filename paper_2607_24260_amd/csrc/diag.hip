// Streaming-read kernel: the HBM read rate a plain, fully coalesced kernel
// reaches on this device -- the practical ceiling the attention kernels'
// bandwidth is compared with.
//
// One workgroup of four wavefronts per compute unit; the wavefronts take the
// buffer's 4 KB blocks round-robin, two blocks (eight 16-byte non-temporal
// loads per lane) in flight. Of the launch shapes tried on MI355X (grid-stride
// loops of 1024-4096 workgroups, 1-4 workgroups per CU, 2 or 4 blocks in
// flight, contiguous or round-robin partitions) this one read fastest at both
// 118 MB and 2 GiB. The words are XOR-folded so the loads cannot be dropped;
// each wavefront adds its fold to the sink with one vector atomic.
#include "kap_internal.h"

namespace kap {
namespace {

constexpr int kThreads = 256;
constexpr int kBlock16 = 256;   // 16-byte words per 4 KB block
constexpr int kInFlight = 2;    // blocks per wavefront per step

__global__ __launch_bounds__(kThreads) void stream_read_kernel(const kv_u32x4 *src, size_t n16,
                                                               uint32_t *sink) {
  const int lane = threadIdx.x & 63;
  const size_t nblk = n16 / kBlock16;
  const size_t nw = (size_t)gridDim.x * (kThreads / 64);
  size_t w = (size_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  uint32_t acc = 0;
  for (; w + (kInFlight - 1) * nw < nblk; w += kInFlight * nw) {
    kv_u32x4 r[kInFlight][4];
#pragma unroll
    for (int u = 0; u < kInFlight; ++u)
#pragma unroll
      for (int c = 0; c < 4; ++c)
        r[u][c] = __builtin_nontemporal_load(src + (w + u * nw) * kBlock16 + c * 64 + lane);
#pragma unroll
    for (int u = 0; u < kInFlight; ++u)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc ^= r[u][c][0] ^ r[u][c][1] ^ r[u][c][2] ^ r[u][c][3];
  }
  for (; w < nblk; w += nw)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const kv_u32x4 r = __builtin_nontemporal_load(src + w * kBlock16 + c * 64 + lane);
      acc ^= r[0] ^ r[1] ^ r[2] ^ r[3];
    }
  // the words past the last whole block
  const size_t t = (size_t)blockIdx.x * kThreads + threadIdx.x;
  for (size_t i = nblk * kBlock16 + t; i < n16; i += (size_t)gridDim.x * kThreads) {
    const kv_u32x4 r = __builtin_nontemporal_load(src + i);
    acc ^= r[0] ^ r[1] ^ r[2] ^ r[3];
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) acc ^= __shfl_xor(acc, o, 64);
  if (lane == 0 && acc) atomicXor(sink, acc);
}

}  // namespace

hipError_t launch_stream_read(const void *src, size_t bytes, uint32_t *sink, hipStream_t s) {
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(stream_read_kernel, dim3(cus > 0 ? cus : 1), dim3(kThreads), 0, s,
                     static_cast<const kv_u32x4 *>(src), bytes / 16, sink);
  return hipGetLastError();
}

}  // namespace kap

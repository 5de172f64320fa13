// KV maintenance kernels: the slot-mapped append of new tokens (Sec. 3.1
// slot mappings; Sec. 3.2 KV^{full,+}) and the copy of a selected-KV view
// into a compact workspace of fixed capacity (Alg. 1, AssignCompactSlots and
// BuildBlockTable; Sec. 3.1 "Selected-KV view materialization").
//
// Both move stored bits only (no arithmetic), so their results are exact.
// The compaction streams whole pages: in the library's layout the K tiles of
// all KV heads of one page are one contiguous block (and so are the V
// tiles), copied with 16-byte nontemporal loads and stores.
#include "kap_internal.h"

namespace kap {
namespace {

constexpr int kThreads = 256;

// ---------------------------------------------------------------------------
// append: one workgroup per new token
// ---------------------------------------------------------------------------

// Copies elements of type T (the stored KV type). K: element (g, d) of the token goes to
// [page][g][d / 8][off][d % 8]; V: to [page][g][d][off].
template <typename T>
__device__ void append_token(const AppendArgs &a, int t, int64_t page, int off) {
  const int Hkv = a.Hkv, D = a.D, C = D / 8;
  const T *kn = static_cast<const T *>(a.k_new) + (size_t)t * Hkv * D;
  const T *vn = static_cast<const T *>(a.v_new) + (size_t)t * Hkv * D;
  T *kp = static_cast<T *>(a.k_pages) + (size_t)page * Hkv * D * kPage;
  T *vp = static_cast<T *>(a.v_pages) + (size_t)page * Hkv * D * kPage;
  for (int e = threadIdx.x; e < Hkv * D; e += blockDim.x) {
    const int g = e / D, d = e - g * D;
    kp[(((size_t)g * C + d / 8) * kPage + off) * 8 + (d & 7)] = kn[e];
    vp[((size_t)g * D + d) * kPage + off] = vn[e];
  }
}

__global__ __launch_bounds__(kThreads) void append_kv_kernel(AppendArgs a) {
  const int t = blockIdx.x;
  const int64_t slot = a.slots[t];
  if (slot < 0) return;                                   // padding
  if (slot >= a.num_pages * kPage) {
    if (threadIdx.x == 0 && a.bad_slots) atomicAdd(a.bad_slots, 1);
    return;
  }
  const int64_t page = slot / kPage;
  const int off = (int)(slot - page * kPage);
  if (a.elem_bytes == 4)
    append_token<uint32_t>(a, t, page, off);
  else if (a.elem_bytes == 2)
    append_token<uint16_t>(a, t, page, off);
  else
    append_token<uint8_t>(a, t, page, off);
}

// ---------------------------------------------------------------------------
// compaction: workgroups stride over (sequence, view entry)
// ---------------------------------------------------------------------------

__device__ __forceinline__ void copy_block(const char *src, char *dst, size_t bytes) {
  // bytes is a multiple of 16 (Hkv * D * 16 elements of >= 1 byte, D % 8 == 0)
  const kv_u32x4 *s = reinterpret_cast<const kv_u32x4 *>(src);
  kv_u32x4 *d = reinterpret_cast<kv_u32x4 *>(dst);
  const size_t n = bytes / 16;
  size_t i = threadIdx.x;
  for (; i + 3 * kThreads < n; i += 4 * kThreads) {
    const kv_u32x4 x0 = __builtin_nontemporal_load(s + i);
    const kv_u32x4 x1 = __builtin_nontemporal_load(s + i + kThreads);
    const kv_u32x4 x2 = __builtin_nontemporal_load(s + i + 2 * kThreads);
    const kv_u32x4 x3 = __builtin_nontemporal_load(s + i + 3 * kThreads);
    __builtin_nontemporal_store(x0, d + i);
    __builtin_nontemporal_store(x1, d + i + kThreads);
    __builtin_nontemporal_store(x2, d + i + 2 * kThreads);
    __builtin_nontemporal_store(x3, d + i + 3 * kThreads);
  }
  for (; i < n; i += kThreads) __builtin_nontemporal_store(__builtin_nontemporal_load(s + i), d + i);
}

__global__ __launch_bounds__(kThreads) void compact_view_kernel(CompactArgs a) {
  const size_t page_bytes = (size_t)a.Hkv * a.D * kPage * a.elem_bytes;
  const long long total = (long long)a.batch * a.capacity;
  for (long long idx = blockIdx.x; idx < total; idx += gridDim.x) {
    const int b = (int)(idx / a.capacity);
    const int j = (int)(idx - (long long)b * a.capacity);
    const int nb = min(a.view_num_blocks[b], a.capacity);
    int dst = -1;
    if (j < nb) {
      const int p = a.view_bt[(size_t)b * a.view_stride + j];
      if (p >= 0 && (int64_t)p < a.src_pages) {
        dst = (int)idx;                                   // b * capacity + j
        copy_block(static_cast<const char *>(a.src_k) + (size_t)p * page_bytes,
                   static_cast<char *>(a.dst_k) + (size_t)dst * page_bytes, page_bytes);
        copy_block(static_cast<const char *>(a.src_v) + (size_t)p * page_bytes,
                   static_cast<char *>(a.dst_v) + (size_t)dst * page_bytes, page_bytes);
        if (a.src_scales && threadIdx.x < 2)
          a.dst_scales[2 * (size_t)dst + threadIdx.x] = a.src_scales[2 * (size_t)p + threadIdx.x];
      }
    }
    if (threadIdx.x == 0) a.compact_bt[idx] = dst;
  }
}

}  // namespace

hipError_t launch_append_kv(const AppendArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(append_kv_kernel, dim3(a.num_tokens), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_compact_view(const CompactArgs &a, int grid, hipStream_t s) {
  hipLaunchKernelGGL(compact_view_kernel, dim3(grid), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace kap

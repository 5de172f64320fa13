// Generic split-KV attention for any KV dtype, any GQA ratio and head_dim in
// {64, 128, 256}: one wavefront per (sequence, query row, key split).
//
// It serves the float32 workload and geometries the tuned kernels do not
// cover. Each work item stages up to 1024 scores in LDS: pass 1 (lanes over
// keys) computes the scaled logits, pass 2 (lanes over head dims) forms the
// normalised partial output. Partials go to the workspace; the LSE merge kernel
// (merge.hip) combines the splits.
#include "kap_internal.h"

namespace kap {
namespace {

// Eight consecutive stored elements starting at element idx (a multiple of
// 4, so every load below is aligned), widened to float: one K chunk of one
// token, or with n4 = 1 the first four only (four tokens of one V row).
template <int KV>
__device__ __forceinline__ void load8(const void *base, size_t idx, float out[8], bool n4 = false) {
  if constexpr (KV == kF32) {
    const float4 *p = reinterpret_cast<const float4 *>(static_cast<const float *>(base) + idx);
    const float4 x = p[0];
    out[0] = x.x; out[1] = x.y; out[2] = x.z; out[3] = x.w;
    if (!n4) {
      const float4 y = p[1];
      out[4] = y.x; out[5] = y.y; out[6] = y.z; out[7] = y.w;
    }
  } else if constexpr (KV == kBF16) {
    const uint16_t *h = static_cast<const uint16_t *>(base) + idx;
    uint32_t w[4];
    const uint2 x = *reinterpret_cast<const uint2 *>(h);
    w[0] = x.x; w[1] = x.y;
    if (!n4) {
      const uint2 y = *reinterpret_cast<const uint2 *>(h + 4);
      w[2] = y.x; w[3] = y.y;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (n4 && e >= 2) break;
      out[2 * e] = __uint_as_float(w[e] << 16);
      out[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
    }
  } else {
    const uint8_t *c = static_cast<const uint8_t *>(base) + idx;
    const uint32_t x = *reinterpret_cast<const uint32_t *>(c);
    const uint32_t y = n4 ? 0u : *reinterpret_cast<const uint32_t *>(c + 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      out[e] = fp8_to_f32((uint8_t)(x >> (8 * e)));
      out[4 + e] = fp8_to_f32((uint8_t)(y >> (8 * e)));
    }
  }
}

template <int KV, int D>
__global__ __launch_bounds__(64) void attn_generic_kernel(AttnArgs a) {
  constexpr int kKeys = kGenericPagesPerSplit * kPage;
  __shared__ float qs[D];
  __shared__ float ps[kKeys];

  const int split = blockIdx.x;
  const int r = blockIdx.y;          // row within the sequence
  const int b = blockIdx.z;
  const int lane = threadIdx.x;
  const int R = a.q_len * a.Hq;
  const int i = r / a.Hq;
  const int h = r % a.Hq;
  const int g = h / a.G;

  const int L = a.seq_lens[b];
  const int np_seq = L > 0 ? (int)(((long long)L + kPage - 1) / kPage) : 0;
  int nb = a.num_blocks ? a.num_blocks[b] : np_seq;
  nb = max(0, min(nb, a.max_blocks));
  const int limit = a.causal ? (L - a.q_len + i + 1) : L;   // visible positions < limit
  // split `split` of n_split takes an even share (<= pages_per_split pages)
  const int k0 = (int)(((long long)split * nb) / a.n_split);
  const int k1 = (int)(((long long)(split + 1) * nb) / a.n_split);
  const size_t row = (size_t)b * R + r;
  float *po = (a.n_split == 1) ? a.out + row * D : a.part_o + (row * a.n_split + split) * D;

  // query row -> LDS (float)
  for (int d = lane; d < D; d += 64) {
    const size_t qi = row * D + d;
    qs[d] = a.q_f32 ? static_cast<const float *>(a.q)[qi]
                    : __uint_as_float(static_cast<uint32_t>(
                          static_cast<const uint16_t *>(a.q)[qi]) << 16);
  }
  __syncthreads();

  // pass 1: scaled logits (log2 units), lanes over keys
  const int nkeys = max(0, k1 - k0) * kPage;
  float mx = -INFINITY;
  for (int t = lane; t < nkeys; t += 64) {
    const int k = k0 + t / kPage;
    const int tok = t % kPage;
    const int page = a.block_table[(size_t)b * a.bt_stride + k];
    const int lb = a.logical_block ? a.logical_block[(size_t)b * a.bt_stride + k] : k;
    const long long pos = (long long)lb * kPage + tok;
    const bool shown =
        !a.token_mask || ((a.token_mask[(size_t)b * a.bt_stride + k] >> tok) & 1u);
    float z = -INFINITY;
    if (shown && page >= 0 && page < a.num_pages && pos < limit && pos < L) {
      // K page tile: [D/8 chunks][16 tokens][8 dims]; one chunk per load
      const size_t kbase = ((size_t)page * a.Hkv + g) * kPage * D + (size_t)tok * 8;
      float acc = 0.f;
      for (int c = 0; c < D / 8; ++c) {
        float kc[8];
        load8<KV>(a.k_pages, kbase + (size_t)c * (kPage * 8), kc);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc = fmaf(qs[8 * c + e], kc[e], acc);
      }
      if constexpr (KV == kFP8) acc *= a.kv_scales[2 * (size_t)page];
      z = acc * a.scale_log2;
    }
    ps[t] = z;
    mx = fmaxf(mx, z);
  }
  mx = wave_max(mx);
  const size_t lse_idx = (a.n_split == 1) ? row : row * a.n_split + split;
  if (mx == -INFINITY) {
    for (int d = lane; d < D; d += 64) po[d] = 0.f;
    if (lane == 0) {
      if (a.n_split == 1) a.lse[lse_idx] = -INFINITY;
      else a.part_lse[lse_idx] = -INFINITY;
    }
    return;
  }
  float sum = 0.f;
  for (int t = lane; t < nkeys; t += 64) {
    const float p = exp2f(ps[t] - mx);
    ps[t] = p;
    sum += p;
  }
  sum = wave_sum(sum);
  __syncthreads();

  // pass 2: lanes over head dims; V rows are dim-major ([D][16 tokens]), so
  // four consecutive tokens of a row come in one load
  for (int d = lane; d < D; d += 64) {
    float acc = 0.f;
    for (int t0 = 0; t0 < nkeys; t0 += 4) {
      const float p0 = ps[t0], p1 = ps[t0 + 1], p2 = ps[t0 + 2], p3 = ps[t0 + 3];
      if (p0 == 0.f && p1 == 0.f && p2 == 0.f && p3 == 0.f) continue;
      const int k = k0 + t0 / kPage;
      const int tok = t0 % kPage;
      const int page = a.block_table[(size_t)b * a.bt_stride + k];
      const size_t vidx = (((size_t)page * a.Hkv + g) * D + d) * kPage + tok;
      float v[8];
      load8<KV>(a.v_pages, vidx, v, true);
      // a zero weight contributes nothing, whatever the slot holds (slots
      // past the sequence end may hold anything, NaN included)
      const float t_0 = p0 != 0.f ? p0 * v[0] : 0.f, t_1 = p1 != 0.f ? p1 * v[1] : 0.f;
      const float t_2 = p2 != 0.f ? p2 * v[2] : 0.f, t_3 = p3 != 0.f ? p3 * v[3] : 0.f;
      float s = (t_0 + t_1) + (t_2 + t_3);
      if constexpr (KV == kFP8) s *= a.kv_scales[2 * (size_t)page + 1];
      acc += s;
    }
    po[d] = acc / sum;
  }
  if (lane == 0) {
    const float l2 = mx + log2f(sum);
    if (a.n_split == 1) a.lse[lse_idx] = l2 * kLn2;
    else a.part_lse[lse_idx] = l2;
  }
}

template <int KV>
hipError_t launch_kv(const AttnArgs &a, hipStream_t s) {
  const dim3 grid(a.n_split, a.q_len * a.Hq, a.batch);
  switch (a.D) {
    case 64: hipLaunchKernelGGL((attn_generic_kernel<KV, 64>), grid, dim3(64), 0, s, a); break;
    case 128: hipLaunchKernelGGL((attn_generic_kernel<KV, 128>), grid, dim3(64), 0, s, a); break;
    case 256: hipLaunchKernelGGL((attn_generic_kernel<KV, 256>), grid, dim3(64), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_generic(const AttnArgs &a, hipStream_t s) {
  switch (a.kv_type) {
    case kF32: return launch_kv<kF32>(a, s);
    case kBF16: return launch_kv<kBF16>(a, s);
    case kFP8: return launch_kv<kFP8>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace kap

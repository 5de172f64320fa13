// Full-KV verification attention on the matrix cores (Sec. 3.2 of the paper,
// "Full-context verification"; Eq. (2)) for bf16 / fp8 KV, head_dim 128, four
// query heads per KV head, window q_len <= 16.
//
// The q_len window tokens times the four heads of one KV head form
// R = 4 * q_len query rows that share every key: a real dense contraction.
// One wavefront owns (key split, KV head, sequence) and walks the split two
// pages (32 keys) at a time with v_mfma_f32_16x16x32_bf16:
//   S^T[key][row] = K[key][:] . Q[row][:]       A = K tile (16 keys x 32 dims,
//                                               one 16-byte load per lane),
//                                               B = Q^T (kept in registers)
//   O^T[dim][row] += V^T[dim][key] P^T[key][row] A = V^T tile (dim-major pages:
//                                               4 keys = 8 contiguous bytes),
//                                               B = P^T, which the S^T
//                                               accumulator layout already
//                                               holds lane for lane.
// Lane (j = lane/16, n = lane%16) thus owns query row n of each 16-row tile and
// keys 4j..4j+3 of both pages, so the online softmax needs only two cross-row
// steps per page pair. P is split into bf16 hi + lo parts (two PV products),
// which keeps the probability rounding error below 2^-16 relative.
// The causal mask and the partial last page are handled on the last pages only.
#include "kap_internal.h"

namespace kap {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kD = 128;

__device__ __forceinline__ f32x4 mfma(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ float xor16_max(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_int(x), __float_as_int(x), false, false);
  return fmaxf(__int_as_float(r[0]), __int_as_float(r[1]));
}
__device__ __forceinline__ float xor32_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_int(x), __float_as_int(x), false, false);
  return fmaxf(__int_as_float(r[0]), __int_as_float(r[1]));
}
__device__ __forceinline__ float xor16_sum(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_int(x), __float_as_int(x), false, false);
  return __int_as_float(r[0]) + __int_as_float(r[1]);
}
__device__ __forceinline__ float xor32_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_int(x), __float_as_int(x), false, false);
  return __int_as_float(r[0]) + __int_as_float(r[1]);
}

__device__ __forceinline__ uint32_t pack_bf16_exact(float lo, float hi) {
  return __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), 0x07060302u);
}

// 4 E4M3FN codes (one dword) -> 2 dwords of bf16 pairs, exact
__device__ __forceinline__ u32x2 fp8x4_to_bf16x4(uint32_t w) {
  const float2 f0 = fp8x2_to_f32<false>(w);
  const float2 f1 = fp8x2_to_f32<true>(w);
  return u32x2{pack_bf16_exact(f0.x, f0.y), pack_bf16_exact(f1.x, f1.y)};
}

// K tile operand of one page for k-block kb: key n, dims 32kb + 8j .. +7
template <int KV>
__device__ __forceinline__ u32x4 load_k(const AttnArgs &a, int page, int g, int n, int j, int kb) {
  if constexpr (KV == kBF16) {
    const uint16_t *p = static_cast<const uint16_t *>(a.k_pages) +
                        ((size_t)page * a.Hkv + g) * (kPage * kD) + n * kD + kb * 32 + j * 8;
    return *reinterpret_cast<const u32x4 *>(p);
  } else {
    const uint8_t *p = static_cast<const uint8_t *>(a.k_pages) +
                       ((size_t)page * a.Hkv + g) * (kPage * kD) + n * kD + kb * 32 + j * 8;
    const u32x2 w = *reinterpret_cast<const u32x2 *>(p);
    const u32x2 lo = fp8x4_to_bf16x4(w[0]), hi = fp8x4_to_bf16x4(w[1]);
    return u32x4{lo[0], lo[1], hi[0], hi[1]};
  }
}

// V^T operand half: dim d, keys 4j .. 4j+3 of one page, as 2 dwords of bf16
template <int KV>
__device__ __forceinline__ u32x2 load_vt(const AttnArgs &a, int page, int g, int d, int j) {
  if constexpr (KV == kBF16) {
    const uint16_t *p = static_cast<const uint16_t *>(a.v_pages) +
                        ((size_t)page * a.Hkv + g) * (kPage * kD) + d * kPage + j * 4;
    return *reinterpret_cast<const u32x2 *>(p);
  } else {
    const uint8_t *p = static_cast<const uint8_t *>(a.v_pages) +
                       ((size_t)page * a.Hkv + g) * (kPage * kD) + d * kPage + j * 4;
    return fp8x4_to_bf16x4(*reinterpret_cast<const uint32_t *>(p));
  }
}

template <int KV, int NT>
__global__ __launch_bounds__(64) void verify_mfma_kernel(AttnArgs a) {
  const int split = blockIdx.x;
  const int g = blockIdx.y;
  const int b = blockIdx.z;
  const int lane = threadIdx.x;
  const int n = lane & 15, j = lane >> 4;
  const int R = a.q_len * 4;

  const int L = a.seq_lens[b];
  int np_seq = L > 0 ? (int)(((long long)L + kPage - 1) / kPage) : 0;
  np_seq = min(np_seq, a.max_blocks);
  const int k0 = split * a.pages_per_split;
  const int k1 = min(np_seq, k0 + a.pages_per_split);
  const int32_t *fbt = a.block_table + (size_t)b * a.bt_stride;

  // Q^T operand: row n of each tile, dims 32kb + 8j .. +7
  u32x4 qop[NT][4];
  int lim[NT];                       // row sees logical positions < lim
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int r = nt * 16 + n;
    const int i = r >> 2, hh = r & 3;
    lim[nt] = (r < R) ? (L - a.q_len + i + 1) : 0;
    const uint16_t *qp = static_cast<const uint16_t *>(a.q) +
                         (((size_t)b * a.q_len + (r < R ? i : 0)) * a.Hq + g * 4 + hh) * kD;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      qop[nt][kb] = (r < R) ? *reinterpret_cast<const u32x4 *>(qp + kb * 32 + j * 8)
                            : u32x4{0u, 0u, 0u, 0u};
    }
  }

  float m[NT], l[NT];
  f32x4 acc[NT][8];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    m[nt] = -INFINITY;
    l[nt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) acc[nt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const int last_full = (L - a.q_len) / kPage;   // pages below this are fully visible to all rows

  for (int k = k0; k < k1; k += 2) {
    const int pA = fbt[k];
    const int pB = (k + 1 < k1) ? fbt[k + 1] : -1;
    const bool okA = pA >= 0 && (int64_t)pA < a.num_pages;
    const bool okB = pB >= 0 && (int64_t)pB < a.num_pages;

    // ---- loads: K tiles of both pages and V^T tiles of both pages ------------
    u32x4 kA[4], kB[4];
    u32x2 vA[8], vB[8];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      kA[kb] = okA ? load_k<KV>(a, pA, g, n, j, kb) : u32x4{0u, 0u, 0u, 0u};
      kB[kb] = okB ? load_k<KV>(a, pB, g, n, j, kb) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      vA[dt] = okA ? load_vt<KV>(a, pA, g, dt * 16 + n, j) : u32x2{0u, 0u};
      vB[dt] = okB ? load_vt<KV>(a, pB, g, dt * 16 + n, j) : u32x2{0u, 0u};
    }
    float kscA = a.scale_log2, kscB = a.scale_log2, vscA = 1.f, vscB = 1.f;
    if constexpr (KV == kFP8) {
      if (okA) { kscA *= a.kv_scales[2 * (size_t)pA]; vscA = a.kv_scales[2 * (size_t)pA + 1]; }
      if (okB) { kscB *= a.kv_scales[2 * (size_t)pB]; vscB = a.kv_scales[2 * (size_t)pB + 1]; }
    }

    // keys at or beyond L hold no data: zero their V so 0 * garbage cannot occur
    const bool tail = (k + 2) * kPage > L;
    if (tail) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bool zA = k * kPage + 4 * j + e >= L;
        const bool zB = (k + 1) * kPage + 4 * j + e >= L;
        const uint32_t mask = (e & 1) ? 0x0000ffffu : 0xffff0000u;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
          if (zA) vA[dt][e >> 1] &= mask;
          if (zB) vB[dt][e >> 1] &= mask;
        }
      }
    }

    // ---- S^T = K Q^T ------------------------------------------------------------
    f32x4 sA[NT], sB[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      sA[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
      sB[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        sA[nt] = mfma(kA[kb], qop[nt][kb], sA[nt]);
        sB[nt] = mfma(kB[kb], qop[nt][kb], sB[nt]);
      }
    }

    const bool needs_mask = !okA || !okB || (k + 2) > last_full;
    u32x4 phi[NT], plo[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      float z[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        z[e] = sA[nt][e] * kscA;
        z[4 + e] = sB[nt][e] * kscB;
      }
      if (needs_mask) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int posA = k * kPage + 4 * j + e;
          const int posB = (k + 1) * kPage + 4 * j + e;
          if (!okA || posA >= lim[nt]) z[e] = -INFINITY;
          if (!okB || posB >= lim[nt]) z[4 + e] = -INFINITY;
        }
      }
      float mx = z[0];
#pragma unroll
      for (int e = 1; e < 8; ++e) mx = fmaxf(mx, z[e]);
      mx = xor16_max(mx);
      mx = xor32_max(mx);
      const float m_new = fmaxf(m[nt], mx);
      const float mref = (m_new == -INFINITY) ? 0.f : m_new;
      if (m_new > m[nt]) {
        const float alpha = exp2f(m[nt] - mref);
        l[nt] *= alpha;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) acc[nt][dt] *= alpha;
        m[nt] = m_new;
      }
      float ps = 0.f;
      uint32_t hb[8], lb[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float p = exp2f(z[e] - mref);
        ps += p;
        const float pv = p * (e < 4 ? vscA : vscB);
        const uint32_t hbits = f32_to_bf16_rne(pv);
        hb[e] = hbits;
        lb[e] = f32_to_bf16_rne(pv - __uint_as_float(hbits << 16));
      }
      l[nt] += ps;
      phi[nt] = u32x4{hb[0] | (hb[1] << 16), hb[2] | (hb[3] << 16), hb[4] | (hb[5] << 16),
                      hb[6] | (hb[7] << 16)};
      plo[nt] = u32x4{lb[0] | (lb[1] << 16), lb[2] | (lb[3] << 16), lb[4] | (lb[5] << 16),
                      lb[6] | (lb[7] << 16)};
    }

    // ---- O^T += V^T P^T -----------------------------------------------------------
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      const u32x4 vop = u32x4{vA[dt][0], vA[dt][1], vB[dt][0], vB[dt][1]};
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        acc[nt][dt] = mfma(vop, phi[nt], acc[nt][dt]);
        acc[nt][dt] = mfma(vop, plo[nt], acc[nt][dt]);
      }
    }
  }

  // ---- write the (partial) result ---------------------------------------------------
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    float lt = xor16_sum(l[nt]);
    lt = xor32_sum(lt);
    const int r = nt * 16 + n;
    if (r >= R) continue;
    const int i = r >> 2, hh = r & 3;
    const size_t row = ((size_t)b * a.q_len + i) * a.Hq + g * 4 + hh;
    const bool empty = (m[nt] == -INFINITY);
    const float inv = empty ? 0.f : 1.f / lt;
    const float lse2 = empty ? -INFINITY : m[nt] + log2f(lt);
    float *dst = (a.n_split == 1) ? a.out + row * kD
                                  : a.part_o + (row * a.n_split + split) * kD;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      const f32x4 o = acc[nt][dt] * inv;
      *reinterpret_cast<f32x4 *>(dst + dt * 16 + 4 * j) = o;
    }
    if (j == 0) {
      if (a.n_split == 1) a.lse[row] = lse2 * kLn2;
      else a.part_lse[row * a.n_split + split] = lse2;
    }
  }
}

template <int KV>
hipError_t launch_kv(const AttnArgs &a, hipStream_t s) {
  const dim3 grid(a.n_split, a.Hkv, a.batch);
  const int nt = (a.q_len * 4 + 15) / 16;
  switch (nt) {
    case 1: hipLaunchKernelGGL((verify_mfma_kernel<KV, 1>), grid, dim3(64), 0, s, a); break;
    case 2: hipLaunchKernelGGL((verify_mfma_kernel<KV, 2>), grid, dim3(64), 0, s, a); break;
    case 3: hipLaunchKernelGGL((verify_mfma_kernel<KV, 3>), grid, dim3(64), 0, s, a); break;
    case 4: hipLaunchKernelGGL((verify_mfma_kernel<KV, 4>), grid, dim3(64), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_verify_mfma(const AttnArgs &a, hipStream_t s) {
  if (a.kv_type == kBF16) return launch_kv<kBF16>(a, s);
  if (a.kv_type == kFP8) return launch_kv<kFP8>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace kap

// Full-KV verification attention on the matrix cores (Sec. 3.2 of the paper,
// "Full-context verification"; Eq. (2)) for bf16 / fp8 KV, head_dim 128, four
// query heads per KV head, window q_len <= 16.
//
// The q_len window tokens times the four heads of one KV head form
// R = 4 * q_len query rows that share every key: a real dense contraction.
// A workgroup of four wavefronts owns (key split, KV head, sequence); each
// wavefront walks its share of the split two pages (32 keys) at a time, with
// the following page pairs' loads in flight (branch-free, so only the oldest
// buffer is waited for), using v_mfma_f32_16x16x32_bf16:
//   S^T[key][row] = K[key][:] . Q[row][:]       A = K tile (16 keys x 32 dims,
//                                               one 16-byte load per lane; K
//                                               pages in 8-dim chunks make it
//                                               1 KB contiguous per load),
//                                               B = Q^T (kept in registers)
//   O^T[dim][row] += V^T[dim][key] P^T[key][row] A = V^T tile (dim-major pages:
//                                               4 keys = 8 contiguous bytes),
//                                               B = P^T, which the S^T
//                                               accumulator layout already
//                                               holds lane for lane.
// Lane (j = lane/16, n = lane%16) thus owns query row n of each 16-row tile and
// keys 4j..4j+3 of both pages, so the online softmax needs only two cross-row
// steps per page pair. P is split into bf16 hi + lo parts (two PV products):
// hi = P truncated to bf16, lo = P - hi (exact in fp32) truncated to bf16,
// which keeps the probability rounding error below 2^-14 relative.
// The causal mask and the partial last page are handled on the last pages only.
// When the last row tile holds a single window token (q_len = 4 t + 1), its
// softmax runs on that token's 4 rows gathered into all 64 lanes rather than
// on 16 rows of which 12 are padding, and its hi and lo weights share one PV
// product (columns 0-3 and 4-7 of the operand) (the C4 kernel instances).
// The four wavefronts combine through LDS; with several splits, the workgroup
// that finishes last for its (sequence, KV head) merges all splits (atomic
// arrival counter in the workspace), so one launch produces the final output.
#include <type_traits>

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
  return max_f(__int_as_float(r[0]), __int_as_float(r[1]));
}
__device__ __forceinline__ float xor32_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_int(x), __float_as_int(x), false, false);
  return max_f(__int_as_float(r[0]), __int_as_float(r[1]));
}
__device__ __forceinline__ float xor16_sum(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_int(x), __float_as_int(x), false, false);
  return __int_as_float(r[0]) + __int_as_float(r[1]);
}
__device__ __forceinline__ float xor32_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_int(x), __float_as_int(x), false, false);
  return __int_as_float(r[0]) + __int_as_float(r[1]);
}

// Moves within each 16-lane row (DPP): lane i of a row reads lane i - N
// (row_shr), i + N (row_shl) or (i - N) mod 16 (row_ror) of the same row.
constexpr int kRowShl(int n) { return 0x100 + n; }
constexpr int kRowShr(int n) { return 0x110 + n; }
constexpr int kRowRor(int n) { return 0x120 + n; }
// src moved by CTRL into the lanes of the 4-lane banks set in BANKS (bank b =
// lanes 4b .. 4b + 3 of every row); the other lanes keep old
template <int CTRL, int BANKS>
__device__ __forceinline__ float dpp_into(float old, float src) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(src), CTRL,
                                                    0xF, BANKS, false));
}
template <int CTRL, int BANKS>
__device__ __forceinline__ uint32_t dpp_into(uint32_t old, uint32_t src) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)src, CTRL, 0xF, BANKS, false);
}
// x moved by CTRL in every lane; a lane whose source lies outside its row reads 0
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_all(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, true);
}
template <int CTRL>
__device__ __forceinline__ float dpp_all(float x) {
  return __uint_as_float(dpp_all<CTRL>(__float_as_uint(x)));
}

__device__ __forceinline__ uint32_t pack_bf16_exact(float lo, float hi) {
  return __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), 0x07060302u);
}

constexpr int kTileBytes(int kv) { return (kv == kBF16 ? 2 : 1) * kPage * kD; }

// Raw registers of one page pair (pages k, k+1 of the sequence) as loaded:
// bf16 operands, or fp8 codes that are widened only where they are used (a
// conversion next to the load would make the load wait at once).
template <int KV> struct PairData;
template <> struct PairData<kBF16> {
  u32x4 kA[4], kB[4];   // K operand: key n, dims 32kb + 8j .. +7 (8 bf16)
  u32x2 vA[8], vB[8];   // V^T operand half: dim 16dt + n, keys 4j .. 4j+3 (4 bf16)
};
template <> struct PairData<kFP8> {
  u32x2 kA[4], kB[4];   // the same elements as fp8 codes
  u32x4 vA[2], vB[2];   // V^T rows 64 c + lane (all 16 keys), rearranged at use (vt_tiles)
  float2 scA, scB;      // (K, V) scales of the two pages
};
template <int KV>
struct PairRegs : PairData<KV> {
  int pA, pB;
  bool okA, okB;
};

// K tile operand of one page for k-block kb: key n, dims 32kb + 8j .. +7
// (chunk 4kb + j of the page's chunk-major K tile)
__device__ __forceinline__ u32x4 load_k(__amdgpu_buffer_rsrc_t r, int n, int j, int kb, u32x4) {
  return tile_load16(r, kb * 1024 + j * 256 + n * 16);
}
__device__ __forceinline__ u32x2 load_k(__amdgpu_buffer_rsrc_t r, int n, int j, int kb, u32x2) {
  return tile_load8(r, kb * 512 + j * 128 + n * 8);
}
// V^T operand half: dim dt*16 + n, keys 4j .. 4j+3 of one page
__device__ __forceinline__ u32x2 load_vt(__amdgpu_buffer_rsrc_t r, int n, int j, int dt, u32x2) {
  return tile_load8(r, dt * 512 + n * 32 + j * 8);
}
// ... and as bf16 operands
__device__ __forceinline__ u32x4 k_operand(u32x4 x) { return x; }
__device__ __forceinline__ u32x4 k_operand(u32x2 x) {
  const u32x2 lo = fp8x4_to_bf16x4(x[0]), hi = fp8x4_to_bf16x4(x[1]);
  return u32x4{lo[0], lo[1], hi[0], hi[1]};
}
__device__ __forceinline__ u32x2 v_operand(u32x2 x) { return x; }
__device__ __forceinline__ u32x2 v_operand(uint32_t x) { return fp8x4_to_bf16x4(x); }

// fp8 V^T: the operand piece of lane (j, n) -- keys 4j .. 4j+3 of dim 16 dt + n
// -- is 4 bytes, and loading it directly puts lane 16 j + n at byte 16 n + 4 j:
// neighbouring lanes 16 bytes apart, which read at ~5.4-5.9 TB/s against ~6.8
// for the same bytes as whole rows (random-page read probes on MI355X). So each
// lane loads whole rows 64 c + lane (16 keys = 4 dwords) and the pieces are
// moved into place at use: row j of the wavefront holds dword w of tile
// 4 c + j and needs dword j of tiles 4 c .. 4 c + 3, a 4 x 4 dword transpose
// across the four 16-lane rows done by two rounds of row swaps.
__device__ __forceinline__ void swap_rows16(uint32_t &a, uint32_t &b) {
  const auto r = __builtin_amdgcn_permlane16_swap(a, b, false, false);
  a = r[0];
  b = r[1];
}
__device__ __forceinline__ void swap_rows32(uint32_t &a, uint32_t &b) {
  const auto r = __builtin_amdgcn_permlane32_swap(a, b, false, false);
  a = r[0];
  b = r[1];
}
__device__ __forceinline__ void vt_tiles(const u32x4 rows[2], uint32_t out[8]) {
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    uint32_t r0 = rows[c][0], r1 = rows[c][1], r2 = rows[c][2], r3 = rows[c][3];
    swap_rows16(r0, r1);
    swap_rows16(r2, r3);
    swap_rows32(r0, r2);
    swap_rows32(r1, r3);
    out[4 * c + 0] = r0;
    out[4 * c + 1] = r1;
    out[4 * c + 2] = r2;
    out[4 * c + 3] = r3;
  }
}

// Pair at pages k, k+1 (k + 1 may lie past the sequence) with physical ids
// pa, pb (pb < 0 if there is no page k + 1). Missing or invalid pages, and
// pairs past the wavefront's share (live == false), load through a zero-byte
// descriptor: zeros, no memory traffic, and no branches. The K half (page
// ids, K tiles, fp8 scales) and the V half (V tiles, from the page ids the K
// half set) can be issued at different times.
template <int KV>
__device__ __forceinline__ void load_pair_k(PairRegs<KV> &r, const AttnArgs &a, int pa, int pb,
                                            int g, int n, int j, bool live) {
  r.okA = live && pa >= 0 && (int64_t)pa < a.num_pages;
  r.okB = live && pb >= 0 && (int64_t)pb < a.num_pages;
  r.pA = r.okA ? pa : 0;
  r.pB = r.okB ? pb : 0;
  const size_t tile = kTileBytes(KV);
  const int ba = r.okA ? (int)tile : 0, bb = r.okB ? (int)tile : 0;
  const auto kra = tile_rsrc(a.k_pages, ((size_t)r.pA * a.Hkv + g) * tile, ba);
  const auto krb = tile_rsrc(a.k_pages, ((size_t)r.pB * a.Hkv + g) * tile, bb);
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    r.kA[kb] = load_k(kra, n, j, kb, r.kA[kb]);
    r.kB[kb] = load_k(krb, n, j, kb, r.kB[kb]);
  }
  if constexpr (KV == kFP8) {
    r.scA = page_scales(a.kv_scales, r.pA, r.okA);
    r.scB = page_scales(a.kv_scales, r.pB, r.okB);
  }
}
template <int KV>
__device__ __forceinline__ void load_pair_v(PairRegs<KV> &r, const AttnArgs &a, int g, int n,
                                            int j) {
  const size_t tile = kTileBytes(KV);
  const int ba = r.okA ? (int)tile : 0, bb = r.okB ? (int)tile : 0;
  const auto vra = tile_rsrc(a.v_pages, ((size_t)r.pA * a.Hkv + g) * tile, ba);
  const auto vrb = tile_rsrc(a.v_pages, ((size_t)r.pB * a.Hkv + g) * tile, bb);
  if constexpr (KV == kBF16) {
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      r.vA[dt] = load_vt(vra, n, j, dt, r.vA[dt]);
      r.vB[dt] = load_vt(vrb, n, j, dt, r.vB[dt]);
    }
  } else {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      r.vA[c] = tile_load16(vra, c * 1024 + (16 * j + n) * 16);
      r.vB[c] = tile_load16(vrb, c * 1024 + (16 * j + n) * 16);
    }
  }
}
template <int KV>
__device__ __forceinline__ void load_pair(PairRegs<KV> &r, const AttnArgs &a, int pa, int pb,
                                          int g, int n, int j, bool live) {
  load_pair_k<KV>(r, a, pa, pb, g, n, j, live);
  load_pair_v<KV>(r, a, g, n, j);
}

constexpr int kVerifyWaves = 4;

// Wavefronts per SIMD the compiler must leave room for. fp8 windows of 5-12
// tokens (two or three row tiles) are issue-bound at one wavefront per SIMD:
// their widening and softmax instructions wait behind their own matrix
// products. Widening at use (and, with three tiles, one page pair in flight
// per wavefront) keeps them within 256 registers, so a second wavefront per
// SIMD fits without spills and overlaps the two (ragged fp8 verify on MI355X:
// 5-token windows 1014 vs 1114 us, 9-token windows 1254 vs 1374 us). bf16
// kernels and fp8 with four tiles would spill; fp8 with one tile already
// runs two per SIMD (asking for it explicitly cost 1%).
constexpr int verify_min_waves(int kv, int nt) { return kv == kFP8 && (nt == 2 || nt == 3) ? 2 : 1; }

// C4: the last row tile holds a single window token (q_len = 4 (NT - 1) + 1),
// i.e. 4 of its 16 rows are real. Its softmax then runs on the 4 x 32 logits
// gathered into all 64 lanes (two per lane) instead of on all 16 rows, which
// removes about 30 vector instructions per page pair and KV head; the
// weights return to the P^T operand layout for the products.
template <int KV, int NT, bool C4>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(verify_min_waves(KV, NT))))
void verify_mfma_kernel(AttnArgs a) {
  __shared__ float s_acc[kVerifyWaves][16][kD + 4];
  __shared__ float s_m[kVerifyWaves][16];
  __shared__ float s_l[kVerifyWaves][16];
  __shared__ int s_flag;
  // Where the combined tiles go: every thread stores its own slice, except in
  // the three-tile fp8 kernel for 10-12-token windows, which stages each tile
  // in LDS for wavefront 0 to store -- at 256 registers there, storing from
  // every thread moved spills into its page loop (ragged fp8 11-token windows
  // 957 vs 1250 us on MI355X).
  constexpr bool kStagedStore = KV == kFP8 && NT == 3 && !C4;
  __shared__ float s_out[kStagedStore ? 16 : 1][kD];
  __shared__ float s_olse[16];

  WorkItem wi;
  int L;
  if (a.ragged) {
    auto load = [&](int bb) {
      const int Lb = a.seq_lens[bb];
      const int np = Lb > 0 ? min((int)(((long long)Lb + kPage - 1) / kPage), a.max_blocks) : 0;
      return SeqLoad{(np + 1) / 2, Lb};
    };
    int pairs_b;
    const SeqLoad first = map_first_loads(a, load);
    if (!ragged_map(a, load, first, blockIdx.x, wi, pairs_b, L)) return;
  } else {
    wi.split = blockIdx.x;
    wi.g = blockIdx.y;
    wi.b = blockIdx.z;
    wi.n_split = a.n_split;
    wi.slot0 = (blockIdx.z * a.Hkv + blockIdx.y) * a.n_split;
    L = a.seq_lens[wi.b];
  }
  // The work item is the same in every lane; saying so keeps it in scalar
  // registers (the balanced map divides in double precision, whose results
  // live in vector registers, and a block-table or descriptor address built
  // from one made the compiler loop over the lanes around every page load).
  wi.split = __builtin_amdgcn_readfirstlane(wi.split);
  wi.g = __builtin_amdgcn_readfirstlane(wi.g);
  wi.b = __builtin_amdgcn_readfirstlane(wi.b);
  wi.n_split = __builtin_amdgcn_readfirstlane(wi.n_split);
  wi.slot0 = __builtin_amdgcn_readfirstlane(wi.slot0);
  const int split = wi.split, g = wi.g, b = wi.b, n_split = wi.n_split;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int n = lane & 15, j = lane >> 4;
  const int R = a.q_len * 4;

  int np_seq = L > 0 ? (int)(((long long)L + kPage - 1) / kPage) : 0;
  np_seq = min(np_seq, a.max_blocks);
  // split `split` of n_split takes an even share of this sequence's page pairs;
  // its four wavefronts take those pairs round-robin
  const int pairs = (np_seq + 1) / 2;
  const int q0 = (int)(((long long)split * pairs) / n_split);
  const int q1 = (int)(((long long)(split + 1) * pairs) / n_split);
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
  // C4 tile: rows 16 (NT - 1) .. + 3 are the four heads of window token
  // 4 (NT - 1), which sees logical positions below lim_c4
  const int lim_c4 = L - a.q_len + 4 * (NT - 1) + 1;

  // RING pair buffers (windows of up to 8 tokens: two -- three were 0.2-0.5%
  // slower for bf16 on MI355X, e.g. 333.0 vs 331.9 us at 128K; 9..12-token
  // windows: bf16 two, fp8 one at two wavefronts per SIMD; 13..16-token
  // windows: bf16 one (two spill: 478 vs 334 us at 4 x 128K), fp8 two (321 vs
  // 353 us)),
  // unrolled: while one pair is processed the loads of the next ones are in
  // flight. Past the end of this wavefront's pairs the loads go through an
  // empty descriptor (no traffic), so the steady state is straight-line code.
  // next_k / next_v issue the loads of the wavefront's next pair into the
  // registers of P as soon as this pair no longer needs them: the K half
  // (with the fp8 scales) once the logits are computed, the V half once V
  // has been taken out of them. With one pair buffer per wavefront this
  // keeps the next pair's loads in flight during most of this pair's work.
  auto process = [&](PairRegs<KV> &P, int k, auto &&next_k, auto &&next_v) {
    float kscA = a.scale_log2, kscB = a.scale_log2, vscA = 1.f, vscB = 1.f;
    if constexpr (KV == kFP8) {
      kscA *= P.scA.x;
      vscA = P.scA.y;
      kscB *= P.scB.x;
      vscB = P.scB.y;
    }
    const bool okA = P.okA, okB = P.okB;
    // V^T pieces of lane (j, n): keys 4j .. 4j+3 of dims 16 dt + n, raw. bf16
    // takes them from the registers here; fp8 rearranges them after the
    // softmax, which frees the raw registers for the next pair's V loads.
    using VPiece = typename std::conditional<KV == kBF16, u32x2, uint32_t>::type;
    VPiece vA[8], vB[8];
    // keys at or beyond L hold no data: zero their V so 0 * garbage cannot
    // occur (on the raw registers: bytes of fp8 codes, halves of bf16 pairs)
    auto zero_past_end = [&] {
      if ((k + 2) * kPage > L) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bool zA = k * kPage + 4 * j + e >= L;
          const bool zB = (k + 1) * kPage + 4 * j + e >= L;
#pragma unroll
          for (int dt = 0; dt < 8; ++dt) {
            if constexpr (KV == kFP8) {
              const uint32_t mask = ~(0xFFu << (8 * e));
              if (zA) vA[dt] &= mask;
              if (zB) vB[dt] &= mask;
            } else {
              const uint32_t mask = (e & 1) ? 0x0000ffffu : 0xffff0000u;
              if (zA) vA[dt][e >> 1] &= mask;
              if (zB) vB[dt][e >> 1] &= mask;
            }
          }
        }
      }
    };
    if constexpr (KV == kBF16) {
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        vA[dt] = P.vA[dt];
        vB[dt] = P.vB[dt];
      }
      zero_past_end();
    }

    // ---- S^T = K Q^T (K operands widened at use) ---------------------------------
    f32x4 sA[NT], sB[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      sA[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
      sB[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const u32x4 kA = k_operand(P.kA[kb]), kB = k_operand(P.kB[kb]);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        sA[nt] = mfma(kA, qop[nt][kb], sA[nt]);
        sB[nt] = mfma(kB, qop[nt][kb], sB[nt]);
      }
    }
    next_k();

    const bool needs_mask = !okA || !okB || (k + 2) > last_full;
    u32x4 phi[NT], plo[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      if constexpr (C4) {
        if (nt == NT - 1) {
          // Lane (j, n < 4) holds row n's keys 4j .. 4j+3 of both pages. Gather
          // them into lane 16 j + 4 c + n: c = 0, 1 take keys 4j + 2c, + 1 of
          // page A; c = 2, 3 keys 4j + 2(c - 2), + 1 of page B. Row n's 32
          // logits then sit two per lane in the 16 lanes with lane % 4 = n.
          float c0 = sA[nt][0], c1 = sA[nt][1];
          c0 = dpp_into<kRowShr(4), 0x2>(c0, sA[nt][2]);
          c1 = dpp_into<kRowShr(4), 0x2>(c1, sA[nt][3]);
          c0 = dpp_into<kRowShr(8), 0x4>(c0, sB[nt][0]);
          c1 = dpp_into<kRowShr(8), 0x4>(c1, sB[nt][1]);
          c0 = dpp_into<kRowShr(12), 0x8>(c0, sB[nt][2]);
          c1 = dpp_into<kRowShr(12), 0x8>(c1, sB[nt][3]);
          const bool onB = (lane & 8) != 0;
          const float ksc = onB ? kscB : kscA;
          float z0 = c0 * ksc, z1 = c1 * ksc;
          if (needs_mask) {
            const int pos = (k + (onB ? 1 : 0)) * kPage + 4 * j + 2 * ((lane >> 2) & 1);
            const bool ok = onB ? okB : okA;
            if (!ok || pos >= lim_c4) z0 = -INFINITY;
            if (!ok || pos + 1 >= lim_c4) z1 = -INFINITY;
          }
          float mx = max_f(z0, z1);
          mx = max_f(mx, dpp_all<kRowRor(4)>(mx));
          mx = max_f(mx, dpp_all<kRowRor(8)>(mx));
          mx = xor16_max(mx);
          mx = xor32_max(mx);
          // every lane now holds the running state of row lane % 4, which
          // for the accumulator lanes (j, n < 4) is their own row
          const float m_new = max_f(m[nt], mx);
          const float mref = (m_new == -INFINITY) ? 0.f : m_new;
          if (m_new > m[nt]) {
            const float alpha = exp2_fast(m[nt] - mref);
            l[nt] *= alpha;
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) acc[nt][dt] *= alpha;
            m[nt] = m_new;
          }
          const float p0 = exp2_fast(z0 - mref), p1 = exp2_fast(z1 - mref);
          l[nt] += p0 + p1;
          const float vsc = onB ? vscB : vscA;
          const float pv0 = p0 * vsc, pv1 = p1 * vsc;
          const float pl0 = pv0 - __uint_as_float(__float_as_uint(pv0) & 0xffff0000u);
          const float pl1 = pv1 - __uint_as_float(__float_as_uint(pv1) & 0xffff0000u);
          const uint32_t h = pack_bf16_exact(pv0, pv1), lw = pack_bf16_exact(pl0, pl1);
          // Back to the P^T operand, with the hi and lo weights side by side
          // so that one product per V tile takes both: column n < 4 (lane
          // (j, n)) gets row n's hi pieces, from lanes 16 j + 4 c + n, c = 0..3;
          // column 4 + n gets row n's lo pieces from the same lanes. The two
          // column groups are added when the wavefronts combine.
          phi[nt] = u32x4{dpp_into<kRowShr(4), 0x2>(h, lw), dpp_into<kRowShl(4), 0x1>(lw, h),
                          dpp_into<kRowShl(4), 0x2>(dpp_all<kRowShl(8)>(h), lw),
                          dpp_into<kRowShl(8), 0x2>(dpp_all<kRowShl(12)>(h), lw)};
          continue;
        }
      }
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
      for (int e = 1; e < 8; ++e) mx = max_f(mx, z[e]);
      mx = xor16_max(mx);
      mx = xor32_max(mx);
      const float m_new = max_f(m[nt], mx);
      const float mref = (m_new == -INFINITY) ? 0.f : m_new;
      if (m_new > m[nt]) {
        const float alpha = exp2_fast(m[nt] - mref);
        l[nt] *= alpha;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) acc[nt][dt] *= alpha;
        m[nt] = m_new;
      }
      float ps = 0.f;
      float pv[8], pl[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float p = exp2_fast(z[e] - mref);
        ps += p;
        pv[e] = p * (e < 4 ? vscA : vscB);
        pl[e] = pv[e] - __uint_as_float(__float_as_uint(pv[e]) & 0xffff0000u);
      }
      l[nt] += ps;
      // bf16 pairs are the upper halves of the floats (truncation)
      phi[nt] = u32x4{pack_bf16_exact(pv[0], pv[1]), pack_bf16_exact(pv[2], pv[3]),
                      pack_bf16_exact(pv[4], pv[5]), pack_bf16_exact(pv[6], pv[7])};
      plo[nt] = u32x4{pack_bf16_exact(pl[0], pl[1]), pack_bf16_exact(pl[2], pl[3]),
                      pack_bf16_exact(pl[4], pl[5]), pack_bf16_exact(pl[6], pl[7])};
    }

    if constexpr (KV == kFP8) {
      vt_tiles(P.vA, vA);
      vt_tiles(P.vB, vB);
      next_v();
      zero_past_end();
    }
    // ---- O^T += V^T P^T -----------------------------------------------------------
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      const u32x2 va = v_operand(vA[dt]), vb = v_operand(vB[dt]);
      const u32x4 vop = u32x4{va[0], va[1], vb[0], vb[1]};
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        acc[nt][dt] = mfma(vop, phi[nt], acc[nt][dt]);
        if (!(C4 && nt == NT - 1)) acc[nt][dt] = mfma(vop, plo[nt], acc[nt][dt]);
      }
    }
    if constexpr (KV == kBF16) next_v();
  };

  const int qw = q0 + wave;
  const int n_my = qw < q1 ? (q1 - qw + kVerifyWaves - 1) / kVerifyWaves : 0;
  if (n_my > 0) {
    auto kpair = [&](int i) { return 2 * (qw + kVerifyWaves * min(i, n_my - 1)); };
    // Every round issues all RING loads unconditionally and skips only the
    // processing of pairs past the end: an early exit inside a round would
    // make the loop header wait for the just-issued loads, draining the ring
    // every round. The block-table entries of the pair a round ahead are read
    // through the vector memory pipe (lanes 0 and 1: pages k and k + 1) right
    // after a slot's pair loads, and used when the slot is refilled next.
    constexpr int RING = NT <= 2 ? 2 : (NT == 3 ? (KV == kBF16 ? 2 : 1) : (KV == kFP8 ? 2 : 1));
    const auto rt = table_rsrc(fbt, np_seq);
    const int voff = (lane & 1) * 4;
    auto second = [&](int k, int v) { return k + 1 < np_seq ? v : -1; };
    PairRegs<KV> rr[RING];
    int ahead[RING];
#pragma unroll
    for (int jr = 0; jr < RING; ++jr) {
      const int k = kpair(jr);
      load_pair<KV>(rr[jr], a, fbt[k], k + 1 < np_seq ? fbt[k + 1] : -1, g, n, j, jr < n_my);
      __builtin_amdgcn_sched_barrier(0);
      ahead[jr] = table_ahead(rt, voff, kpair(jr + RING));
      __builtin_amdgcn_sched_barrier(0);
    }
    auto none = [] {};
    if constexpr (RING == 1 && KV == kFP8) {
      // one buffer: the next pair's K and V halves are issued inside process
      for (int i = 0; i < n_my; ++i) {
        const int k = kpair(i + 1);
        const int pa = lane_value(ahead[0], 0), pb = second(k, lane_value(ahead[0], 1));
        process(
            rr[0], kpair(i),
            [&] { load_pair_k<KV>(rr[0], a, pa, pb, g, n, j, i + 1 < n_my); },
            [&] {
              load_pair_v<KV>(rr[0], a, g, n, j);
              ahead[0] = table_ahead(rt, voff, kpair(i + 2));
            });
      }
    } else {
      for (int i = 0; i < n_my; i += RING) {
#pragma unroll
        for (int jr = 0; jr < RING; ++jr) {
          if (i + jr < n_my) process(rr[jr], kpair(i + jr), none, none);
          const int k = kpair(i + jr + RING);
          load_pair<KV>(rr[jr], a, lane_value(ahead[jr], 0), second(k, lane_value(ahead[jr], 1)),
                        g, n, j, i + jr + RING < n_my);
          ahead[jr] = table_ahead(rt, voff, kpair(i + jr + 2 * RING));
        }
      }
    }
  }

  // ---- combine the four wavefronts, tile by tile, then write ----------------------
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    float lt = l[nt];
    if (C4 && nt == NT - 1) {   // the gathered tile's sums are spread over lane bits 2, 3 too
      lt += dpp_all<kRowRor(4)>(lt);
      lt += dpp_all<kRowRor(8)>(lt);
    }
    lt = xor16_sum(lt);
    lt = xor32_sum(lt);
    if (C4 && nt == NT - 1) {   // the gathered tile: row n's lo part sits in column 4 + n
#pragma unroll
      for (int dt = 0; dt < 8; ++dt)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[nt][dt][e] += dpp_all<kRowShl(4)>(acc[nt][dt][e]);
    }
#pragma unroll
    for (int dt = 0; dt < 8; ++dt)
      *reinterpret_cast<f32x4 *>(&s_acc[wave][n][dt * 16 + 4 * j]) = acc[nt][dt];
    if (j == 0) {
      s_m[wave][n] = m[nt];
      s_l[wave][n] = lt;
    }
    __syncthreads();
    // thread (rn, d8) combines row rn's dims d8 .. d8 + 7
    const int rn = threadIdx.x >> 4;            // row of the tile
    const int d8 = (threadIdx.x & 15) * 8;      // 8 dims
    const int r = nt * 16 + rn;
    float o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = 0.f;
    float lse2 = -INFINITY;
    if (r < R) {
      float M = -INFINITY;
#pragma unroll
      for (int w = 0; w < kVerifyWaves; ++w) M = fmaxf(M, s_m[w][rn]);
      if (M != -INFINITY) {
        float den = 0.f;
#pragma unroll
        for (int w = 0; w < kVerifyWaves; ++w) {
          const float ew = exp2f(s_m[w][rn] - M);
          den = fmaf(ew, s_l[w][rn], den);
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = fmaf(ew, s_acc[w][rn][d8 + e], o[e]);
        }
        const float inv = 1.f / den;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] *= inv;
        lse2 = M + log2f(den);
      }
    }
    const float4 v0 = make_float4(o[0], o[1], o[2], o[3]);
    const float4 v1 = make_float4(o[4], o[5], o[6], o[7]);
    if constexpr (kStagedStore) {
      // staged in LDS; wavefront 0 writes the tile
      *reinterpret_cast<float4 *>(&s_out[rn][d8]) = v0;
      *reinterpret_cast<float4 *>(&s_out[rn][d8 + 4]) = v1;
      if (d8 == 0) s_olse[rn] = lse2;
      __syncthreads();
      if (threadIdx.x < 64) {
        const auto ro = partial_rsrc(a.part_o);
        const auto rl = partial_rsrc(a.part_lse);
#pragma unroll
        for (int t8 = 0; t8 < 8; ++t8) {
          const int f = threadIdx.x + 64 * t8;      // float4 index in [16][128]
          const int rr = f >> 5, d4 = (f & 31) * 4;
          const int rw = nt * 16 + rr;
          if (rw < R) {
            const size_t row = out_row(a, b, g, rw);
            const float4 v = *reinterpret_cast<const float4 *>(&s_out[rr][d4]);
            if (n_split == 1)
              *reinterpret_cast<float4 *>(a.out + row * kD + d4) = v;
            else
              partial_store4(ro, (((size_t)(wi.slot0 + split) * R + rw) * kD + d4) * 4, v);
          }
        }
        if (threadIdx.x < 16 && nt * 16 + threadIdx.x < R) {
          const size_t row = out_row(a, b, g, nt * 16 + threadIdx.x);
          if (n_split == 1) a.lse[row] = s_olse[threadIdx.x] * kLn2;
          else partial_store1(rl, ((size_t)(wi.slot0 + split) * R + nt * 16 + threadIdx.x) * 4,
                              s_olse[threadIdx.x]);
        }
      }
      __syncthreads();
    } else {
      // each thread writes its slice: the final output, or its part of this
      // split's partial
      if (r < R) {
        if (n_split == 1) {
          const size_t row = out_row(a, b, g, r);
          *reinterpret_cast<float4 *>(a.out + row * kD + d8) = v0;
          *reinterpret_cast<float4 *>(a.out + row * kD + d8 + 4) = v1;
          if (d8 == 0) a.lse[row] = lse2 * kLn2;
        } else {
          const size_t pr = (size_t)(wi.slot0 + split) * R + r;
          const auto ro = partial_rsrc(a.part_o);
          partial_store4(ro, (pr * kD + d8) * 4, v0);
          partial_store4(ro, (pr * kD + d8 + 4) * 4, v1);
          if (d8 == 0) partial_store1(partial_rsrc(a.part_lse), pr * 4, lse2);
        }
      }
      if (nt + 1 < NT) __syncthreads();   // the next tile reuses s_acc, s_m, s_l
    }
  }

  // ---- the last workgroup of (b, g) merges the splits ---------------------------------
  if (n_split > 1 && (kStagedStore ? last_arrival(a, b, g, n_split, &s_flag)
                                    : last_arrival_all(a, b, g, n_split, &s_flag)))
    merge_rows<3>(a, b, g, R, wi.slot0, n_split);
}

// q_len -> row tiles, and whether the last tile holds a single window token
constexpr bool c4_window(int q_len) { return q_len % 4 == 1; }

template <int KV, int NT>
void launch_nt(const AttnArgs &a, dim3 grid, hipStream_t s) {
  if (c4_window(a.q_len))
    hipLaunchKernelGGL((verify_mfma_kernel<KV, NT, true>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((verify_mfma_kernel<KV, NT, false>), grid, dim3(256), 0, s, a);
}

template <int KV>
hipError_t launch_kv(const AttnArgs &a, hipStream_t s) {
  const dim3 grid = a.ragged ? dim3(a.n_split) : dim3(a.n_split, a.Hkv, a.batch);
  const int nt = (a.q_len * 4 + 15) / 16;
  switch (nt) {
    case 1: launch_nt<KV, 1>(a, grid, s); break;
    case 2: launch_nt<KV, 2>(a, grid, s); break;
    case 3: launch_nt<KV, 3>(a, grid, s); break;
    case 4: launch_nt<KV, 4>(a, grid, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int KV, int NT>
hipError_t occupancy_nt(int *nb, bool c4) {
  return c4 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(nb, verify_mfma_kernel<KV, NT, true>, 256, 0)
            : hipOccupancyMaxActiveBlocksPerMultiprocessor(nb, verify_mfma_kernel<KV, NT, false>, 256, 0);
}

template <int KV>
int blocks_kv(int nt, bool c4) {
  int nb = 0;
  hipError_t e = hipErrorInvalidValue;
  switch (nt) {
    case 1: e = occupancy_nt<KV, 1>(&nb, c4); break;
    case 2: e = occupancy_nt<KV, 2>(&nb, c4); break;
    case 3: e = occupancy_nt<KV, 3>(&nb, c4); break;
    case 4: e = occupancy_nt<KV, 4>(&nb, c4); break;
    default: break;
  }
  return e == hipSuccess ? nb : 0;
}

}  // namespace

hipError_t launch_verify_mfma(const AttnArgs &a, hipStream_t s) {
  if (a.kv_type == kBF16) return launch_kv<kBF16>(a, s);
  if (a.kv_type == kFP8) return launch_kv<kFP8>(a, s);
  return hipErrorInvalidValue;
}

int verify_mfma_blocks_per_cu(int kv_type, int q_len) {
  const int nt = (q_len * 4 + 15) / 16;
  const bool c4 = c4_window(q_len);
  return kv_type == kFP8 ? blocks_kv<kFP8>(nt, c4) : blocks_kv<kBF16>(nt, c4);
}

}  // namespace kap

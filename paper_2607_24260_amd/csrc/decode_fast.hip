// Selected-view decode (q_prop = 1) for bf16 / fp8 KV, head_dim 128, four
// query heads per KV head -- the proposal step of Sec. 3.2 of the paper.
//
// Work decomposition: one 256-thread workgroup per (key split, KV head,
// sequence). The 4 n wavefronts of the n splits of (sequence, KV head) take the
// view's nb entries round-robin (an even share of the actual view), keep the
// next pages' loads in flight while one is processed, keep their own
// online-softmax state, and merge through LDS at the end of the workgroup. With more than one
// split the workgroup writes a partial (o, lse); the workgroup that finishes
// last for its (sequence, KV head) merges all splits (atomic arrival counter
// in the workspace), so one launch produces the final output.
//
// Per page (16 tokens x 128 dims = 4 KB of bf16 K and 4 KB of V^T):
//  * K phase: lane (t = lane/4, c = lane%4) loads dims {32i + 8c .. +7}, i<4,
//    of token t: four 16-byte loads, and since K pages are stored in 8-dim
//    chunks ([chunk][token][8]) each instruction reads 1 KB contiguously. It
//    forms partial dot products for the four query heads with v_dot2_f32_bf16. A transposing reduction inside each
//    lane quad leaves lane (t, c) holding the full logit of token t, head c.
//  * softmax: page maxima per head come from row rotations plus permlane16 /
//    permlane32 swaps; the running max, rescale factor and sum are kept per
//    head in every lane that owns that head.
//  * V phase: the V^T page is read as four contiguous 1 KB rows of 16-byte
//    loads; lane owns dims {32i + lane/2} for tokens 8*(lane%2) .. +7, takes
//    the probabilities of those tokens from LDS and accumulates o in fp32.
// Everything is memory-bound: 4 flop per KV byte against a VALU ridge of
// ~20 flop/byte, so no matrix cores are used here.
#include "kap_internal.h"

namespace kap {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kD = 128;
constexpr int kWaves = 4;
// pages in flight per wavefront (register ring depth). Two beat three and
// four on MI355X for both dtypes (128K workload: 24.6 vs 24.9 / 26.9 us per
// call; ragged fp8 full context: 959 vs 981 / 969 us): a deeper ring does not
// raise the read rate and costs registers and loop overhead.
#ifndef KAP_DECODE_RING_BF16
#define KAP_DECODE_RING_BF16 2
#endif
#ifndef KAP_DECODE_RING_FP8
#define KAP_DECODE_RING_FP8 2
#endif
constexpr int kRingBF16 = KAP_DECODE_RING_BF16;
constexpr int kRingFP8 = KAP_DECODE_RING_FP8;

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a),
                                         __builtin_bit_cast(bf16x2, b), c, false);
}

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, true));
}
constexpr int kQuadXor1 = 0xB1;  // quad_perm [1,0,3,2]
constexpr int kQuadXor2 = 0x4E;  // quad_perm [2,3,0,1]
constexpr int kRowRor4 = 0x124;
constexpr int kRowRor8 = 0x128;

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

// Raw registers of one page: K slice and V^T slice of this lane.
template <int KV> struct PageRegs;
template <> struct PageRegs<kBF16> { u32x4 k[4]; u32x4 v[4]; };
template <> struct PageRegs<kFP8> { u32x2 k[4]; u32x2 v[4]; float2 sc; };   // sc: (K, V) scales

// Loads of one (page, head) tile. With live == false the descriptor covers
// zero bytes: the loads return zeros without touching memory (used for
// invalid pages and for the ring's prefetches past a wavefront's last page).
template <int KV>
__device__ __forceinline__ void load_page(PageRegs<KV> &r, const AttnArgs &a, int page, int g,
                                          int lane, bool live) {
  const int t = lane >> 2, c = lane & 3;
  constexpr int kTile = (KV == kBF16 ? 2 : 1) * kPage * kD;   // bytes per (page, head) tile
  const size_t off = ((size_t)page * a.Hkv + g) * kTile;
  const int bytes = live ? kTile : 0;
  const auto kr = tile_rsrc(a.k_pages, off, bytes);
  const auto vr = tile_rsrc(a.v_pages, off, bytes);
  if constexpr (KV == kBF16) {
    // K: chunk 4i + c of token t; V^T: 1 KB row block i, 16 bytes per lane
#pragma unroll
    for (int i = 0; i < 4; ++i) r.k[i] = tile_load16(kr, i * 1024 + c * 256 + t * 16);
#pragma unroll
    for (int i = 0; i < 4; ++i) r.v[i] = tile_load16(vr, i * 1024 + lane * 16);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) r.k[i] = tile_load8(kr, i * 512 + c * 128 + t * 8);
#pragma unroll
    for (int i = 0; i < 4; ++i) r.v[i] = tile_load8(vr, i * 512 + lane * 8);
    r.sc = page_scales(a.kv_scales, page, live);
  }
}

// K slice of this lane as bf16 pairs: kk[i][w] holds dims 32i + 8c + 2w, +1.
template <int KV>
__device__ __forceinline__ void k_pairs(const PageRegs<KV> &r, uint32_t kk[4][4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if constexpr (KV == kBF16) {
#pragma unroll
      for (int w = 0; w < 4; ++w) kk[i][w] = r.k[i][w];
    } else {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const kv_u32x2 w = fp8x4_to_bf16x4(r.k[i][h]);
        kk[i][2 * h] = w[0];
        kk[i][2 * h + 1] = w[1];
      }
    }
  }
}

// V^T slice as floats: vv[i][j] = V[token 8*(lane%2) + j][dim 32i + lane/2].
template <int KV>
__device__ __forceinline__ void v_floats(const PageRegs<KV> &r, float vv[4][8]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if constexpr (KV == kBF16) {
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        vv[i][2 * w] = bf16_lo(r.v[i][w]);
        vv[i][2 * w + 1] = bf16_hi(r.v[i][w]);
      }
    } else {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float2 f0 = fp8x2_to_f32<false>(r.v[i][h]);
        const float2 f1 = fp8x2_to_f32<true>(r.v[i][h]);
        vv[i][4 * h + 0] = f0.x;
        vv[i][4 * h + 1] = f0.y;
        vv[i][4 * h + 2] = f1.x;
        vv[i][4 * h + 3] = f1.y;
      }
    }
  }
}

template <int KV, int RING, bool BALANCED, bool MASKED>
__global__ __launch_bounds__(256) void decode_fast_kernel(AttnArgs a) {
  __shared__ float pbuf[kWaves][64];
  __shared__ float wstat[2][kWaves][4];            // per-wave m (log2) and l per head
  __shared__ float wacc[kWaves][4][kD];
  __shared__ float s_part[4][kD];
  __shared__ float s_plse[4];
  __shared__ int s_flag;

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int t = lane >> 2, c = lane & 3, hf = lane & 1;

  // Work unit. Balanced mode: the map needs the view lengths of the whole
  // batch, so the first table entries are read for a guess while it is
  // computed -- the even assignment, a.guess_splits splits per unit, which
  // the map produces for equal views -- and read again if the map differs.
  WorkItem wi;
  if constexpr (BALANCED) {
    const int ng = a.guess_splits;
    const int w = blockIdx.x;
    const int q = div_small(w, ng);
    wi.n_split = ng;
    wi.split = w - q * ng;
    const int bq = div_small(q, a.Hkv);
    wi.g = q - bq * a.Hkv;
    wi.b = min(bq, a.batch - 1);
  } else {
    wi.split = blockIdx.x;
    wi.g = blockIdx.y;
    wi.b = blockIdx.z;
    wi.n_split = a.n_split;
    wi.slot0 = (blockIdx.z * a.Hkv + blockIdx.y) * a.n_split;
  }

  // The n_split * 4 wavefronts of (b, g) take the view's entries round-robin:
  // wavefront u = 4 * split + wave takes entries u, u + nw, u + 2 nw, ...
  // (an even share of the actual view, within one page). Table reads are
  // clamped to the row, not to the view, so they need not wait for the view
  // length. (With max_blocks == 0 the host points both tables at seq_lens
  // with row stride 0, so entry 0 of the row is always readable.)
  const int last_entry = max(a.max_blocks - 1, 0);
  int raw_pg[RING], raw_lb[RING];
  uint32_t raw_mk[RING];
  auto first_entries = [&](const WorkItem &x) {
    const int32_t *bt = a.block_table + (size_t)x.b * a.bt_stride;
    const int32_t *lb = a.logical_block + (size_t)x.b * a.bt_stride;
    const uint32_t *mk = MASKED ? a.token_mask + (size_t)x.b * a.bt_stride : nullptr;
#pragma unroll
    for (int j = 0; j < RING; ++j) {
      const int kk = min(x.split * kWaves + wave + x.n_split * kWaves * j, last_entry);
      raw_pg[j] = bt[kk];
      raw_lb[j] = lb[kk];
      raw_mk[j] = MASKED ? mk[kk] : 0xFFFFu;
    }
  };
  int L, nb;
  if constexpr (BALANCED) {
    // view pages of sequence bb (per KV head) decide its split count
    auto load = [&](int bb) {
      return SeqLoad{max(0, min(a.num_blocks[bb], a.max_blocks)), a.seq_lens[bb]};
    };
    const SeqLoad first = map_first_loads(a, load);
    first_entries(wi);
    const WorkItem guess = wi;
    if (!ragged_map(a, load, first, blockIdx.x, wi, nb, L)) return;
    if (wi.b != guess.b || wi.split != guess.split || wi.n_split != guess.n_split)
      first_entries(wi);
  } else {
    first_entries(wi);
    L = a.seq_lens[wi.b];
    nb = max(0, min(a.num_blocks[wi.b], a.max_blocks));
  }
  const int split = wi.split, g = wi.g, b = wi.b, n_split = wi.n_split;
  const int nw = n_split * kWaves;
  const int u = split * kWaves + wave;
  const int32_t *vbt = a.block_table + (size_t)b * a.bt_stride;
  const int32_t *vlb = a.logical_block + (size_t)b * a.bt_stride;
  const uint32_t *vmk = MASKED ? a.token_mask + (size_t)b * a.bt_stride : nullptr;
  // Entries of the pages a ring round ahead, read through the vector memory
  // pipe (see table_ahead): issued when a ring slot is refilled, used when the
  // slot is refilled next, one round later.
  const int vz = opaque_zero();
  const auto rbt = table_rsrc(vbt, last_entry + 1);
  const auto rlb = table_rsrc(vlb, last_entry + 1);
  const auto rmk = table_rsrc(MASKED ? reinterpret_cast<const int32_t *>(vmk) : vbt, last_entry + 1);
  int ahead_pg[RING], ahead_lb[RING], ahead_mk[RING];
  auto table_issue = [&](int entry, int j) {
    const int kk = min(entry, last_entry);
    ahead_pg[j] = table_ahead(rbt, vz, kk);
    ahead_lb[j] = table_ahead(rlb, vz, kk);
    ahead_mk[j] = MASKED ? table_ahead(rmk, vz, kk) : 0xFFFF;
  };

  // query slices of the four heads, as bf16 pairs matching the K slice
  uint32_t qr[4][4][4];
  {
    const uint16_t *qb = static_cast<const uint16_t *>(a.q) + ((size_t)b * a.Hq + g * 4) * kD;
#pragma unroll
    for (int hh = 0; hh < 4; ++hh)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const u32x4 v = *reinterpret_cast<const u32x4 *>(qb + hh * kD + i * 32 + c * 8);
#pragma unroll
        for (int w = 0; w < 4; ++w) qr[hh][i][w] = v[w];
      }
  }

  float m_c = -INFINITY;     // running max (log2 units) of head c
  float l_c = 0.f;           // partial sum of p over this lane's tokens, head c
  float acc[4][4];           // [head][dim i] over this lane's token half
#pragma unroll
  for (int hh = 0; hh < 4; ++hh)
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[hh][i] = 0.f;

  const int n_my = u < nb ? div_small(nb - 1 - u, nw) + 1 : 0;

  // The i-th view entry of this wavefront -> its page (0 for an invalid id)
  // and its visible tokens as a 16-bit mask, bit t = token t (none if the id
  // is invalid, the block lies past the sequence, or i is past this
  // wavefront's entries): tokens below the sequence length, and with a token
  // mask only those whose bit is set.
  auto validate = [&](bool live, int raw_page, int raw_lblk, uint32_t raw_mask, int &page,
                      uint32_t &vis) {
    const long long rem = (long long)L - (long long)raw_lblk * kPage;
    const int nvalid = (int)(rem < 0 ? 0 : (rem > kPage ? kPage : rem));
    vis = (0xFFFFu >> (kPage - nvalid)) & raw_mask;
    page = raw_page;
    if (page < 0 || (int64_t)page >= a.num_pages || !live) {
      vis = 0u;
      page = 0;
    }
  };
  auto page_info = [&](bool live, int j, int &page, uint32_t &vis) {   // entries from table_issue
    validate(live, lane_value(ahead_pg[j], 0), lane_value(ahead_lb[j], 0),
             MASKED ? (uint32_t)lane_value(ahead_mk[j], 0) : 0xFFFFu, page, vis);
  };

  auto process = [&](const PageRegs<KV> &cur, int page, uint32_t vis) {
    float ksc = a.scale_log2, vsc = 1.f;
    if constexpr (KV == kFP8) {
      ksc *= cur.sc.x;
      vsc = cur.sc.y;
    }
    // ---- logits --------------------------------------------------------------
    uint32_t kk[4][4];
    k_pairs<KV>(cur, kk);
    float d0 = 0.f, d1 = 0.f, d2 = 0.f, d3 = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        d0 = dot2(kk[i][w], qr[0][i][w], d0);
        d1 = dot2(kk[i][w], qr[1][i][w], d1);
        d2 = dot2(kk[i][w], qr[2][i][w], d2);
        d3 = dot2(kk[i][w], qr[3][i][w], d3);
      }
    // transposing reduction inside the quad: lane c ends with head c
    const bool o1 = c & 1, o2 = c & 2;
    float keep0 = o1 ? d1 : d0, send0 = o1 ? d0 : d1;
    float keep1 = o1 ? d3 : d2, send1 = o1 ? d2 : d3;
    keep0 += dpp<kQuadXor1>(send0);
    keep1 += dpp<kQuadXor1>(send1);
    float s = o2 ? keep1 : keep0;
    s += dpp<kQuadXor2>(o2 ? keep0 : keep1);
    s = ((vis >> t) & 1u) ? s * ksc : -INFINITY;

    // ---- online softmax ------------------------------------------------------
    float pm = fmaxf(s, dpp<kRowRor4>(s));
    pm = fmaxf(pm, dpp<kRowRor8>(pm));
    pm = xor16_max(pm);
    pm = xor32_max(pm);
    const float m_new = fmaxf(m_c, pm);
    if (__any(m_new > m_c)) {
      const float alpha = exp2_fast(m_c - (m_new == -INFINITY ? 0.f : m_new));
      l_c *= alpha;
      float al[4];
#pragma unroll
      for (int hh = 0; hh < 4; ++hh)
        al[hh] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(alpha), hh));
#pragma unroll
      for (int hh = 0; hh < 4; ++hh)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[hh][i] *= al[hh];
      m_c = m_new;
    }
    const float p = exp2_fast(s - (m_c == -INFINITY ? 0.f : m_c));
    l_c += p;
    pbuf[wave][lane] = p * vsc;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // ---- o += p V --------------------------------------------------------------
    float vv[4][8];
    v_floats<KV>(cur, vv);
    if (vis != 0xFFFFu) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const bool ok = (vis >> (hf * 8 + j)) & 1u;
#pragma unroll
        for (int i = 0; i < 4; ++i) vv[i][j] = ok ? vv[i][j] : 0.f;
      }
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float4 pj = *reinterpret_cast<const float4 *>(&pbuf[wave][(hf * 8 + j) * 4]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[0][i] = fmaf(pj.x, vv[i][j], acc[0][i]);
        acc[1][i] = fmaf(pj.y, vv[i][j], acc[1][i]);
        acc[2][i] = fmaf(pj.z, vv[i][j], acc[2][i]);
        acc[3][i] = fmaf(pj.w, vv[i][j], acc[3][i]);
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  };

  // RING page buffers, unrolled by RING: while one page is processed the loads
  // of the next RING - 1 are in flight. Loads are unconditional (past the end
  // of this wavefront's pages they go through an empty descriptor and read
  // nothing), so the steady state is straight-line code. The main loop runs
  // whole rounds of RING pages with no early exit -- an exit inside the round
  // would merge a just-issued load into the loop header's wait and drain the
  // ring every round -- and the remaining pages are processed after it.
  PageRegs<KV> r[RING];
  int pg[RING];
  uint32_t nv[RING];
  // (each slot's table reads follow its page loads, as in the loop, so the
  // wait counts at the loop header are the steady-state ones)
#pragma unroll
  for (int j = 0; j < RING; ++j) {
    validate(j < n_my, raw_pg[j], raw_lb[j], raw_mk[j], pg[j], nv[j]);
    load_page<KV>(r[j], a, pg[j], g, lane, nv[j] != 0u);
    __builtin_amdgcn_sched_barrier(0);
    table_issue(u + nw * (j + RING), j);
    __builtin_amdgcn_sched_barrier(0);
  }
  const int full = n_my - n_my % RING;
  for (int i = 0; i < full; i += RING) {
#pragma unroll
    for (int j = 0; j < RING; ++j) {
      process(r[j], pg[j], nv[j]);
      page_info(i + j + RING < n_my, j, pg[j], nv[j]);
      load_page<KV>(r[j], a, pg[j], g, lane, nv[j] != 0u);
      table_issue(u + nw * (i + j + 2 * RING), j);
    }
  }
#pragma unroll
  for (int j = 0; j < RING - 1; ++j)
    if (full + j < n_my) process(r[j], pg[j], nv[j]);

  // ---- per-wave totals -------------------------------------------------------
  float lt = l_c + dpp<kRowRor4>(l_c);
  lt += dpp<kRowRor8>(lt);
  lt = xor16_sum(lt);
  lt = xor32_sum(lt);
#pragma unroll
  for (int hh = 0; hh < 4; ++hh)
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[hh][i] += dpp<kQuadXor1>(acc[hh][i]);
  if (lane < 4) {
    wstat[0][wave][lane] = m_c;
    wstat[1][wave][lane] = lt;
  }
  if (hf == 0) {
#pragma unroll
    for (int hh = 0; hh < 4; ++hh)
#pragma unroll
      for (int i = 0; i < 4; ++i) wacc[wave][hh][i * 32 + (lane >> 1)] = acc[hh][i];
  }
  __syncthreads();

  // ---- merge the four wavefronts ------------------------------------------------
  const int hh = threadIdx.x >> 6;
  const int d0 = (threadIdx.x & 63) * 2;
  float M = -INFINITY;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) M = fmaxf(M, wstat[0][w][hh]);
  const size_t row = (size_t)b * a.Hq + g * 4 + hh;
  float o0 = 0.f, o1v = 0.f, lse2 = -INFINITY;
  if (M != -INFINITY) {
    float den = 0.f, n0 = 0.f, n1 = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float e = exp2f(wstat[0][w][hh] - M);
      den = fmaf(e, wstat[1][w][hh], den);
      n0 = fmaf(e, wacc[w][hh][d0], n0);
      n1 = fmaf(e, wacc[w][hh][d0 + 1], n1);
    }
    o0 = n0 / den;
    o1v = n1 / den;
    lse2 = M + log2f(den);
  }
  if (n_split == 1) {
    *reinterpret_cast<float2 *>(a.out + row * kD + d0) = make_float2(o0, o1v);
    if ((threadIdx.x & 63) == 0) a.lse[row] = lse2 * kLn2;
    return;
  }
  // several splits: stage the partial in LDS, wavefront 0 writes it and takes
  // the arrival ticket; the last workgroup of (b, g) merges the splits
  *reinterpret_cast<float2 *>(&s_part[hh][d0]) = make_float2(o0, o1v);
  if ((threadIdx.x & 63) == 0) s_plse[hh] = lse2;
  __syncthreads();
  if (threadIdx.x < 64) {
    const auto ro = partial_rsrc(a.part_o);
    const auto rl = partial_rsrc(a.part_lse);
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
      const int f = threadIdx.x + 64 * t2;       // float4 index in [4][128]
      const int h4 = f >> 5, d4 = (f & 31) * 4;
      const size_t pr = (size_t)(wi.slot0 + split) * 4 + h4;
      partial_store4(ro, (pr * kD + d4) * 4, *reinterpret_cast<const float4 *>(&s_part[h4][d4]));
    }
    if (threadIdx.x < 4) {
      const size_t pr = (size_t)(wi.slot0 + split) * 4 + threadIdx.x;
      partial_store1(rl, pr * 4, s_plse[threadIdx.x]);
    }
  }
  if (last_arrival(a, b, g, n_split, &s_flag)) merge_rows(a, b, g, 4, wi.slot0, n_split);
}

template <int KV, int RING, bool MASKED>
void launch_mode(const AttnArgs &a, hipStream_t s) {
  if (a.ragged)
    hipLaunchKernelGGL((decode_fast_kernel<KV, RING, true, MASKED>), dim3(a.n_split), dim3(256),
                       0, s, a);
  else
    hipLaunchKernelGGL((decode_fast_kernel<KV, RING, false, MASKED>),
                       dim3(a.n_split, a.Hkv, a.batch), dim3(256), 0, s, a);
}

template <int KV, int RING>
hipError_t launch_kv(const AttnArgs &a, hipStream_t s) {
  if (a.token_mask)
    launch_mode<KV, RING, true>(a, s);
  else
    launch_mode<KV, RING, false>(a, s);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_decode_fast(const AttnArgs &a, hipStream_t s) {
  if (a.kv_type == kBF16) return launch_kv<kBF16, kRingBF16>(a, s);
  if (a.kv_type == kFP8) return launch_kv<kFP8, kRingFP8>(a, s);
  return hipErrorInvalidValue;
}

int decode_fast_blocks_per_cu(int kv_type) {
  int nb = 0;
  const hipError_t e =
      kv_type == kFP8
          ? hipOccupancyMaxActiveBlocksPerMultiprocessor(
                &nb, decode_fast_kernel<kFP8, kRingFP8, true, false>, 256, 0)
          : hipOccupancyMaxActiveBlocksPerMultiprocessor(
                &nb, decode_fast_kernel<kBF16, kRingBF16, true, false>, 256, 0);
  return e == hipSuccess ? nb : 0;
}

}  // namespace kap

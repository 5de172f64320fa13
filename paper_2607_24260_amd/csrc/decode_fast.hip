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
// Both products of a page run on the matrix cores with the 4x4x4 bf16
// instruction (16 independent 4x4 blocks per wavefront), whose 4-row blocks
// fit the four query heads of a KV head. Lane l = 16 tg + 4 dg + j:
//  * logits: block (tg, dg) multiplies the four heads' query slice of dims
//    32 dg .. 32 dg + 31 with token 4 tg + j's K slice, 4 dims per step, 8
//    steps. K pages are stored in 8-dim chunks ([chunk][token][8]), so a lane
//    reads four chunks of its token and each load instruction reads four full
//    chunk rows (4 x 128 / 256 bytes). Row rotations sum the four dim groups;
//    lane l then keeps the logit of head dg, token 4 tg + j.
//  * softmax: page maxima per head over lane bits 0-1 (quad swaps) and 4-5
//    (permlane16 / permlane32 swaps); running max and sum per head in every
//    lane that owns that head.
//  * o += p V: every block multiplies the four heads' weights of 4 tokens with
//    the V values of 4 dims; lane l reads V^T rows l and l + 64 (1 KB
//    contiguous per load instruction for fp8) and accumulates o for the four
//    heads at dims l and l + 64. The weights travel through LDS as bf16
//    hi + lo parts (error below 2^-15 relative), so the matrix product keeps
//    near-fp32 weights.
// fp8 KV is widened to bf16 at use (exact); per-page scales fold into the
// logit scale and the weights. Moving the 4 flop per KV byte off the vector
// ALU leaves it the widening and the softmax, and the loads set the pace.
#include "kap_internal.h"

namespace kap {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kD = 128;
constexpr int kWaves = 4;
// pages in flight per wavefront (register ring depth). Two beat one and
// three on MI355X for both dtypes (128K workload: 23.8 vs 26.4 / 24.1 us per
// call; ragged fp8 full context: 773 vs 799 / 776 us): a deeper ring does not
// raise the read rate and costs registers and loop overhead.
constexpr int kRingBF16 = 2;
constexpr int kRingFP8 = 2;

// D += A B on 16 blocks of 4x4 (K = 4, bf16 operands, fp32 accumulation):
// block b = lane / 4; A row i of block b comes from lane 4 b + i, B column j
// from lane 4 b + j, and D[i][j] lands in element i of lane 4 b + j.
__device__ __forceinline__ f32x4 mfma4(u32x2 a, u32x2 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(__builtin_bit_cast(s16x4, a),
                                                 __builtin_bit_cast(s16x4, b), c, 0, 0, 0);
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

// Raw registers of one page. k[cc]: chunk 4 dg + cc (dims 32 dg + 8 cc ..
// + 7) of token 4 tg + j; v: V^T rows l and l + 64 (16 tokens each).
template <int KV> struct PageRegs;
template <> struct PageRegs<kBF16> { u32x4 k[4]; u32x4 v[4]; };   // v[0..1]: row l, v[2..3]: row l + 64
template <> struct PageRegs<kFP8> { u32x2 k[4]; u32x4 v[2]; float2 sc; };   // sc: (K, V) scales

// Loads of one (page, head) tile. With live == false the descriptor covers
// zero bytes: the loads return zeros without touching memory (used for
// invalid pages and for the ring's prefetches past a wavefront's last page).
template <int KV>
__device__ __forceinline__ void load_page(PageRegs<KV> &r, const AttnArgs &a, int page, int g,
                                          int lane, bool live) {
  const int t = ((lane >> 4) << 2) | (lane & 3), dg = (lane >> 2) & 3;
  constexpr int kTile = (KV == kBF16 ? 2 : 1) * kPage * kD;   // bytes per (page, head) tile
  const size_t off = ((size_t)page * a.Hkv + g) * kTile;
  const int bytes = live ? kTile : 0;
  const auto kr = tile_rsrc(a.k_pages, off, bytes);
  const auto vr = tile_rsrc(a.v_pages, off, bytes);
  if constexpr (KV == kBF16) {
#pragma unroll
    for (int cc = 0; cc < 4; ++cc) r.k[cc] = tile_load16(kr, (4 * dg + cc) * 256 + t * 16);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      r.v[2 * h] = tile_load16(vr, (64 * h + lane) * 32);
      r.v[2 * h + 1] = tile_load16(vr, (64 * h + lane) * 32 + 16);
    }
  } else {
#pragma unroll
    for (int cc = 0; cc < 4; ++cc) r.k[cc] = tile_load8(kr, (4 * dg + cc) * 128 + t * 8);
#pragma unroll
    for (int h = 0; h < 2; ++h) r.v[h] = tile_load16(vr, (64 * h + lane) * 16);
    r.sc = page_scales(a.kv_scales, page, live);
  }
}

// K operand of logit step st (dims 32 dg + 4 st .. + 3 of this lane's token)
// as four bf16 values.
template <int KV>
__device__ __forceinline__ u32x2 k_operand(const PageRegs<KV> &r, int st) {
  const int cc = st >> 1, h = st & 1;
  if constexpr (KV == kBF16)
    return u32x2{r.k[cc][2 * h], r.k[cc][2 * h + 1]};
  else
    return fp8x4_to_bf16x4(r.k[cc][h]);
}

// V operand of weight step st (tokens 4 st .. 4 st + 3 of V^T row
// 64 half + l) as four bf16 values, after the page's visibility masks were
// applied to the raw registers.
template <int KV>
__device__ __forceinline__ u32x2 v_operand(const PageRegs<KV> &r, int half, int st) {
  if constexpr (KV == kBF16) {
    const u32x4 &w = r.v[2 * half + (st >> 1)];
    return (st & 1) ? u32x2{w[2], w[3]} : u32x2{w[0], w[1]};
  } else {
    return fp8x4_to_bf16x4(r.v[half][st]);
  }
}

// Clears the V values of tokens whose bit in vis is 0, so that their zero
// weights meet zeros (not whatever the page holds there). vis is the same in
// every lane, so the byte / half-word masks are scalar work.
template <int KV>
__device__ __forceinline__ void mask_v(PageRegs<KV> &r, uint32_t vis) {
  if constexpr (KV == kBF16) {
    // dword w of a row holds tokens 2 w, 2 w + 1 (w = 0..7 over v[2h], v[2h+1])
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      const uint32_t m = ((vis >> (2 * w)) & 1u ? 0x0000FFFFu : 0u) |
                         ((vis >> (2 * w + 1)) & 1u ? 0xFFFF0000u : 0u);
#pragma unroll
      for (int h = 0; h < 2; ++h) r.v[2 * h + (w >> 2)][w & 3] &= m;
    }
  } else {
    // dword w of a row holds tokens 4 w .. 4 w + 3, one byte each
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const uint32_t nib = (vis >> (4 * w)) & 0xFu;
      const uint32_t m = ((nib & 1u) ? 0x000000FFu : 0u) | ((nib & 2u) ? 0x0000FF00u : 0u) |
                         ((nib & 4u) ? 0x00FF0000u : 0u) | ((nib & 8u) ? 0xFF000000u : 0u);
#pragma unroll
      for (int h = 0; h < 2; ++h) r.v[h][w] &= m;
    }
  }
}

// How a workgroup finds its work item: uniform splits (the grid is
// (n_split, Hkv, batch)), the balanced map computed here, or the balanced
// map's record precomputed for the view by decode_schedule_kernel.
enum DecodeMode { kUniform, kBalanced, kScheduled };

template <int KV, int RING, int MODE, bool MASKED>
__global__ __launch_bounds__(256) void decode_fast_kernel(AttnArgs a) {
  constexpr bool BALANCED = MODE == kBalanced;
  static_assert(MODE != kScheduled || RING == 2, "schedule records hold two ring entries");
  __shared__ __attribute__((aligned(16))) uint16_t pw_hi[kWaves][4][kPage];   // weights (x V scale), bf16 hi + lo
  __shared__ __attribute__((aligned(16))) uint16_t pw_lo[kWaves][4][kPage];
  __shared__ float wstat[2][kWaves][4];            // per-wave m (log2) and l per head
  __shared__ float wacc[kWaves][4][kD];
  __shared__ float s_part[4][kD];
  __shared__ float s_plse[4];
  __shared__ int s_flag;

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  // lane roles: logits of token t = 4 tg + j, dim group / owned head dg;
  // weight rows: head hq; output columns: dims lane and lane + 64
  const int t = ((lane >> 4) << 2) | (lane & 3), dg = (lane >> 2) & 3, hq = lane & 3;

  // Work unit. Balanced mode: the map needs the view lengths of the whole
  // batch, so the first table entries are read for a guess while it is
  // computed -- the even assignment, a.guess_splits splits per unit, which
  // the map produces for equal views -- and read again if the map differs.
  WorkItem wi;
  if constexpr (MODE == kScheduled) {
  } else if constexpr (BALANCED) {
    const int ng = a.guess_splits;
    const int w = blockIdx.x;
    const int q = div_u21(w, ng);   // w < slots < 2^21
    wi.n_split = ng;
    wi.split = w - q * ng;
    const int bq = div_u21(q, a.Hkv);
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
  if constexpr (MODE == kScheduled) {
    // the record of this workgroup (uniform address: scalar loads), clamped
    // so that a record that does not belong to these arguments cannot lead
    // outside the arrays
    const int32_t *rec = a.schedule + (size_t)blockIdx.x * kSchedInts;
    wi.n_split = rec[kSchedNSplit];
    if (wi.n_split <= 0) return;
    wi.n_split = min(wi.n_split, a.n_split);
    wi.b = min(max(rec[kSchedB], 0), a.batch - 1);
    wi.g = min(max(rec[kSchedG], 0), a.Hkv - 1);
    wi.split = min(max(rec[kSchedSplit], 0), wi.n_split - 1);
    wi.slot0 = min(max(rec[kSchedSlot0], 0), a.n_split - wi.n_split);
    L = rec[kSchedL];
    nb = min(max(rec[kSchedNb], 0), a.max_blocks);
#pragma unroll
    for (int j = 0; j < RING; ++j) {
      const int32_t *e = rec + kSchedEntries + 3 * (2 * wave + j);
      raw_pg[j] = e[0];
      raw_lb[j] = e[1];
      raw_mk[j] = MASKED ? (uint32_t)e[2] : 0xFFFFu;
    }
  } else if constexpr (BALANCED) {
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

  // query operand of logit step st: head hq, dims 32 dg + 4 st .. + 3 (bf16)
  u32x2 qa[8];
  {
    const uint16_t *qb =
        static_cast<const uint16_t *>(a.q) + ((size_t)b * a.Hq + g * 4 + hq) * kD + 32 * dg;
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const u32x4 v = *reinterpret_cast<const u32x4 *>(qb + 8 * q4);
      qa[2 * q4] = u32x2{v[0], v[1]};
      qa[2 * q4 + 1] = u32x2{v[2], v[3]};
    }
  }

  float m_c = -INFINITY;     // running max (log2 units) of head dg
  float l_c = 0.f;           // partial sum of p over this lane's tokens, head dg
  f32x4 o_lo = {0.f, 0.f, 0.f, 0.f};   // o[head i][dim lane]
  f32x4 o_hi = {0.f, 0.f, 0.f, 0.f};   // o[head i][dim lane + 64]

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

  auto process = [&](PageRegs<KV> &cur, int page, uint32_t vis) {
    float ksc = a.scale_log2, vsc = 1.f;
    if constexpr (KV == kFP8) {
      ksc *= cur.sc.x;
      vsc = cur.sc.y;
    }
    // ---- logits: partial over this lane's dim group, then summed ---------------
    f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < 8; st += 2) {
      sa = mfma4(qa[st], k_operand<KV>(cur, st), sa);
      sb = mfma4(qa[st + 1], k_operand<KV>(cur, st + 1), sb);
    }
    f32x4 sc4 = sa + sb;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sc4[i] += dpp<kRowRor4>(sc4[i]);
      sc4[i] += dpp<kRowRor8>(sc4[i]);
    }
    float s = dg == 0 ? sc4[0] : dg == 1 ? sc4[1] : dg == 2 ? sc4[2] : sc4[3];
    s = ((vis >> t) & 1u) ? s * ksc : -INFINITY;

    // ---- online softmax ------------------------------------------------------
    float pm = max_f(s, dpp<kQuadXor1>(s));
    pm = max_f(pm, dpp<kQuadXor2>(pm));
    pm = xor16_max(pm);
    pm = xor32_max(pm);
    const float m_new = max_f(m_c, pm);
    if (__any(m_new > m_c)) {
      const float alpha = exp2_fast(m_c - (m_new == -INFINITY ? 0.f : m_new));
      l_c *= alpha;
#pragma unroll
      for (int hh = 0; hh < 4; ++hh) {
        // lane 4 hh owns head hh
        const float al = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(alpha), 4 * hh));
        o_lo[hh] *= al;
        o_hi[hh] *= al;
      }
      m_c = m_new;
    }
    const float p = exp2_fast(s - (m_c == -INFINITY ? 0.f : m_c));
    l_c += p;
    const float pv = p * vsc;
    const uint32_t hi = __float_as_uint(pv) & 0xFFFF0000u;
    pw_hi[wave][dg][t] = (uint16_t)(hi >> 16);
    pw_lo[wave][dg][t] = (uint16_t)(__float_as_uint(pv - __uint_as_float(hi)) >> 16);
    if (vis != 0xFFFFu) mask_v<KV>(cur, vis);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // ---- o += p V --------------------------------------------------------------
    const u32x4 ph0 = *reinterpret_cast<const u32x4 *>(&pw_hi[wave][hq][0]);
    const u32x4 ph1 = *reinterpret_cast<const u32x4 *>(&pw_hi[wave][hq][8]);
    const u32x4 pl0 = *reinterpret_cast<const u32x4 *>(&pw_lo[wave][hq][0]);
    const u32x4 pl1 = *reinterpret_cast<const u32x4 *>(&pw_lo[wave][hq][8]);
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      const u32x4 &h4 = st < 2 ? ph0 : ph1;
      const u32x4 &l4 = st < 2 ? pl0 : pl1;
      const u32x2 ah = (st & 1) ? u32x2{h4[2], h4[3]} : u32x2{h4[0], h4[1]};
      const u32x2 al = (st & 1) ? u32x2{l4[2], l4[3]} : u32x2{l4[0], l4[1]};
      const u32x2 v0 = v_operand<KV>(cur, 0, st), v1 = v_operand<KV>(cur, 1, st);
      o_lo = mfma4(ah, v0, o_lo);
      o_hi = mfma4(ah, v1, o_hi);
      o_lo = mfma4(al, v0, o_lo);
      o_hi = mfma4(al, v1, o_hi);
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
  float lt = l_c + dpp<kQuadXor1>(l_c);
  lt += dpp<kQuadXor2>(lt);
  lt = xor16_sum(lt);
  lt = xor32_sum(lt);
  if ((lane & 0x33) == 0) {   // lanes 0, 4, 8, 12: heads 0..3
    wstat[0][wave][dg] = m_c;
    wstat[1][wave][dg] = lt;
  }
#pragma unroll
  for (int hh = 0; hh < 4; ++hh) {
    wacc[wave][hh][lane] = o_lo[hh];
    wacc[wave][hh][64 + lane] = o_hi[hh];
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
  if (last_arrival(a, b, g, n_split, &s_flag)) merge_rows<1>(a, b, g, 4, wi.slot0, n_split);
}

template <int KV, int RING, bool MASKED>
void launch_mode(const AttnArgs &a, hipStream_t s) {
  if (a.ragged && a.schedule)
    hipLaunchKernelGGL((decode_fast_kernel<KV, RING, kScheduled, MASKED>), dim3(a.n_split),
                       dim3(256), 0, s, a);
  else if (a.ragged)
    hipLaunchKernelGGL((decode_fast_kernel<KV, RING, kBalanced, MASKED>), dim3(a.n_split),
                       dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((decode_fast_kernel<KV, RING, kUniform, MASKED>),
                       dim3(a.n_split, a.Hkv, a.batch), dim3(256), 0, s, a);
}

// One wavefront per balanced-mode workgroup w: the map's work item for w and
// the first two view entries of each of its four wavefronts, as a record.
// Workgroups past the last slot get a record with no work.
__global__ __launch_bounds__(64) void decode_schedule_kernel(AttnArgs a) {
  const int lane = threadIdx.x;
  auto load = [&](int bb) {
    return SeqLoad{max(0, min(a.num_blocks[bb], a.max_blocks)), a.seq_lens[bb]};
  };
  const SeqLoad first = map_first_loads(a, load);
  WorkItem wi;
  int nb = 0, L = 0;
  const bool live = ragged_map(a, load, first, blockIdx.x, wi, nb, L);
  int32_t *rec = a.schedule_out + (size_t)blockIdx.x * kSchedInts;
  if (!live) {
    if (lane < kSchedEntries) rec[lane] = 0;
    return;
  }
  if (lane < kSchedEntries) {
    const int v[kSchedEntries] = {wi.b, wi.g, wi.split, wi.n_split, wi.slot0, L, nb, 0};
    int x = 0;
#pragma unroll
    for (int f = 0; f < kSchedEntries; ++f) x = lane == f ? v[f] : x;
    rec[lane] = x;
  }
  if (lane < 2 * kWaves) {
    // lane 2 w + j: ring slot j of wavefront w, view entry
    // (4 split + w) + 4 n_split j of the sequence (clamped to the row)
    const int w = lane >> 1, j = lane & 1;
    const int last_entry = max(a.max_blocks - 1, 0);
    const int kk = min(wi.split * kWaves + w + wi.n_split * kWaves * j, last_entry);
    const size_t at = (size_t)wi.b * a.bt_stride + kk;
    int32_t *e = rec + kSchedEntries + 3 * lane;
    e[0] = a.block_table[at];
    e[1] = a.logical_block[at];
    e[2] = a.token_mask ? (int32_t)a.token_mask[at] : 0xFFFF;
  }
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

hipError_t launch_decode_schedule(const AttnArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(decode_schedule_kernel, dim3(a.n_split), dim3(64), 0, s, a);
  return hipGetLastError();
}

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
                &nb, decode_fast_kernel<kFP8, kRingFP8, kBalanced, false>, 256, 0)
          : hipOccupancyMaxActiveBlocksPerMultiprocessor(
                &nb, decode_fast_kernel<kBF16, kRingBF16, kBalanced, false>, 256, 0);
  return e == hipSuccess ? nb : 0;
}

}  // namespace kap

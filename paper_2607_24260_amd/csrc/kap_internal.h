// Internal declarations shared by the HIP sources of libkap (not installed).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace kap {

constexpr int kPage = 16;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kPlanThreads = 256;
constexpr int kGenericPagesPerSplit = 64;   // 1024 keys staged per generic work item
constexpr int kMaxPlanPages = 262144;       // pages per sequence the plan bitmap covers

enum KvType { kF32 = 0, kBF16 = 1, kFP8 = 2 };

// Arguments of kap_compile_plan after host validation.
struct PlanArgs {
  int batch;
  const int32_t *seq_lens;
  const int32_t *fbt;
  int fbt_stride;
  const int32_t *span_offsets;
  int num_spans;
  const int32_t *span_start;
  const int32_t *span_len;
  const float *span_prior;
  const int32_t *prefix;
  const int32_t *suffix;
  const int32_t *budget;
  int policy;
  int64_t num_pages;
  int capacity;
  int32_t *view_bt;
  int32_t *view_lblk;
  int32_t *view_nblk;
  int32_t *view_tokens;
  int32_t *spans_taken;
  int32_t *status;
  int32_t *span_selected;
  int32_t *perm;  // workspace: [num_spans] rank -> local span index
};

// One attention call (decode or verify) after host validation.
// Rows per sequence: R = q_len * Hq; row r is window token r / Hq, head r % Hq.
struct AttnArgs {
  int batch, Hq, Hkv, G, D;
  int kv_type;
  const void *k_pages;
  const void *v_pages;
  const float *kv_scales;
  int64_t num_pages;
  const void *q;          // [batch][q_len][Hq][D], bf16 or f32
  int q_f32;              // 1 if q is float32
  int q_len;
  const int32_t *seq_lens;
  const int32_t *block_table;    // decode: view table; verify: full table
  int bt_stride;
  const int32_t *logical_block;  // decode: view logical pages; verify: NULL (identity)
  const int32_t *num_blocks;     // decode: view_num_blocks; verify: NULL (ceil(L/16))
  int max_blocks;                // host bound on pages read per sequence
  int causal;                    // verify: row i sees positions < L - q_len + i + 1
  float scale_log2;              // sm_scale * log2(e)
  int n_split;
  int pages_per_split;
  float *part_o;    // [batch * R][n_split][D]   (normalised partial outputs)
  float *part_lse;  // [batch * R][n_split]      (log2-domain partial LSE)
  float *out;       // [batch * R][D]
  float *lse;       // [batch * R]
};

hipError_t launch_compile_plan(const PlanArgs &a, hipStream_t s);
hipError_t launch_attn_generic(const AttnArgs &a, hipStream_t s);
hipError_t launch_decode_fast(const AttnArgs &a, hipStream_t s);
hipError_t launch_verify_mfma(const AttnArgs &a, hipStream_t s);
hipError_t launch_merge(const AttnArgs &a, hipStream_t s);

// ---------------------------------------------------------------------------
// device helpers
// ---------------------------------------------------------------------------

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Round-to-nearest-even float -> bfloat16 bits (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

// Two OCP E4M3FN codes (bytes 0,1 or 2,3 of w) -> two floats, exact.
template <bool HIGH>
__device__ __forceinline__ float2 fp8x2_to_f32(uint32_t w) {
  auto v = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(w), HIGH);
  return make_float2(v[0], v[1]);
}

// One E4M3FN code -> float (generic path).
__device__ __forceinline__ float fp8_to_f32(uint8_t b) {
  return __builtin_amdgcn_cvt_f32_fp8(static_cast<int>(b), 0);
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}
__device__ __forceinline__ int wave_sum_i(int x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

}  // namespace kap

/*
 * The kap.h C ABI used from plain C (no Python, no torch): the library is
 * linked like any C library and driven with HIP runtime allocations.
 *
 *   kap_c_smoke cpu   version, status strings and host-side validation
 *                     (nothing is enqueued; needs no GPU)
 *   kap_c_smoke gpu   the worked plan vector of the selection rule (L = 100,
 *                     FBT = [7,3,9,0,5,2,8], spans (20,10,.5) (40,30,.9)
 *                     (90,5,.9) (0,5,.1), prefix 16, suffix 8, budget 60) in
 *                     page and token mode under both policies, and decode,
 *                     scheduled decode and verify over one visible token,
 *                     whose closed form is out = v and lse = sm_scale * <q, k>
 *
 * Prints one line per check and exits non-zero on the first failure.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "kap.h"
#include "kap_diag.h"

static int failures = 0;

#define CHECK(cond, ...)                  \
  do {                                    \
    if (!(cond)) {                        \
      printf("FAIL %s:%d: ", __FILE__, __LINE__); \
      printf(__VA_ARGS__);                \
      printf("\n");                       \
      failures++;                         \
      return;                             \
    }                                     \
  } while (0)

#define HIP_OK(x) CHECK((x) == hipSuccess, "%s failed", #x)

static void *const FAKE = (void *)0x10000;

static void cpu_checks(void) {
  CHECK(kap_abi_version() == KAP_ABI_VERSION, "abi version %d", kap_abi_version());
  CHECK(strcmp(kap_status_string(KAP_ERR_WORKSPACE_TOO_SMALL), "KAP_ERR_WORKSPACE_TOO_SMALL") == 0,
        "status string");
  kap_kv_cache kv = {32, 8, 128, 16, KAP_DT_BF16, KAP_DT_BF16, FAKE, FAKE, NULL, 100};
  /* bad geometry and arguments are refused before anything is enqueued */
  kv.page_size = 32;
  CHECK(kap_selected_decode(&kv, 2, FAKE, FAKE, FAKE, FAKE, 8, FAKE, 8, 1.0f, 0, FAKE, FAKE,
                            NULL, 0, NULL) == KAP_ERR_UNSUPPORTED, "page size 32 accepted");
  kv.page_size = 16;
  CHECK(kap_verify(&kv, 2, 17, FAKE, FAKE, FAKE, 8, 128, 1.0f, 0, FAKE, FAKE, NULL, 0, NULL) ==
            KAP_ERR_INVALID_ARGUMENT, "q_len 17 accepted");
  CHECK(strlen(kap_last_error()) > 0, "no error message");
  CHECK(kap_compile_plan(1, FAKE, FAKE, 8, FAKE, 4, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 7, 100, 8,
                         FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, NULL, NULL, 0, NULL) ==
            KAP_ERR_INVALID_ARGUMENT, "unknown policy accepted");
  /* batch 0 is a successful no-op */
  CHECK(kap_verify(&kv, 0, 5, FAKE, FAKE, FAKE, 8, 128, 1.0f, 0, FAKE, FAKE, NULL, 0, NULL) ==
            KAP_OK, "batch 0");
  CHECK(kap_stream_read(FAKE, 0, NULL, NULL) == KAP_OK, "empty read");
  CHECK(kap_compile_plan_workspace_bytes(1, 4, 8) == 256, "plan workspace");
  printf("ok cpu checks\n");
}

/* ---- the worked plan vector ------------------------------------------------ */

static void plan_vector(int token_mode, int policy, const int32_t *want_lblk,
                        const int32_t *want_vbt, int want_n, int want_used, int want_taken,
                        const int32_t *want_sel, const uint32_t *want_mask) {
  const int32_t L = 100, fbt[7] = {7, 3, 9, 0, 5, 2, 8}, offs[2] = {0, 4};
  const int32_t st[4] = {20, 40, 90, 0}, ln[4] = {10, 30, 5, 5};
  const float pr[4] = {0.5f, 0.9f, 0.9f, 0.1f};
  const int32_t pre = 16, suf = 8, bud = 60;
  enum { CAP = 8 };
  int32_t *d_in, *d_out;
  float *d_pr;
  void *ws;
  HIP_OK(hipMalloc((void **)&d_in, 64 * sizeof(int32_t)));
  HIP_OK(hipMalloc((void **)&d_out, 64 * sizeof(int32_t)));
  HIP_OK(hipMalloc((void **)&d_pr, 4 * sizeof(float)));
  HIP_OK(hipMalloc(&ws, 256));
  int32_t host[64];
  memset(host, 0, sizeof host);
  /* inputs: [0] L, [1..7] fbt, [8..9] offsets, [10..13] start, [14..17] len,
     [18] prefix, [19] suffix, [20] budget */
  host[0] = L;
  memcpy(host + 1, fbt, sizeof fbt);
  memcpy(host + 8, offs, sizeof offs);
  memcpy(host + 10, st, sizeof st);
  memcpy(host + 14, ln, sizeof ln);
  host[18] = pre;
  host[19] = suf;
  host[20] = bud;
  HIP_OK(hipMemcpy(d_in, host, sizeof host, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_pr, pr, sizeof pr, hipMemcpyHostToDevice));
  HIP_OK(hipMemset(d_out, 0xff, 64 * sizeof(int32_t)));
  /* outputs: [0..7] view table, [8..15] logical pages, [16..23] masks,
     [24] blocks, [25] tokens, [26] taken, [27] status, [28..31] selected */
  int32_t *o = d_out;
  kap_status s;
  if (token_mode)
    s = kap_compile_plan_masked(1, d_in, d_in + 1, 7, d_in + 8, 4, d_in + 10, d_in + 14, d_pr,
                                d_in + 18, d_in + 19, d_in + 20, policy, 10, CAP, o, o + 8,
                                (uint32_t *)(o + 16), o + 24, o + 25, o + 26, o + 27, o + 28,
                                ws, 256, NULL);
  else
    s = kap_compile_plan(1, d_in, d_in + 1, 7, d_in + 8, 4, d_in + 10, d_in + 14, d_pr, d_in + 18,
                         d_in + 19, d_in + 20, policy, 10, CAP, o, o + 8, o + 24, o + 25, o + 26,
                         o + 27, o + 28, ws, 256, NULL);
  CHECK(s == KAP_OK, "compile_plan: %s", kap_last_error());
  HIP_OK(hipDeviceSynchronize());
  HIP_OK(hipMemcpy(host, d_out, sizeof host, hipMemcpyDeviceToHost));
  CHECK(host[27] == KAP_PLAN_OK, "status %d", host[27]);
  CHECK(host[24] == want_n, "blocks %d, want %d", host[24], want_n);
  CHECK(host[25] == want_used, "tokens %d, want %d", host[25], want_used);
  CHECK(host[26] == want_taken, "taken %d, want %d", host[26], want_taken);
  for (int k = 0; k < want_n; ++k) {
    CHECK(host[8 + k] == want_lblk[k] && host[k] == want_vbt[k], "entry %d: (%d, %d)", k,
          host[8 + k], host[k]);
    if (token_mode)
      CHECK((uint32_t)host[16 + k] == want_mask[k], "mask %d: %x", k, (unsigned)host[16 + k]);
  }
  for (int i = 0; i < 4; ++i) CHECK(host[28 + i] == want_sel[i], "span %d flag %d", i, host[28 + i]);
  hipFree(d_in);
  hipFree(d_out);
  hipFree(d_pr);
  hipFree(ws);
  printf("ok plan vector (%s, %s)\n", token_mode ? "token" : "page", policy ? "stop" : "skip");
}

/* ---- one visible token: out = v, lse = sm_scale * <q, k> ----------------- */

static uint16_t bf16(float x) { /* the values below are exact in bf16 */
  uint32_t u;
  memcpy(&u, &x, 4);
  return (uint16_t)(u >> 16);
}

static void one_token(void) {
  enum { HQ = 4, D = 128, PAGES = 2, TILE = 16 * D };
  static uint16_t k[PAGES * TILE], v[PAGES * TILE], q[HQ * D];
  float kf[D], vf[D], qf[HQ][D];
  memset(k, 0, sizeof k);
  memset(v, 0, sizeof v);
  for (int d = 0; d < D; ++d) {
    kf[d] = (float)((d % 7) - 3) * 0.25f;
    vf[d] = (float)(d % 5) * 0.5f - 1.0f;
    /* token 0 of physical page 1: K in 8-dim chunks, V dim-major */
    k[TILE + (d / 8) * 16 * 8 + d % 8] = bf16(kf[d]);
    v[TILE + d * 16] = bf16(vf[d]);
  }
  for (int h = 0; h < HQ; ++h)
    for (int d = 0; d < D; ++d) {
      qf[h][d] = (float)(((h + d) % 3) - 1) * 0.125f;
      q[h * D + d] = bf16(qf[h][d]);
    }
  void *dk, *dv, *dq, *ws;
  int32_t *dt;
  float *dout, *dlse;
  HIP_OK(hipMalloc(&dk, sizeof k));
  HIP_OK(hipMalloc(&dv, sizeof v));
  HIP_OK(hipMalloc(&dq, sizeof q));
  HIP_OK(hipMalloc((void **)&dt, 4 * sizeof(int32_t)));
  HIP_OK(hipMalloc((void **)&dout, HQ * D * sizeof(float)));
  HIP_OK(hipMalloc((void **)&dlse, HQ * sizeof(float)));
  HIP_OK(hipMemcpy(dk, k, sizeof k, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(dv, v, sizeof v, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(dq, q, sizeof q, hipMemcpyHostToDevice));
  /* seq_len 1; view table [1]; logical block [0]; view length 1 */
  const int32_t tables[4] = {1, 1, 0, 1};
  HIP_OK(hipMemcpy(dt, tables, sizeof tables, hipMemcpyHostToDevice));
  kap_kv_cache kv = {HQ, 1, D, 16, KAP_DT_BF16, KAP_DT_BF16, dk, dv, NULL, PAGES};
  const float scale = 0.5f;
  size_t need = kap_selected_decode_workspace_bytes(&kv, 1, 1, 0);
  size_t need_v = kap_verify_workspace_bytes(&kv, 1, 1, 1, 0);
  if (need_v > need) need = need_v;
  HIP_OK(hipMalloc(&ws, need + 256));
  HIP_OK(hipMemset(ws, 0, need + 256));
  /* the decode schedule of this view: the call refuses to run without it */
  const size_t sched_bytes = kap_decode_schedule_bytes(&kv, 1, 1);
  CHECK(sched_bytes > 0, "no schedule for a balanced decode");
  int32_t *dsched = NULL;
  HIP_OK(hipMalloc((void **)&dsched, sched_bytes));
  CHECK(kap_selected_decode_scheduled(&kv, 1, dq, dt, dt + 1, dt + 2, NULL, 1, dt + 3, 1, NULL,
                                      scale, dout, dlse, ws, need + 256, NULL) ==
            KAP_ERR_INVALID_ARGUMENT, "scheduled decode without a schedule accepted");
  CHECK(kap_decode_schedule(&kv, 1, dt, dt + 1, dt + 2, NULL, 1, dt + 3, 1, dsched, sched_bytes,
                            NULL) == KAP_OK, "decode_schedule: %s", kap_last_error());
  static const char *names[3] = {"decode", "verify", "scheduled decode"};
  float out[HQ * D], lse[HQ];
  for (int call = 0; call < 3; ++call) {
    kap_status s = call == 0
        ? kap_selected_decode(&kv, 1, dq, dt, dt + 1, dt + 2, 1, dt + 3, 1, scale, 0, dout, dlse,
                              ws, need + 256, NULL)
        : call == 1
        ? kap_verify(&kv, 1, 1, dq, dt, dt + 1, 1, 1, scale, 0, dout, dlse, ws, need + 256, NULL)
        : kap_selected_decode_scheduled(&kv, 1, dq, dt, dt + 1, dt + 2, NULL, 1, dt + 3, 1,
                                        dsched, scale, dout, dlse, ws, need + 256, NULL);
    CHECK(s == KAP_OK, "%s: %s", names[call], kap_last_error());
    HIP_OK(hipDeviceSynchronize());
    HIP_OK(hipMemcpy(out, dout, sizeof out, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(lse, dlse, sizeof lse, hipMemcpyDeviceToHost));
    for (int h = 0; h < HQ; ++h) {
      double z = 0;
      for (int d = 0; d < D; ++d) z += (double)qf[h][d] * kf[d];
      z *= scale;
      CHECK(fabs(lse[h] - z) <= 1e-5 * (1.0 + fabs(z)), "%s head %d lse %g, want %g",
            names[call], h, lse[h], z);
      for (int d = 0; d < D; ++d)
        CHECK(fabs(out[h * D + d] - vf[d]) <= 1e-6, "%s head %d dim %d: %g, want %g",
              names[call], h, d, out[h * D + d], vf[d]);
    }
    printf("ok one visible token (%s)\n", names[call]);
  }
  hipFree(dsched);
  hipFree(dk);
  hipFree(dv);
  hipFree(dq);
  hipFree(dt);
  hipFree(dout);
  hipFree(dlse);
  hipFree(ws);
}

int main(int argc, char **argv) {
  const int gpu = argc > 1 && strcmp(argv[1], "gpu") == 0;
  cpu_checks();
  if (gpu && !failures) {
    const int32_t lblk_skip[4] = {0, 1, 5, 6}, vbt_skip[4] = {7, 3, 2, 8};
    const int32_t sel_skip[4] = {1, 0, 1, 1};
    plan_vector(0, KAP_SELECT_SKIP, lblk_skip, vbt_skip, 4, 52, 3, sel_skip, NULL);
    const int32_t lblk_stop[3] = {0, 5, 6}, vbt_stop[3] = {7, 2, 8}, sel_stop[4] = {0, 0, 0, 0};
    plan_vector(0, KAP_SELECT_STOP, lblk_stop, vbt_stop, 3, 36, 0, sel_stop, NULL);
    const int32_t lblk_tok[6] = {0, 2, 3, 4, 5, 6}, vbt_tok[6] = {7, 9, 0, 5, 2, 8};
    const uint32_t mask_tok[6] = {0xFFFF, 0xFF00, 0xFFFF, 0x003F, 0xFC00, 0x000F};
    const int32_t sel_tok_skip[4] = {0, 1, 1, 1}, sel_tok_stop[4] = {0, 1, 1, 0};
    plan_vector(1, KAP_SELECT_SKIP, lblk_tok, vbt_tok, 6, 56, 3, sel_tok_skip, mask_tok);
    plan_vector(1, KAP_SELECT_STOP, lblk_tok, vbt_tok, 6, 56, 2, sel_tok_stop, mask_tok);
    one_token();
  }
  printf("%s\n", failures ? "FAILED" : "PASSED");
  return failures ? 1 : 0;
}

/*
 * A C99 client of the library's C ABI (include/wdc.h), built together with a
 * copy of the library whose host code carries AddressSanitizer and
 * UndefinedBehaviorSanitizer (the GPU kernels are compiled as usual). It walks
 * the host-side code of every entry point and its error paths; the sanitizers
 * turn any out-of-bounds access, use after free or undefined operation in that
 * host code into a failing exit status.
 *
 *   abi_driver cpu   context and descriptor handling only (no HIP call)
 *   abi_driver gpu   the above, then rollouts, step calls, batched calls and
 *                    kernel entry points of a small model on the current device
 *
 * It checks statuses and the finiteness of results, not their values (the
 * parity tests compare values with the oracle).
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "wdc.h"

static int g_fail = 0;

#define EXPECT(cond, ...)                                      \
  do {                                                         \
    if (!(cond)) {                                             \
      fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__);     \
      fprintf(stderr, __VA_ARGS__);                            \
      fprintf(stderr, "\n");                                   \
      g_fail = 1;                                              \
    }                                                          \
  } while (0)

#define OK(call)                                                                       \
  do {                                                                                 \
    wdc_status s_ = (call);                                                            \
    EXPECT(s_ == WDC_OK, "%s -> %d (%s)", #call, (int)s_, wdc_last_error(ctx_for_err)); \
  } while (0)

#define HIPOK(call)                                                          \
  do {                                                                       \
    hipError_t e_ = (call);                                                  \
    if (e_ != hipSuccess) {                                                  \
      fprintf(stderr, "HIP failure %s:%d: %s -> %d\n", __FILE__, __LINE__, #call, (int)e_); \
      exit(3);                                                               \
    }                                                                        \
  } while (0)

static const wdc_ctx *ctx_for_err = NULL;

/* The small float32 model of the parity tests: two sequential blocks, D = 256,
 * 4 x 64 heads, latent 16 x 4 x 16 x 16, patch 1 x 2 x 2. */
static wdc_model_desc tiny_desc(void) {
  wdc_model_desc d;
  memset(&d, 0, sizeof d);
  d.dtype = WDC_F32;
  d.hidden = 256;
  d.heads = 4;
  d.head_dim = 64;
  d.mlp_ratio = 4;
  d.n_seq = 2;
  d.cond_dim = 256;
  d.lat_c = 16;
  d.lat_f = 4;
  d.lat_h = 16;
  d.lat_w = 16;
  d.patch_t = 1;
  d.patch_h = 2;
  d.patch_w = 2;
  d.rope_t = 16;
  d.rope_h = 24;
  d.rope_w = 24;
  d.qk_norm = 1;
  d.max_batch = 2;
  return d;
}

/* A bf16 model with every block kind, text tokens and a camera vector. */
static wdc_model_desc joint_desc(void) {
  wdc_model_desc d = tiny_desc();
  d.dtype = WDC_BF16;
  d.n_seq = 1;
  d.n_dual = 1;
  d.n_single = 1;
  d.cam_dim = 96;
  d.text_tokens = 21;
  d.text_dim = 128;
  d.cond_dim = 64;
  d.lat_f = 3;
  d.lat_h = 10;
  d.lat_w = 14;
  return d;
}

static void host_checks(void) {
  wdc_params p;
  wdc_params_default(&p);
  EXPECT(p.age_max == 6, "anchor-age limit %d", p.age_max);
  EXPECT(p.bank_capacity >= 1 && p.bank_capacity <= WDC_MAX_BANK, "bank capacity %d", p.bank_capacity);

  wdc_model_desc descs[3];
  descs[0] = tiny_desc();
  descs[1] = joint_desc();
  descs[2] = joint_desc();
  descs[2].hidden = 3072;
  descs[2].heads = 24;
  descs[2].head_dim = 128;
  descs[2].rope_t = 16;
  descs[2].rope_h = 56;
  descs[2].rope_w = 56;
  descs[2].n_seq = 0;
  descs[2].n_dual = 20;
  descs[2].n_single = 40;
  descs[2].cond_dim = 4096;
  descs[2].cam_dim = 0;
  descs[2].text_tokens = 256;
  descs[2].text_dim = 4096;
  descs[2].lat_f = 33;
  descs[2].lat_h = 68;
  descs[2].lat_w = 120;
  for (int i = 0; i < 3; ++i) {
    wdc_ctx *ctx = NULL;
    OK(wdc_create(&descs[i], &p, NULL, &ctx));
    if (!ctx) continue;
    ctx_for_err = ctx;
    const int32_t n = wdc_weight_count(ctx);
    EXPECT(n > 0, "weight count %d", (int)n);
    size_t end = 0;
    for (int32_t j = 0; j < n; ++j) {
      const char *name = NULL;
      int64_t shape[2] = {0, 0};
      int32_t nd = 0;
      size_t off = 0;
      OK(wdc_weight_info(ctx, j, &name, shape, &nd, &off));
      EXPECT(name && strlen(name) > 2 && (nd == 1 || nd == 2) && off % 256 == 0, "tensor %d", (int)j);
      EXPECT(off >= end, "tensor %d overlaps the previous one", (int)j);
      end = off + (size_t)shape[0] * (size_t)(nd == 2 ? shape[1] : 1) * (descs[i].dtype == WDC_BF16 ? 2 : 4);
    }
    EXPECT(end <= wdc_weights_bytes(ctx), "weights blob too small");
    EXPECT(wdc_weight_info(ctx, n, NULL, NULL, NULL, NULL) != WDC_OK, "tensor index past the end accepted");
    EXPECT(wdc_workspace_bytes(ctx) > 0 && wdc_state_bytes(ctx) > 0, "sizes");
    /* no workspace bound: no scratch, so no key-range split */
    int32_t qbm = -1, ks = -1;
    OK(wdc_attention_plan(ctx, 67576, &qbm, &ks));
    EXPECT(qbm == 264 && ks == 1, "attention plan without a workspace: %d blocks, %d ranges", (int)qbm, (int)ks);
    EXPECT(wdc_attention_plan(ctx, 0, &qbm, &ks) == WDC_E_ARG, "empty attention plan accepted");
    /* calls before weights and workspace are bound fail cleanly */
    float dummy = 0.f;
    EXPECT(wdc_dit_forward(ctx, &dummy, 0.5, NULL, NULL, NULL, &dummy) != WDC_OK, "unbound forward accepted");
    EXPECT(strlen(wdc_last_error(ctx)) > 0, "no error message");
    ctx_for_err = NULL;
    OK(wdc_destroy(ctx));
  }

  /* rejected descriptors and parameters */
  wdc_ctx *ctx = NULL;
  wdc_model_desc bad = tiny_desc();
  bad.head_dim = 32;
  bad.heads = 8;
  EXPECT(wdc_create(&bad, &p, NULL, &ctx) != WDC_OK && ctx == NULL, "head size 32 accepted");
  EXPECT(strlen(wdc_last_error(NULL)) > 0, "no creation error message");
  bad = tiny_desc();
  bad.lat_h = 15;
  EXPECT(wdc_create(&bad, &p, NULL, &ctx) != WDC_OK, "latent not divisible by the patch accepted");
  bad = tiny_desc();
  bad.dtype = 7;
  EXPECT(wdc_create(&bad, &p, NULL, &ctx) == WDC_E_DTYPE, "dtype 7 accepted");
  wdc_params q = p;
  q.bank_capacity = WDC_MAX_BANK + 1;
  wdc_model_desc good = tiny_desc();
  EXPECT(wdc_create(&good, &q, NULL, &ctx) == WDC_E_ARG, "bank capacity past the maximum accepted");
  EXPECT(wdc_create(NULL, &p, NULL, &ctx) == WDC_E_ARG, "null descriptor accepted");
  EXPECT(wdc_destroy(NULL) != WDC_OK, "null context accepted");
  EXPECT(wdc_attention_plan(NULL, 10, NULL, NULL) == WDC_E_ARG, "attention plan of a null context accepted");
  EXPECT(wdc_weights_bytes(NULL) == 0 && wdc_weight_count(NULL) == 0, "null context sizes");
}

/* Seeded host data (a 64-bit LCG; values in [-1, 1)). */
static uint64_t g_rng = 0x9E3779B97F4A7C15ull;
static float urand(void) {
  g_rng = g_rng * 6364136223846793005ull + 1442695040888963407ull;
  return (float)((double)(g_rng >> 11) * (1.0 / 4503599627370496.0) - 1.0);
}

static void *dev_fill(size_t n_floats) {
  float *h = (float *)malloc(n_floats * sizeof(float));
  for (size_t i = 0; i < n_floats; ++i) h[i] = urand();
  void *d = NULL;
  HIPOK(hipMalloc(&d, n_floats * sizeof(float)));
  HIPOK(hipMemcpy(d, h, n_floats * sizeof(float), hipMemcpyHostToDevice));
  free(h);
  return d;
}

/* n bfloat16 values (the upper halves of seeded floats in [-1, 1)) */
static void *dev_fill_bf16(size_t n) {
  uint16_t *h = (uint16_t *)malloc(n * sizeof(uint16_t));
  for (size_t i = 0; i < n; ++i) {
    const float f = urand();
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    h[i] = (uint16_t)(u >> 16);
  }
  void *d = NULL;
  HIPOK(hipMalloc(&d, n * sizeof(uint16_t)));
  HIPOK(hipMemcpy(d, h, n * sizeof(uint16_t), hipMemcpyHostToDevice));
  free(h);
  return d;
}

static int all_finite(const void *d, size_t n_floats) {
  float *h = (float *)malloc(n_floats * sizeof(float));
  HIPOK(hipMemcpy(h, d, n_floats * sizeof(float), hipMemcpyDeviceToHost));
  int ok = 1;
  for (size_t i = 0; i < n_floats; ++i) ok &= isfinite(h[i]) ? 1 : 0;
  free(h);
  return ok;
}

static void gpu_checks(void) {
  int ndev = 0;
  HIPOK(hipGetDeviceCount(&ndev));
  EXPECT(ndev > 0, "no device");
  if (ndev <= 0) return;
  HIPOK(hipSetDevice(0));
  hipStream_t stream;
  HIPOK(hipStreamCreate(&stream));

  wdc_params p;
  wdc_params_default(&p);
  wdc_model_desc d = tiny_desc();
  wdc_ctx *ctx = NULL;
  OK(wdc_create(&d, &p, (wdc_stream)stream, &ctx));
  if (!ctx) return;
  ctx_for_err = ctx;
  void *w = NULL, *ws = NULL, *sm[2] = {NULL, NULL};
  const size_t wb = wdc_weights_bytes(ctx), wsb = wdc_workspace_bytes(ctx), sb = wdc_state_bytes(ctx);
  HIPOK(hipMalloc(&w, wb));
  HIPOK(hipMalloc(&ws, wsb));
  OK(wdc_init_weights_random(ctx, w, wb, 42, 0.02f));
  OK(wdc_bind_weights(ctx, w, wb));
  EXPECT(wdc_bind_workspace(ctx, ws, wsb - 256) != WDC_OK, "short workspace accepted");
  OK(wdc_bind_workspace(ctx, ws, wsb));
  wdc_state *st[2] = {NULL, NULL};
  for (int b = 0; b < 2; ++b) {
    HIPOK(hipMalloc(&sm[b], sb));
    OK(wdc_state_create(ctx, sm[b], sb, &st[b]));
  }

  const size_t E = (size_t)d.lat_c * d.lat_f * d.lat_h * d.lat_w;
  const int S = 8;
  float *z0 = (float *)dev_fill(E), *z = NULL, *zhat = NULL, *v = NULL, *zn = NULL;
  void *cond = dev_fill((size_t)d.cond_dim);
  HIPOK(hipMalloc((void **)&z, E * sizeof(float)));
  HIPOK(hipMalloc((void **)&zhat, E * sizeof(float)));
  HIPOK(hipMalloc((void **)&v, E * sizeof(float)));
  HIPOK(hipMalloc((void **)&zn, E * sizeof(float)));

  /* the whole rollout in every mode, with logs */
  uint8_t sched[8], forced[8] = {0, 1, 1, 0, 1, 1, 1, 0};
  wdc_step_log logs[8];
  const int modes[4] = {WDC_MODE_RISK, WDC_MODE_FORCED, WDC_MODE_ALL_EXACT, WDC_MODE_PERIODIC};
  for (int m = 0; m < 4; ++m) {
    HIPOK(hipMemcpy(z, z0, E * sizeof(float), hipMemcpyDeviceToDevice));
    OK(wdc_rollout(ctx, st[0], z, S, cond, NULL, NULL, modes[m], modes[m] == WDC_MODE_FORCED ? forced : NULL,
                   NULL, sched, logs));
    EXPECT(all_finite(z, E), "mode %d: non-finite latent", modes[m]);
    EXPECT(sched[0] == 0, "mode %d: step 0 not exact", modes[m]);
    for (int k = 0; k < S; ++k) EXPECT(logs[k].k == k && (sched[k] == 0 || sched[k] == 1), "log %d", k);
  }
  EXPECT(wdc_rollout(ctx, st[0], z, S, cond, NULL, NULL, WDC_MODE_FORCED, NULL, NULL, sched, logs) != WDC_OK,
         "forced mode without a mask accepted");

  /* the same loop through the step calls, alternating the allocation-free
   * candidate call with the ordinary one */
  HIPOK(hipMemcpy(z, z0, E * sizeof(float), hipMemcpyDeviceToDevice));
  OK(wdc_state_reset(st[1], NULL));
  for (int k = 0; k < S; ++k) {
    wdc_step_log lg;
    memset(&lg, 0, sizeof lg);
    if (k % 2)
      OK(wdc_surrogate_step_noalloc(ctx, st[1], z, k, S, zhat, &lg));
    else
      OK(wdc_surrogate_step(ctx, st[1], z, k, S, zhat, &lg));
    OK(wdc_risk_update(ctx, st[1], WDC_PRE_DECISION, k, S, NULL, NULL, &lg));
    const double t = (double)(S - k) / S, tn = (double)(S - k - 1) / S;
    if (lg.exact) {
      OK(wdc_dit_forward(ctx, z, t, cond, NULL, NULL, v));
      OK(wdc_scheduler_step(ctx, z, v, t, tn, zn, (int64_t)E));
      OK(wdc_risk_update(ctx, st[1], WDC_POST_EXACT, k, S, z, zn, &lg));
      HIPOK(hipMemcpy(z, zn, E * sizeof(float), hipMemcpyDeviceToDevice));
    } else {
      OK(wdc_risk_update(ctx, st[1], WDC_POST_SURROGATE, k, S, NULL, NULL, &lg));
      HIPOK(hipMemcpy(z, zhat, E * sizeof(float), hipMemcpyDeviceToDevice));
    }
  }
  EXPECT(all_finite(z, E), "step calls: non-finite latent");
  float *slot = NULL;
  int32_t inserts = 0;
  OK(wdc_state_bank_slot(st[1], 0, &slot, &inserts));
  EXPECT(slot != NULL && inserts >= 1, "bank slot");
  EXPECT(wdc_state_bank_slot(st[1], WDC_MAX_BANK, &slot, &inserts) != WDC_OK, "bank slot past the end accepted");

  /* batched rollouts and forward */
  float *zs[2];
  const float *zsc[2];
  float *vs[2];
  const void *conds[2] = {cond, cond};
  uint8_t scheds[16];
  wdc_step_log blogs[16];
  for (int b = 0; b < 2; ++b) {
    HIPOK(hipMalloc((void **)&zs[b], E * sizeof(float)));
    HIPOK(hipMalloc((void **)&vs[b], E * sizeof(float)));
    HIPOK(hipMemcpy(zs[b], z0, E * sizeof(float), hipMemcpyDeviceToDevice));
    zsc[b] = zs[b];
  }
  OK(wdc_rollout_batch(ctx, st, 2, zs, S, conds, NULL, NULL, WDC_MODE_RISK, NULL, NULL, scheds, blogs));
  OK(wdc_dit_forward_batch(ctx, 2, zsc, 0.3, conds, NULL, NULL, vs));
  for (int b = 0; b < 2; ++b) EXPECT(all_finite(zs[b], E) && all_finite(vs[b], E), "batch sample %d", b);
  EXPECT(wdc_rollout_batch(ctx, st, 3, zs, S, conds, NULL, NULL, WDC_MODE_RISK, NULL, NULL, scheds, blogs) !=
             WDC_OK, "batch past max_batch accepted");

  /* conditioning, one block, the kernels alone, timing */
  const int64_t N = (int64_t)(d.lat_f / d.patch_t) * (d.lat_h / d.patch_h) * (d.lat_w / d.patch_w);
  float *cemb = NULL, *x = (float *)dev_fill((size_t)N * d.hidden);
  HIPOK(hipMalloc((void **)&cemb, d.hidden * sizeof(float)));
  OK(wdc_set_timing(ctx, 1));
  OK(wdc_cond_embed(ctx, 0.6, cond, NULL, cemb));
  OK(wdc_dit_block_forward(ctx, 1, x, cemb));
  EXPECT(wdc_dit_block_forward(ctx, 2, x, cemb) != WDC_OK, "block index past the end accepted");
  EXPECT(all_finite(x, (size_t)N * d.hidden), "block output");
  const int64_t np = wdc_attn_pad(N);
  float *q = (float *)dev_fill((size_t)d.heads * np * d.head_dim), *o = NULL;
  HIPOK(hipMalloc((void **)&o, (size_t)N * d.hidden * sizeof(float)));
  OK(wdc_attention(ctx, q, q, q, N, o, d.hidden));
  int32_t qbm = -1, ks = -1;
  OK(wdc_attention_plan(ctx, N, &qbm, &ks));
  EXPECT(qbm >= 0 && qbm <= (int32_t)(np / 256) && ks >= 1 && ks <= 8, "attention plan %d blocks, %d ranges", (int)qbm,
         (int)ks);
  EXPECT(wdc_attention(ctx, q, q, q, N, o, d.hidden - 1) == WDC_E_ARG, "overlapping output rows accepted");
  EXPECT(wdc_attention(ctx, (const char *)q + 4, q, q, N, o, d.hidden) == WDC_E_ALIGN, "misaligned q accepted");
  OK(wdc_linear(ctx, x, d.hidden, w, NULL, o, d.hidden, N, d.hidden, d.hidden));
  double ms[WDC_T_COUNT], work[WDC_T_COUNT];
  int64_t cnt[WDC_T_COUNT];
  OK(wdc_timing(ctx, ms, cnt, work));
  EXPECT(cnt[WDC_T_ATTENTION] >= 2 && cnt[WDC_T_GEMM] >= 1 && ms[WDC_T_GEMM] > 0.0, "timing counts");
  OK(wdc_set_timing(ctx, 0));

  HIPOK(hipStreamSynchronize(stream));
  for (int b = 0; b < 2; ++b) {
    OK(wdc_state_destroy(st[b]));
    HIPOK(hipFree(sm[b]));
    HIPOK(hipFree(zs[b]));
    HIPOK(hipFree(vs[b]));
  }
  ctx_for_err = NULL;
  OK(wdc_destroy(ctx));
  void *bufs[] = {w, ws, z0, z, zhat, v, zn, cond, cemb, x, q, o};
  for (size_t i = 0; i < sizeof bufs / sizeof bufs[0]; ++i) HIPOK(hipFree(bufs[i]));

  /* the bf16 model with every block kind: one forward through the C ABI */
  d = joint_desc();
  OK(wdc_create(&d, &p, (wdc_stream)stream, &ctx));
  if (ctx) {
    ctx_for_err = ctx;
    const size_t wb2 = wdc_weights_bytes(ctx), wsb2 = wdc_workspace_bytes(ctx);
    HIPOK(hipMalloc(&w, wb2));
    HIPOK(hipMalloc(&ws, wsb2));
    OK(wdc_init_weights_random(ctx, w, wb2, 7, 0.02f));
    OK(wdc_bind_weights(ctx, w, wb2));
    OK(wdc_bind_workspace(ctx, ws, wsb2));
    const size_t E2 = (size_t)d.lat_c * d.lat_f * d.lat_h * d.lat_w;
    void *z2 = dev_fill(E2), *v2 = NULL, *cond2 = dev_fill_bf16(64), *text2 = dev_fill_bf16(21 * 128),
         *cam2 = dev_fill_bf16(96);
    HIPOK(hipMalloc(&v2, E2 * sizeof(float)));
    OK(wdc_dit_forward(ctx, (const float *)z2, 0.45, cond2, text2, cam2, (float *)v2));
    EXPECT(all_finite(v2, E2), "bf16 forward");
    ctx_for_err = NULL;
    OK(wdc_destroy(ctx));
    void *bufs2[] = {w, ws, z2, v2, cond2, text2, cam2};
    for (size_t i = 0; i < sizeof bufs2 / sizeof bufs2[0]; ++i) HIPOK(hipFree(bufs2[i]));
  }
  HIPOK(hipStreamDestroy(stream));
}

int main(int argc, char **argv) {
  const int gpu = argc > 1 && strcmp(argv[1], "gpu") == 0;
  setvbuf(stdout, NULL, _IONBF, 0);  /* the verdict line survives an exit forced by the sanitizers */
  host_checks();
  if (gpu) gpu_checks();
  if (g_fail) {
    fprintf(stderr, "abi_driver: FAILED\n");
    return 1;
  }
  printf("abi_driver %s: ok\n", gpu ? "gpu" : "cpu");
  return 0;
}

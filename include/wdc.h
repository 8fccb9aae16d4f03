/*
 * wdc.h -- C ABI of the WorldDynCache denoising-rollout library for MI355X (gfx950).
 *
 * The library runs the rollout of Eq. (1) of "WorldDynCache: Risk-Controlled
 * Latent Dynamics Approximation for Diffusion World Models":
 *     exact step      z_{t-1} = Psi_t(z_t, F_theta(z_t, t, c))
 *     surrogate step  z_hat_{t-1} = G_t(z_t, H_t)
 * with F_theta a synthetic video diffusion transformer (the paper does not fix
 * its architecture), Psi_t the flow-matching Euler step, G_t the lifted latent
 * surrogate of Eq. (2)-(5) and the choice between them made by the transition
 * risk controller of Eq. (6)-(10).
 *
 * Conventions shared by every call
 *  - Pointers prefixed d_ are device pointers, h_ host pointers. The caller owns
 *    every buffer; the library borrows them for the duration of the call and
 *    never frees them. Device buffers must be 16-byte aligned (E_ALIGN).
 *  - Element types: float32, or bfloat16 passed as raw uint16 bit patterns
 *    ("model dtype" = the dtype field of the model descriptor).
 *  - Work is enqueued on the context's stream. Calls returning host-side
 *    decisions (wdc_surrogate_step, wdc_risk_update, wdc_rollout) synchronise
 *    that stream before they return; the others are asynchronous.
 *  - Every call returns wdc_status; nothing throws across the ABI. After a
 *    failure wdc_last_error() describes it. One context serves one host thread.
 */
#ifndef WDC_H_
#define WDC_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct wdc_ctx wdc_ctx;
typedef struct wdc_state wdc_state;
typedef void *wdc_stream; /* a hipStream_t; NULL = the null stream */

typedef enum {
  WDC_OK = 0,
  WDC_E_ARG = 1,         /* null pointer or out-of-range argument */
  WDC_E_SHAPE = 2,       /* sizes inconsistent with the model descriptor */
  WDC_E_DTYPE = 3,       /* unsupported element type */
  WDC_E_ALIGN = 4,       /* device pointer not 16-byte aligned */
  WDC_E_WORKSPACE = 5,   /* workspace/weights not bound or too small */
  WDC_E_STATE = 6,       /* call not valid in the current state */
  WDC_E_HIP = 7,         /* a HIP runtime call failed */
  WDC_E_NONFINITE = 8,   /* a non-finite value where a finite one is required */
  WDC_E_UNSUPPORTED = 9  /* configuration the kernels do not cover */
} wdc_status;

enum { WDC_F32 = 0, WDC_BF16 = 1 };

/* Rollout modes. RISK: Eq. (10) as written. FORCED: the decision of step k is
 * h_forced[k] (1 = surrogate), still falling back to exact when the candidate is
 * unsupported (Sec. 4.3, last sentence of "Reliability Decision"). ALL_EXACT:
 * every step exact; candidates are still built and logged. PERIODIC: exact when
 * k mod params.period == 0, otherwise the surrogate whenever it is available
 * (the periodic placement of the ablation study, Sec. 5.4). */
enum { WDC_MODE_RISK = 0, WDC_MODE_FORCED = 1, WDC_MODE_ALL_EXACT = 2, WDC_MODE_PERIODIC = 3 };

/* Surrogate construction (wdc_params.surrogate). LIFTED: Eq. (2)-(5). SECANT:
 * native latent secant of the ablation study (Sec. 5.4): the latest exact
 * transition z_a -> z_out over phases q_a -> q_{a-1} extrapolated from z_t,
 * z_hat = z_t + (q_{t-1} - q_t) / (q_{a-1} - q_a) * (z_out - z_a). */
enum { WDC_SURROGATE_LIFTED = 0, WDC_SURROGATE_SECANT = 1 };

/* Observation (wdc_params.observation). KERNEL: Eq. (5). LINEAR: the evolved
 * lifted state is read back linearly by undoing the RMS normalisation of its
 * latent block, z_hat = rho(z_t) * (nu(z_t) + alpha * sum_{i in N_t} pi_i
 * (nu(z_i^out) - nu(z_i^in))), rho(x) = sqrt(mean(x^2) + eps_nu); the state then
 * also keeps each record's input latent. */
enum { WDC_OBS_KERNEL = 0, WDC_OBS_LINEAR = 1 };

/* Phases of wdc_risk_update. */
enum { WDC_PRE_DECISION = 0, WDC_POST_EXACT = 1, WDC_POST_SURROGATE = 2 };

/* Synthetic denoiser F_theta. The token grid is
 * (lat_f/patch_t, lat_h/patch_h, lat_w/patch_w); video token n = (f*H'+h)*W'+w;
 * text tokens follow the video tokens in the joint sequence. Blocks are
 * numbered globally: n_seq sequential, then n_dual dual-stream, then
 * n_single single-stream. rope_{t,h,w}: rotary dims per axis (sum = head_dim,
 * all 0 = no RoPE). */
typedef struct {
  int32_t dtype;      /* WDC_F32 or WDC_BF16: weights, activations, cond/text/cam inputs */
  int32_t hidden;     /* D */
  int32_t heads;
  int32_t head_dim;   /* 64 or 128 */
  int32_t mlp_ratio;  /* MLP width = mlp_ratio * D */
  int32_t n_seq, n_dual, n_single;
  int32_t cond_dim;   /* pooled condition length (0: none) */
  int32_t cam_dim;    /* camera/geometry vector length (0: none) */
  int32_t text_tokens, text_dim;
  int32_t lat_c, lat_f, lat_h, lat_w;
  int32_t patch_t, patch_h, patch_w;
  int32_t rope_t, rope_h, rope_w;
  int32_t qk_norm;    /* 1: per-head RMSNorm on q and k */
  int32_t max_batch;  /* most samples one batched forward takes (0 or 1: one); sizes the workspace */
} wdc_model_desc;

/* Constants of the method. The paper fixes the anchor-age limit (six) and the
 * cap of 2 on w_t; the rest are set in its supplementary material and are
 * readings here (wdc_params_default fills them). */
typedef struct {
  int32_t bank_capacity;            /* M, FIFO capacity of the exact-transition bank (<= WDC_MAX_BANK) */
  int32_t age_max, n_min, k_init, k_ref;
  double theta_sim, theta_q;        /* compatibility thresholds of N_t (Eq. (3)) */
  double tau_in, tau_obs, gamma_q;  /* temperatures and phase penalty (Eq. (3), (5)) */
  double alpha_min, alpha_max, eps; /* Eq. (4) */
  double eps_nu;                    /* RMS normalisation of Eq. (2) */
  double w_z, w_age, w_phase, w_cam, w_depth; /* Eq. (6) */
  double eta0, beta_d, eta_min, eta_max;      /* Eq. (8) */
  double a_cam, a_depth, a_phase, lam, r0;    /* Eq. (9) */
  double tau_risk;                            /* Eq. (10) */
  /* Variants of the ablation study (Sec. 5.4); the defaults are the full method. */
  int32_t period;             /* WDC_MODE_PERIODIC: exact when k mod period == 0 (>= 1) */
  int32_t surrogate;          /* WDC_SURROGATE_* */
  int32_t observation;        /* WDC_OBS_* */
  int32_t lift_condition;     /* 0: camera/depth blocks zero, retrieval without the phase terms of Eq. (3) */
  int32_t impact_weight;      /* 0: w_t = 1 (no future-impact weighting, Eq. (9)) */
  int32_t calibrate;          /* 0: eta_d stays at eta0 (no counterfactual calibration, Eq. (8)) */
  int32_t support_constraint; /* 0: availability does not require |N_t| >= n_min */
  int32_t pad_;
} wdc_params;

#define WDC_MAX_BANK 8
#define WDC_SUMMARY_DIM 256

/* Per-step record of the controller (one per denoising step). */
typedef struct {
  int32_t k, exact, bank, support, finite, available, slot;
  int32_t pad_;
  double t, alpha;
  double pi[WDC_MAX_BANK], kappa[WDC_MAX_BANK], sims_in[WDC_MAX_BANK]; /* slot order */
  double d_z, d_age, d_phase, p, d_hat, w, r_cand, margin, sim_margin;
  double d_cf, eta, R; /* d_cf is NaN when no supported counterfactual existed */
} wdc_step_log;

/* ---------------------------------------------------------------- context */

/* Fill *p with the default constants. */
void wdc_params_default(wdc_params *p);

/* Create a context for one model on one stream (the current HIP device).
 * desc may describe zero blocks (surrogate-only use). bf16: WDC_E_SHAPE if
 * the joint sequence (video + text tokens, padded) holds more than 2^30 bytes
 * per head of q, k or v (about 4.2 million tokens at head size 128): the bf16
 * attention kernel addresses one head's rows with 32-bit offsets. */
wdc_status wdc_create(const wdc_model_desc *desc, const wdc_params *params, wdc_stream stream, wdc_ctx **out);
wdc_status wdc_destroy(wdc_ctx *ctx);
/* Message of the last failure on this context ("" if none). ctx may be NULL
 * for failures of wdc_create. */
const char *wdc_last_error(const wdc_ctx *ctx);

/* Weights: one caller-allocated device blob of wdc_weights_bytes() bytes in the
 * model dtype. Tensor i (0 <= i < wdc_weight_count) has a name such as
 * "single.3.lin1.w", a shape (Linear weights are [out, in], biases [out]) and a
 * byte offset inside the blob (256-byte aligned). */
size_t wdc_weights_bytes(const wdc_ctx *ctx);
int32_t wdc_weight_count(const wdc_ctx *ctx);
wdc_status wdc_weight_info(const wdc_ctx *ctx, int32_t i, const char **name, int64_t shape[2], int32_t *ndim,
                           size_t *offset);
wdc_status wdc_bind_weights(wdc_ctx *ctx, const void *d_weights, size_t bytes);
/* Fill a weights blob with N(0, std^2) values from a counter-based generator
 * keyed by seed (throughput runs at sizes where host generation is too slow). */
wdc_status wdc_init_weights_random(wdc_ctx *ctx, void *d_weights, size_t bytes, uint64_t seed, float std);

/* Workspace for the denoiser and the rollout loop: caller-allocated device
 * memory of wdc_workspace_bytes() bytes, bound once. */
size_t wdc_workspace_bytes(const wdc_ctx *ctx);
wdc_status wdc_bind_workspace(wdc_ctx *ctx, void *d_ws, size_t bytes);

/* Rollout state: bank B_t (M exact output latents), anchor, history summary,
 * risk R, eta_d and counters (Sec. 4.2-4.3), plus the latents a rollout runs on. Its device memory
 * (wdc_state_bytes) is caller-allocated; the state object itself is freed by
 * wdc_state_destroy. h_cam: host float camera vector of cam_dim values for the
 * lifted state's camera descriptor, or NULL (descriptor zero). */
size_t wdc_state_bytes(const wdc_ctx *ctx);
wdc_status wdc_state_create(wdc_ctx *ctx, void *d_mem, size_t bytes, wdc_state **out);
wdc_status wdc_state_reset(wdc_state *st, const float *h_cam);
wdc_status wdc_state_destroy(wdc_state *st);
/* Bank introspection: device pointer of slot i's exact output latent, and the
 * number of records inserted so far. */
wdc_status wdc_state_bank_slot(wdc_state *st, int32_t i, float **d_slot, int32_t *inserts);

/* ---------------------------------------------------------------- denoiser F_theta */

/* c_emb = MLP(sinusoid(1000 t)) + Linear(cond) + Linear(cam): the conditioning
 * vector every block modulates from. d_cond [cond_dim], d_cam [cam_dim] in the
 * model dtype (NULL when the descriptor has none); d_cemb [D] float32 out. */
wdc_status wdc_cond_embed(wdc_ctx *ctx, double t, const void *d_cond, const void *d_cam, float *d_cemb);

/* One block (global index) of F_theta, in place on the joint residual stream.
 * d_x: [N_video + text_tokens, D] float32, video rows first; d_cemb: [D] float32.
 * Sequential blocks act on all rows with shared weights; dual-stream blocks
 * use per-stream weights for the video and text rows and one joint attention;
 * single-stream blocks use the fused linear1/linear2 form. */
wdc_status wdc_dit_block_forward(wdc_ctx *ctx, int32_t block, float *d_x, const float *d_cemb);

/* v = F_theta(z, t, c). d_z, d_v: [C, F, H, W] float32; d_cond/d_text/d_cam in
 * the model dtype (text [text_tokens, text_dim]), NULL when absent. */
wdc_status wdc_dit_forward(wdc_ctx *ctx, const float *d_z, double t, const void *d_cond, const void *d_text,
                           const void *d_cam, float *d_v);

/* Batched F_theta (Sec. 4.4 run for several rollouts at once): v_b =
 * F_theta(z_b, t, c_b) for b < B <= max_batch, all at the same t. Host arrays
 * of B device pointers; d_cond/d_text/d_cam may be NULL (no such input) or hold
 * one pointer per sample. The samples' tokens go through every GEMM as one
 * batch and through attention as one launch of B x heads; each sample keeps its
 * own conditioning, modulation and joint attention. Same result per sample as
 * wdc_dit_forward up to float32 summation order. */
wdc_status wdc_dit_forward_batch(wdc_ctx *ctx, int32_t B, const float *const *d_z, double t,
                                 const void *const *d_cond, const void *const *d_text, const void *const *d_cam,
                                 float *const *d_v);

/* ---------------------------------------------------------------- scheduler Psi_t */

/* Flow-matching Euler step of Eq. (1): z_next = z + (t_next - t_cur) * v,
 * numel float32 elements. d_z_next may equal d_z. */
wdc_status wdc_scheduler_step(wdc_ctx *ctx, const float *d_z, const float *d_v, double t_cur, double t_next,
                              float *d_z_next, int64_t numel);

/* ---------------------------------------------------------------- surrogate and risk */

/* Candidate of step k of an S-step rollout (t_k = (S-k)/S), Eq. (2)-(5):
 * lifts d_z with the state's anchor and history, retrieves compatible records,
 * evolves the lifted state and writes z_hat = sum_i kappa_i z_i^out into
 * d_zhat [numel of the latent]. With an empty bank nothing is written. The
 * candidate is kept in the state (d_zhat must stay valid until the matching
 * wdc_risk_update) and described in *h_log (candidate fields). */
wdc_status wdc_surrogate_step(wdc_ctx *ctx, wdc_state *st, const float *d_z, int32_t k, int32_t S, float *d_zhat,
                              wdc_step_log *h_log);

/* wdc_surrogate_step for callers that cannot allocate memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same kernels, host arithmetic, results and state update, with the
 * statistics kernels' partial sums and float64 reductions kept in one fixed
 * device array of the library (337,920 bytes per device, held until the
 * process ends) instead of the state's memory. It makes no device or pinned
 * host allocation and records no timing events. That array is shared by every
 * call on the device and keeps the last call's contents (each call overwrites
 * what it reads): calls that overlap on one device, from several streams or
 * threads, race. A latent whose statistics would not fit the array is
 * rejected with WDC_E_WORKSPACE (none does: 16 channels x 8 segments x 64
 * slices is the largest plan). Synchronises the stream like wdc_surrogate_step. */
wdc_status wdc_surrogate_step_noalloc(wdc_ctx *ctx, wdc_state *st, const float *d_z, int32_t k, int32_t S,
                                      float *d_zhat, wdc_step_log *h_log);

/* Transition risk controller, Eq. (6)-(10).
 * PRE_DECISION (after wdc_surrogate_step of the same k): proxy p_k, weight w_k,
 *   R_cand, availability and the decision; h_log->exact = 1 means Exact.
 * POST_EXACT: d_z_cur = z_k, d_z_next = the exact z_{k+1}; computes the
 *   counterfactual defect of the kept candidate (Eq. (7)), calibrates eta_d
 *   (Eq. (8)) when that candidate was supported, decays R, inserts the record
 *   (FIFO), moves the anchor to z_k and resets the surrogate count.
 * POST_SURROGATE: R <- R_cand, one more consecutive surrogate step.
 * Synchronises the stream. */
wdc_status wdc_risk_update(wdc_ctx *ctx, wdc_state *st, int32_t phase, int32_t k, int32_t S, const float *d_z_cur,
                           const float *d_z_next, wdc_step_log *h_log);

/* The whole rollout of Sec. 4.4: S steps from d_z (in: z_T, out: z_0).
 * mode: WDC_MODE_*; h_forced [S] (FORCED only); d_replay_v: NULL to evaluate
 * F_theta, or [S, C, F, H, W] float32 velocities used at exact steps in place
 * of F_theta. h_schedule [S] out: 0 = exact, 1 = surrogate; h_log [S] or NULL.
 * The state is reset at the start (camera descriptor from d_cam). */
wdc_status wdc_rollout(wdc_ctx *ctx, wdc_state *st, float *d_z, int32_t S, const void *d_cond, const void *d_text,
                       const void *d_cam, int32_t mode, const uint8_t *h_forced, const float *d_replay_v,
                       uint8_t *h_schedule, wdc_step_log *h_log);

/* B rollouts at once, each with its own state, latent, conditioning and
 * schedule (B <= max_batch). Every step runs each sample's candidate and
 * decision; the samples that take an exact step are evaluated by one batched
 * F_theta call (or their recorded velocities), the others commit their
 * candidates. Arrays: states[B]; d_z[B] (in: z_T, out: z_0); d_cond/d_text/d_cam
 * NULL or [B] pointers; h_forced [B][S] (FORCED only); d_replay_v NULL or [B]
 * pointers to [S, C, F, H, W] velocities; h_schedule [B][S]; h_log [B][S] or
 * NULL. Per sample the schedule, log and latent equal those of wdc_rollout on
 * that sample alone (latents up to float32 summation order). */
wdc_status wdc_rollout_batch(wdc_ctx *ctx, wdc_state *const *states, int32_t B, float *const *d_z, int32_t S,
                             const void *const *d_cond, const void *const *d_text, const void *const *d_cam,
                             int32_t mode, const uint8_t *h_forced, const float *const *d_replay_v,
                             uint8_t *h_schedule, wdc_step_log *h_log);

/* ---------------------------------------------------------------- kernels exposed for tests and benchmarks */

/* softmax(q k^T / sqrt(hd)) v over the full sequence, the attention of every
 * block. bf16: float32 accumulation, q multiplied by log2(e)/sqrt(hd) and
 * rounded to bf16 once in the kernel, attention weights rounded to bf16 before
 * the product with v and the row sum. d_q, d_k: [heads, n_pad, hd]. d_vt for bf16: [heads, hd, n_pad], V
 * transposed with the keys of each aligned group of 16 stored in the order
 * 0-3, 8-11, 4-7, 12-15 (key j at column j with bits 2 and 3 swapped); for
 * float32: [heads, n_pad, hd]. n valid tokens, n_pad = wdc_attn_pad(n); rows
 * (keys) >= n of q/k/v must be zero. d_o: [n, ldo], head h written at columns
 * [h*hd, (h+1)*hd); ldo >= heads*hd (else WDC_E_ARG). q, k, vt 16-byte
 * aligned; for bf16 d_o 8-byte aligned and ldo a multiple of 4 (else
 * WDC_E_ALIGN); bf16 with n_pad * hd * 2 above 2^30 bytes (32-bit offsets
 * within a head) is WDC_E_SHAPE. bf16 may use the bound workspace as scratch
 * (wdc_attention_plan), so q, k, vt and o must not lie in it. */
int64_t wdc_attn_pad(int64_t n);
wdc_status wdc_attention(wdc_ctx *ctx, const void *d_q, const void *d_k, const void *d_vt, int64_t n, void *d_o,
                         int64_t ldo);
/* How the bf16 attention of this context runs n tokens (one sample, the
 * context's heads): query blocks of 256 per head that run over all keys
 * (*qb_main), and the number of key ranges (*kv_splits, 1 = none) each of
 * the remaining blocks of the last, partly filled dispatch round runs as;
 * those ranges are combined by a second launch. A split uses the bound
 * workspace's projection area as scratch (its contents are not kept), so
 * without a workspace, or when it is too small, *kv_splits is 1. The
 * environment variable WDC_ATTN_SPLITS, read at wdc_create, overrides the
 * estimate (1: never split; s >= 2: s ranges whenever a round is partial,
 * at most one per key tile). Float32 contexts: *qb_main = every block,
 * *kv_splits = 1. Either output may be NULL. */
wdc_status wdc_attention_plan(const wdc_ctx *ctx, int64_t n, int32_t *qb_main, int32_t *kv_splits);

/* c[m, n] = sum_k a[m, k] * w[n, k] + bias[n] in the model dtype with float32
 * accumulation; a row stride lda, c row stride ldc. */
wdc_status wdc_linear(wdc_ctx *ctx, const void *d_a, int64_t lda, const void *d_w, const void *d_bias, void *d_c,
                      int64_t ldc, int64_t m, int64_t n, int64_t k);

/* Kernel timing for benchmarks. While timing is on (wdc_set_timing(ctx, 1),
 * which also clears the totals), every launch of the classes below on the
 * context's stream is bracketed by HIP events; wdc_timing synchronises the
 * stream and returns, per class, the summed milliseconds, the number of
 * launches and (out_work, may be NULL) the summed algorithmic work of those
 * launches: FLOPs for the matrix classes (attention 4 n^2 hd per head, GEMM
 * 2 m n k), bytes that must cross HBM for the streaming classes (each input
 * read once, each output written once). Off by default (no events). */
enum {
  WDC_T_ATTENTION = 0,  /* flash attention */
  WDC_T_GEMM = 1,       /* linear layers */
  WDC_T_STATS = 2,      /* pass-1 lift statistics of a latent (Eq. (2), (6)) */
  WDC_T_OBSERVE = 3,    /* kernel observation combine (Eq. (5)) */
  WDC_T_EXACT_POST = 4, /* exact-step epilogue: Psi, counterfactual sums, bank and anchor writes */
  WDC_T_PSI = 5,        /* standalone scheduler step (wdc_scheduler_step) */
  WDC_T_NORM = 6,       /* LayerNorm + modulation of the residual stream */
  WDC_T_COUNT = 7
};
wdc_status wdc_set_timing(wdc_ctx *ctx, int32_t on);
wdc_status wdc_timing(wdc_ctx *ctx, double out_ms[WDC_T_COUNT], int64_t out_count[WDC_T_COUNT],
                      double out_work[WDC_T_COUNT]);

#ifdef __cplusplus
}
#endif
#endif /* WDC_H_ */

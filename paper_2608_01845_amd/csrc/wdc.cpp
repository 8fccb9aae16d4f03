// Host side of the WorldDynCache rollout library: context, weight layout,
// workspace, the denoiser's launch sequence, and the surrogate / risk-controller
// state machine (host float64 scalars) behind the C ABI of include/wdc.h.
#include "../../include/wdc.h"
#include "common.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <string>
#include <vector>

using namespace wdc;

namespace {
constexpr int S_DIM = WDC_SUMMARY_DIM;
constexpr int G8 = 8, G4 = 4, G2 = 2, GCAM = 16;

struct TensorInfo {
  std::string name;
  int64_t shape[2];
  int ndim;
  size_t offset, numel;
};

struct TimedEvent {
  hipEvent_t a, b;
  int cls;
};
}  // namespace

struct wdc_ctx {
  wdc_model_desc d{};
  wdc_params p{};
  hipStream_t stream = nullptr;
  std::string err;
  int esz = 4;
  // derived shapes
  int64_t nv = 0, nt = 0, n = 0, n_pad = 0, E = 0, T = 0;
  int mb = 1;  // most samples of one batched forward (workspace sizing)
  int nb = 1;  // samples of the forward in progress
  int P = 0, D = 0, H = 0, hd = 0, F = 0;
  // weights
  std::vector<TensorInfo> tensors;
  std::map<std::string, int> index;
  size_t wbytes = 0;
  const char *w = nullptr;
  // workspace
  char *ws = nullptr;
  size_t ws_need = 0, ws_bytes = 0;
  float *x = nullptr, *mod = nullptr, *cemb = nullptr, *tfeat = nullptr, *tmp = nullptr, *cvec = nullptr;
  void *h = nullptr, *qkv = nullptr, *cat = nullptr, *q = nullptr, *k = nullptr, *v = nullptr, *patches = nullptr;
  float *tok = nullptr;
  float2 *rope = nullptr;
  float *r_v = nullptr;  // [mb, E] velocities of a batched forward inside a rollout
  // q/k/v preparation in the projection's epilogue where the GEMM allows it
  // (WDC_FUSE_QKV=0: always the separate kernels, for comparison)
  bool fuse_qkv = true;
  // products that would not fill one dispatch round of 256 x 256 tiles run on
  // 128 x 128 tiles (WDC_FILL_TILES=0: tile size by shape alone, so tests can
  // reach the 256 x 256 kernels and the fused q/k/v epilogue at small sizes)
  bool fill_tiles = true;
  // key-range split of the attention's last partial dispatch round
  // (WDC_ATTN_SPLITS: unset or 0 by the cost estimate, 1 never, s >= 2 always
  // s ranges, for tests)
  int attn_splits = 0;
  size_t qkv_bytes = 0;  // the projection buffer, scratch of the split attention
  // timing
  bool timing = false;
  std::vector<TimedEvent> events;
  double t_ms[WDC_T_COUNT] = {};
  int64_t t_cnt[WDC_T_COUNT] = {};
  double t_work[WDC_T_COUNT] = {};
};

namespace {
struct Record {
  double s_in[S_DIM], s_out[S_DIM];
  double q_in, q_out;
  double rho_in, rho_out;  // sqrt(mean(z^2) + eps_nu) of the input and output latents
};
}  // namespace

struct wdc_state {
  wdc_ctx *ctx = nullptr;
  SegPlan plan{};
  float *anchor[2] = {nullptr, nullptr};
  int acur = 0;
  bool has_anchor = false;
  double q_a = 0, q_am1 = 0;
  float *bank[WDC_MAX_BANK] = {};
  float *bank_in[WDC_MAX_BANK] = {};  // input latents of the records (linear observation only)
  Record rec[WDC_MAX_BANK];
  bool filled[WDC_MAX_BANK] = {};
  int inserts = 0;
  double hsum[32];
  double cam[GCAM];
  double R = 0, eta = 1;
  int n_s = 0;
  float *rz[3] = {nullptr, nullptr, nullptr};  // current latent, candidate, next exact latent of a rollout
  float *partials = nullptr;
  double *d_red = nullptr;
  double *h_red = nullptr;  // pinned host
  std::vector<double> n8;   // element count of each fine segment [C*8]
  // pass-1 statistics [nseg, PRE_NV] of the latent the next step starts from,
  // emitted by the kernel that produced it (observation or exact epilogue);
  // only the rollout loop, which owns that latent, reads them
  std::vector<double> pre_obs, pre_post;
  // pending pre-decision data of step k
  int pend_k = -1;
  bool pend_cand = false;   // a candidate exists (bank non-empty)
  const float *pend_zhat = nullptr;
  int pend_support = 0;
  bool pend_finite = false;
  double s_phi[S_DIM];
  double rho_cur = 0;  // sqrt(mean(z_k^2) + eps_nu) of the pending step's latent
  double proxy = 0, r_cand = 0, d_hat = 0, wgt = 1, margin = 0;
  bool pend_avail = false, pend_decided = false, pend_surrogate = false;
};

namespace {

void set_err(wdc_ctx *c, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  if (c) c->err = buf;
}

thread_local std::string g_create_err;

#define HIPCHK(ctx, expr)                                                                  \
  do {                                                                                     \
    hipError_t e_ = (expr);                                                                \
    if (e_ != hipSuccess) {                                                                \
      set_err(ctx, "%s failed: %s (%s:%d)", #expr, hipGetErrorString(e_), __FILE__, __LINE__); \
      return WDC_E_HIP;                                                                    \
    }                                                                                      \
  } while (0)

#define CHK(expr)                    \
  do {                               \
    wdc_status s_ = (expr);          \
    if (s_ != WDC_OK) return s_;     \
  } while (0)

bool aligned16(const void *p) { return ((uintptr_t)p & 15) == 0; }

double t_at(int k, int S) { return (double)(S - k) / (double)S; }

// ---------------------------------------------------------------- weights
void add_tensor(wdc_ctx *c, const std::string &name, int64_t d0, int64_t d1) {
  TensorInfo t;
  t.name = name;
  t.shape[0] = d0;
  t.shape[1] = d1;
  t.ndim = d1 > 0 ? 2 : 1;
  t.numel = (size_t)d0 * (size_t)(d1 > 0 ? d1 : 1);
  t.offset = c->wbytes;
  c->wbytes += ((t.numel * c->esz + 255) / 256) * 256;
  c->index[name] = (int)c->tensors.size();
  c->tensors.push_back(t);
}

void add_linear(wdc_ctx *c, const std::string &name, int64_t out, int64_t in) {
  add_tensor(c, name + ".w", out, in);
  add_tensor(c, name + ".b", out, 0);
}

void build_layout(wdc_ctx *c) {
  const int64_t d = c->D, f = (int64_t)c->d.mlp_ratio * c->D;
  add_linear(c, "t_embed.fc1", d, 256);
  add_linear(c, "t_embed.fc2", d, d);
  if (c->d.cond_dim) add_linear(c, "cond_embed", d, c->d.cond_dim);
  if (c->d.cam_dim) add_linear(c, "cam_embed", d, c->d.cam_dim);
  if (c->d.text_tokens) add_linear(c, "text_proj", d, c->d.text_dim);
  add_linear(c, "patch_embed", d, c->P);
  for (int i = 0; i < c->d.n_seq; ++i) {
    std::string pre = "seq." + std::to_string(i);
    add_linear(c, pre + ".ada", 6 * d, d);
    add_linear(c, pre + ".qkv", 3 * d, d);
    add_linear(c, pre + ".out", d, d);
    add_linear(c, pre + ".fc1", f, d);
    add_linear(c, pre + ".fc2", d, f);
  }
  for (int i = 0; i < c->d.n_dual; ++i)
    for (const char *s : {"vid", "txt"}) {
      std::string pre = "dual." + std::to_string(i) + "." + s;
      add_linear(c, pre + ".ada", 6 * d, d);
      add_linear(c, pre + ".qkv", 3 * d, d);
      add_linear(c, pre + ".out", d, d);
      add_linear(c, pre + ".fc1", f, d);
      add_linear(c, pre + ".fc2", d, f);
    }
  for (int i = 0; i < c->d.n_single; ++i) {
    std::string pre = "single." + std::to_string(i);
    add_linear(c, pre + ".ada", 3 * d, d);
    add_linear(c, pre + ".lin1", 3 * d + f, d);
    add_linear(c, pre + ".lin2", d, d + f);
  }
  add_linear(c, "final.ada", 2 * d, d);
  add_linear(c, "final.lin", c->P, d);
}

const void *W(wdc_ctx *c, const std::string &name) {
  auto it = c->index.find(name);
  if (it == c->index.end() || !c->w) return nullptr;
  return c->w + c->tensors[it->second].offset;
}

// ---------------------------------------------------------------- workspace
struct Carve {
  size_t off = 0;
  size_t take(size_t bytes) {
    size_t o = off;
    off += ((bytes + 255) / 256) * 256;
    return o;
  }
};

struct WsLayout {
  size_t x, h, qkv, cat, q, k, v, mod, cemb, tfeat, tmp, cvec, patches, tok, rope, rv, total;
};

// per-sample stride of the modulation vectors (dual blocks use 12 D)
int64_t mod_stride(const wdc_ctx *c) { return 12 * (int64_t)c->D; }

WsLayout ws_layout(const wdc_ctx *c) {
  WsLayout L;
  Carve cv;
  const size_t e = c->esz, D = c->D, B = c->mb, N = c->n * B;
  const size_t f = (size_t)c->d.mlp_ratio * D;
  const size_t E = c->E;
  L.x = cv.take(N * D * 4);
  L.h = cv.take(N * D * e);
  L.qkv = cv.take(N * 3 * D * e);
  L.cat = cv.take(N * (D + f) * e);
  size_t qk = B * c->H * c->n_pad * c->hd * e;
  L.q = cv.take(qk);
  L.k = cv.take(qk);
  L.v = cv.take(qk);
  L.mod = cv.take(B * mod_stride(c) * 4);
  L.cemb = cv.take(B * D * 4);
  L.tfeat = cv.take(256 * 4);
  L.tmp = cv.take(D * 4);
  size_t cdim = std::max({(size_t)c->d.cond_dim, (size_t)c->d.cam_dim, (size_t)1});
  L.cvec = cv.take(cdim * 4);
  L.patches = cv.take(B * c->nv * c->P * e);
  L.tok = cv.take(B * c->nv * c->P * 4);
  L.rope = cv.take((size_t)c->nv * (c->hd / 2) * 8);
  L.rv = cv.take(B * E * 4);
  L.total = cv.off;
  return L;
}

// ---------------------------------------------------------------- timing
// work: algorithmic FLOPs (matrix classes) or HBM bytes (streaming classes) of the launch
template <typename F>
hipError_t timed(wdc_ctx *c, int cls, double work, F &&fn) {
  if (!c->timing) return fn();
  TimedEvent ev{};
  ev.cls = cls;
  hipError_t e = hipEventCreate(&ev.a);
  if (e != hipSuccess) return e;
  if ((e = hipEventCreate(&ev.b)) != hipSuccess || (e = hipEventRecord(ev.a, c->stream)) != hipSuccess) {
    (void)hipEventDestroy(ev.a);
    if (ev.b) (void)hipEventDestroy(ev.b);
    return e;
  }
  e = fn();
  const hipError_t r = hipEventRecord(ev.b, c->stream);
  c->events.push_back(ev);  // released by wdc_timing, wdc_set_timing or wdc_destroy
  c->t_work[cls] += work;
  return e != hipSuccess ? e : r;
}

void release_events(wdc_ctx *c) {
  for (auto &e : c->events) {
    (void)hipEventDestroy(e.a);
    (void)hipEventDestroy(e.b);
  }
  c->events.clear();
}

// ---------------------------------------------------------------- kernel wrappers
char *elem(wdc_ctx *c, void *base, int64_t off) { return (char *)base + off * c->esz; }
const char *elem(wdc_ctx *c, const void *base, int64_t off) { return (const char *)base + off * c->esz; }

// a batch of n products sharing weights; strides in elements (gate in floats)
struct Batch {
  int n = 1;
  int64_t a_bs = 0, c_bs = 0, gate_bs = 0;
};

wdc_status gemm(wdc_ctx *c, const void *a, int64_t lda, const void *w, const void *b, void *out, int64_t ldc,
                int64_t m, int64_t n, int64_t k, int epi, const float *gate = nullptr, Batch bt = Batch()) {
  if (m <= 0 || bt.n <= 0) return WDC_OK;
  if (!w) {
    set_err(c, "weights not bound");
    return WDC_E_WORKSPACE;
  }
  GemmArgs g{};
  g.a = a;
  g.w = w;
  g.bias = b;
  g.c = out;
  g.gate = gate;
  g.lda = lda;
  g.ldc = ldc;
  g.m = m;
  g.n = n;
  g.k = k;
  g.epi = epi;
  g.batch = bt.n;
  g.a_bs = bt.a_bs;
  g.c_bs = bt.c_bs;
  g.gate_bs = bt.gate_bs;
  g.fill_tiles = c->fill_tiles;
  HIPCHK(c, timed(c, WDC_T_GEMM, 2.0 * m * n * k * bt.n, [&] { return launch_gemm(c->d.dtype, g, c->stream); }));
  return WDC_OK;
}

wdc_status gemv(wdc_ctx *c, const std::string &name, const float *x, float *y, int silu_in, int acc) {
  const auto &t = c->tensors[c->index.at(name + ".w")];
  const void *w = W(c, name + ".w"), *b = W(c, name + ".b");
  if (!w) {
    set_err(c, "weights not bound");
    return WDC_E_WORKSPACE;
  }
  HIPCHK(c, launch_gemv(c->d.dtype, w, b, x, y, (int)t.shape[0], (int)t.shape[1], silu_in, acc, c->stream));
  return WDC_OK;
}

// the modulation GEMV of every sample: y_b = W SiLU(cemb_b) + b, at mod + b * mod_stride + off
wdc_status mod_gemv(wdc_ctx *c, const std::string &name, int64_t off) {
  for (int b = 0; b < c->nb; ++b)
    CHK(gemv(c, name, c->cemb + (int64_t)b * c->D, c->mod + b * mod_stride(c) + off, 1, 0));
  return WDC_OK;
}

// The projection buffer is free while attention runs (q, k and v^T are in
// their own buffers by then): scratch for the split of the last round.
void attn_scratch(const wdc_ctx *c, AttnArgs &a) {
  a.part = c->ws ? (float *)c->qkv : nullptr;
  a.part_bytes = c->ws ? c->qkv_bytes : 0;
  a.force_splits = c->attn_splits;
}

// joint attention of every sample: q/k/v hold nb x H heads, O rows follow the samples
wdc_status attention(wdc_ctx *c, void *o, int64_t ldo) {
  const int hb = c->H * c->nb;
  HIPCHK(c, launch_qkv_pad(c->d.dtype, c->q, c->k, c->v, hb, c->hd, c->n, c->n_pad, c->stream));
  AttnArgs a{};
  a.q = c->q;
  a.k = c->k;
  a.v = c->v;
  a.o = o;
  a.n = c->n;
  a.n_pad = c->n_pad;
  a.ldo = ldo;
  a.heads = hb;
  a.hd = c->hd;
  a.hpb = c->H;
  attn_scratch(c, a);
  const double aw = 4.0 * (double)c->n * (double)c->n * c->hd * hb;
  HIPCHK(c, timed(c, WDC_T_ATTENTION, aw, [&] { return launch_attention(c->d.dtype, a, c->stream); }));
  return WDC_OK;
}

// q/k/v of every sample from the fused projection rows [row0, row0 + rows) of
// each sample (row stride ld) into the attention layouts of its heads
wdc_status qkv_prep(wdc_ctx *c, const void *src, int64_t ld, int64_t row0, int64_t rows) {
  const int64_t hs = (int64_t)c->H * c->n_pad * c->hd;  // elements per sample of q/k/v
  for (int b = 0; b < c->nb; ++b) {
    QKVPrepArgs a;
    a.src = elem(c, src, (int64_t)b * c->n * ld);
    a.ld = ld;
    a.row0 = row0;
    a.rows = rows;
    a.n_video = c->nv;
    a.n_pad = c->n_pad;
    a.q = elem(c, c->q, b * hs);
    a.k = elem(c, c->k, b * hs);
    a.v = elem(c, c->v, b * hs);
    a.heads = c->H;
    a.hd = c->hd;
    a.d = c->D;
    a.qk_norm = c->d.qk_norm;
    a.rope = (c->d.rope_t + c->d.rope_h + c->d.rope_w) ? c->rope : nullptr;
    HIPCHK(c, launch_qkv_prep(c->d.dtype, a, c->stream));
  }
  return WDC_OK;
}

// q/k/v projection of the modulated rows [row0, row0 + rows) of every sample
// (a: the first of them, row stride D). batched: one batch entry per sample
// (sample stride N rows); else one product over all samples' rows (row0 = 0,
// rows = N). The 256 x 256 GEMM writes q, k and v^T straight into the
// attention layouts (per-head RMSNorm and RoPE in its epilogue); products it
// does not run (few rows) take the plain GEMM into the qkv buffer and the
// separate preparation kernels, with the same arithmetic.
wdc_status qkv_project(wdc_ctx *c, const void *a, const void *w, const void *bias, int64_t row0, int64_t rows,
                       bool batched) {
  const int64_t D = c->D, N = c->n, NB = c->nb;
  if (!w) {
    set_err(c, "weights not bound");
    return WDC_E_WORKSPACE;
  }
  GemmArgs g{};
  g.a = a;
  g.w = w;
  g.bias = bias;
  g.lda = D;
  g.ldc = 3 * D;
  g.m = batched ? rows : NB * rows;
  g.n = 3 * D;
  g.k = D;
  g.epi = EPI_QKV;
  g.fill_tiles = c->fill_tiles;
  g.batch = batched ? (int)NB : 1;
  g.a_bs = batched ? N * D : 0;
  QkvOut &o = g.qkv;
  o.q = c->q;
  o.k = c->k;
  o.v = c->v;
  o.rope = (c->d.rope_t + c->d.rope_h + c->d.rope_w) ? c->rope : nullptr;
  o.n_pad = c->n_pad;
  o.n_video = c->nv;
  o.rps = batched ? rows : N;
  o.row0 = row0;
  o.heads = c->H;
  o.hd = c->hd;
  o.d = (int)D;
  o.qk_norm = c->d.qk_norm;
  if (c->fuse_qkv && gemm_qkv_fusable(c->d.dtype, g)) {
    HIPCHK(c, timed(c, WDC_T_GEMM, 2.0 * g.m * g.n * g.k * g.batch, [&] { return launch_gemm(c->d.dtype, g, c->stream); }));
    return WDC_OK;
  }
  void *out = elem(c, c->qkv, row0 * 3 * D);
  CHK(gemm(c, a, D, w, bias, out, 3 * D, g.m, 3 * D, D, EPI_STORE, nullptr,
           batched ? Batch{(int)NB, N * D, N * 3 * D, 0} : Batch()));
  return qkv_prep(c, out, 3 * D, row0, rows);
}

// LayerNorm + modulation of rows [row0, row0 + rows) of every sample, with the
// shift/scale vectors of sample 0 given (the others follow at mod_stride)
wdc_status ln_mod(wdc_ctx *c, int64_t row0, int64_t rows, const float *shift, const float *scale) {
  LnRows r;
  r.rows = rows * c->nb;
  r.rps = rows;
  r.sstride = c->n;
  r.mstride = mod_stride(c);
  HIPCHK(c, timed(c, WDC_T_NORM, (double)r.rows * c->D * (4 + c->esz), [&] {
    return launch_ln_mod(c->d.dtype, c->x + row0 * c->D, c->D, elem(c, c->h, row0 * c->D), c->D, r, c->D, shift,
                         scale, c->stream);
  }));
  return WDC_OK;
}

// ---------------------------------------------------------------- blocks
// Every block works on all nb samples of the residual stream x [nb, N, D]:
// products that share weights and need no per-sample vector run as one GEMM
// over all rows; gated residual products run as a batch (one gate per sample).
wdc_status seq_block(wdc_ctx *c, int i) {
  const int64_t D = c->D, N = c->n, F = c->F, LC = D + F, NB = c->nb, MS = mod_stride(c);
  const std::string pre = "seq." + std::to_string(i);
  float *m = c->mod;
  const Batch gr{(int)NB, N * LC, N * D, MS};
  CHK(mod_gemv(c, pre + ".ada", 0));
  CHK(ln_mod(c, 0, N, m, m + D));
  CHK(qkv_project(c, c->h, W(c, pre + ".qkv.w"), W(c, pre + ".qkv.b"), 0, N, false));
  CHK(attention(c, c->cat, LC));
  CHK(gemm(c, c->cat, LC, W(c, pre + ".out.w"), W(c, pre + ".out.b"), c->x, D, N, D, D, EPI_GATE_RES, m + 2 * D, gr));
  CHK(ln_mod(c, 0, N, m + 3 * D, m + 4 * D));
  CHK(gemm(c, c->h, D, W(c, pre + ".fc1.w"), W(c, pre + ".fc1.b"), elem(c, c->cat, D), LC, NB * N, F, D,
           EPI_GELU));
  CHK(gemm(c, elem(c, c->cat, D), LC, W(c, pre + ".fc2.w"), W(c, pre + ".fc2.b"), c->x, D, N, D, F, EPI_GATE_RES,
           m + 5 * D, gr));
  return WDC_OK;
}

wdc_status dual_block(wdc_ctx *c, int i) {
  const int64_t D = c->D, N = c->n, F = c->F, LC = D + F, NV = c->nv, NT = c->nt, NB = c->nb, MS = mod_stride(c);
  const std::string pre = "dual." + std::to_string(i);
  float *mv = c->mod, *mt = c->mod + 6 * D;
  CHK(mod_gemv(c, pre + ".vid.ada", 0));
  CHK(mod_gemv(c, pre + ".txt.ada", 6 * D));
  const struct {
    const char *s;
    int64_t r0, rows;
    float *m;
  } st[2] = {{"vid", 0, NV, mv}, {"txt", NV, NT, mt}};
  for (auto &s : st) {
    std::string p = pre + "." + s.s;
    CHK(ln_mod(c, s.r0, s.rows, s.m, s.m + D));
    CHK(qkv_project(c, elem(c, c->h, s.r0 * D), W(c, p + ".qkv.w"), W(c, p + ".qkv.b"), s.r0, s.rows, true));
  }
  CHK(attention(c, c->cat, LC));
  for (auto &s : st) {
    std::string p = pre + "." + s.s;
    CHK(gemm(c, elem(c, c->cat, s.r0 * LC), LC, W(c, p + ".out.w"), W(c, p + ".out.b"), c->x + s.r0 * D, D, s.rows,
             D, D, EPI_GATE_RES, s.m + 2 * D, Batch{(int)NB, N * LC, N * D, MS}));
    CHK(ln_mod(c, s.r0, s.rows, s.m + 3 * D, s.m + 4 * D));
    CHK(gemm(c, elem(c, c->h, s.r0 * D), D, W(c, p + ".fc1.w"), W(c, p + ".fc1.b"), elem(c, c->cat, s.r0 * LC + D),
             LC, s.rows, F, D, EPI_GELU, nullptr, Batch{(int)NB, N * D, N * LC, 0}));
    CHK(gemm(c, elem(c, c->cat, s.r0 * LC + D), LC, W(c, p + ".fc2.w"), W(c, p + ".fc2.b"), c->x + s.r0 * D, D,
             s.rows, D, F, EPI_GATE_RES, s.m + 5 * D, Batch{(int)NB, N * LC, N * D, MS}));
  }
  return WDC_OK;
}

wdc_status single_block(wdc_ctx *c, int i) {
  const int64_t D = c->D, N = c->n, F = c->F, LC = D + F, NB = c->nb, MS = mod_stride(c);
  const std::string pre = "single." + std::to_string(i);
  float *m = c->mod;
  CHK(mod_gemv(c, pre + ".ada", 0));
  CHK(ln_mod(c, 0, N, m, m + D));
  const char *w1 = (const char *)W(c, pre + ".lin1.w"), *b1 = (const char *)W(c, pre + ".lin1.b");
  if (!w1) {
    set_err(c, "weights not bound");
    return WDC_E_WORKSPACE;
  }
  CHK(qkv_project(c, c->h, w1, b1, 0, N, false));
  CHK(gemm(c, c->h, D, w1 + 3 * D * D * c->esz, b1 + 3 * D * c->esz, elem(c, c->cat, D), LC, NB * N, F, D,
           EPI_GELU));
  CHK(attention(c, c->cat, LC));
  CHK(gemm(c, c->cat, LC, W(c, pre + ".lin2.w"), W(c, pre + ".lin2.b"), c->x, D, N, D, LC, EPI_GATE_RES, m + 2 * D,
           Batch{(int)NB, N * LC, N * D, MS}));
  return WDC_OK;
}

wdc_status block_forward(wdc_ctx *c, int b) {
  if (b < c->d.n_seq) return seq_block(c, b);
  b -= c->d.n_seq;
  if (b < c->d.n_dual) return dual_block(c, b);
  b -= c->d.n_dual;
  return single_block(c, b);
}

wdc_status need_ws(wdc_ctx *c) {
  if (!c->ws) {
    set_err(c, "workspace not bound");
    return WDC_E_WORKSPACE;
  }
  return WDC_OK;
}
wdc_status need_w(wdc_ctx *c) {
  if (!c->w) {
    set_err(c, "weights not bound");
    return WDC_E_WORKSPACE;
  }
  return WDC_OK;
}

wdc_status cond_embed(wdc_ctx *c, double t, const void *cond, const void *cam, float *out) {
  HIPCHK(c, launch_timestep_features(t, c->tfeat, c->stream));
  CHK(gemv(c, "t_embed.fc1", c->tfeat, c->tmp, 0, 0));
  CHK(gemv(c, "t_embed.fc2", c->tmp, out, 1, 0));
  if (c->d.cond_dim) {
    if (!cond) {
      set_err(c, "model has a condition vector but d_cond is NULL");
      return WDC_E_ARG;
    }
    HIPCHK(c, launch_to_f32(c->d.dtype, cond, c->cvec, c->d.cond_dim, c->stream));
    CHK(gemv(c, "cond_embed", c->cvec, out, 0, 1));
  }
  if (c->d.cam_dim) {
    if (!cam) {
      set_err(c, "model has a camera vector but d_cam is NULL");
      return WDC_E_ARG;
    }
    HIPCHK(c, launch_to_f32(c->d.dtype, cam, c->cvec, c->d.cam_dim, c->stream));
    CHK(gemv(c, "cam_embed", c->cvec, out, 0, 1));
  }
  return WDC_OK;
}

// F_theta of nb samples at one time t (inputs per sample; cond/text/cam arrays may be null)
wdc_status dit_forward_batch(wdc_ctx *c, int nb, const float *const *z, double t, const void *const *cond,
                             const void *const *text, const void *const *cam, float *const *vout) {
  CHK(need_ws(c));
  CHK(need_w(c));
  if (nb < 1 || nb > c->mb) {
    set_err(c, "batch of %d samples outside 1..%d (max_batch)", nb, c->mb);
    return WDC_E_ARG;
  }
  struct Restore {
    wdc_ctx *c;
    ~Restore() { c->nb = 1; }
  } restore{c};
  c->nb = nb;
  const int64_t D = c->D, N = c->n, NV = c->nv, P = c->P;
  const auto &d = c->d;
  for (int b = 0; b < nb; ++b)
    CHK(cond_embed(c, t, cond ? cond[b] : nullptr, cam ? cam[b] : nullptr, c->cemb + b * D));
  for (int b = 0; b < nb; ++b)
    HIPCHK(c, launch_patchify(d.dtype, z[b], elem(c, c->patches, b * NV * P), d.lat_c, d.lat_f, d.lat_h, d.lat_w,
                              d.patch_t, d.patch_h, d.patch_w, c->stream));
  CHK(gemm(c, c->patches, P, W(c, "patch_embed.w"), W(c, "patch_embed.b"), c->x, D, NV, D, P, EPI_STORE_F32, nullptr,
           Batch{nb, NV * P, N * D, 0}));
  if (d.text_tokens) {
    for (int b = 0; b < nb; ++b) {
      if (!text || !text[b]) {
        set_err(c, "model has text tokens but d_text is NULL");
        return WDC_E_ARG;
      }
      CHK(gemm(c, text[b], d.text_dim, W(c, "text_proj.w"), W(c, "text_proj.b"), c->x + (b * N + NV) * D, D, c->nt,
               D, d.text_dim, EPI_STORE_F32));
    }
  }
  for (int b = 0; b < d.n_seq + d.n_dual + d.n_single; ++b) CHK(block_forward(c, b));
  CHK(mod_gemv(c, "final.ada", 0));
  CHK(ln_mod(c, 0, NV, c->mod, c->mod + D));
  CHK(gemm(c, c->h, D, W(c, "final.lin.w"), W(c, "final.lin.b"), c->tok, P, NV, P, D, EPI_STORE_F32, nullptr,
           Batch{nb, N * D, NV * P, 0}));
  for (int b = 0; b < nb; ++b)
    HIPCHK(c, launch_unpatchify(c->tok + b * NV * P, vout[b], d.lat_c, d.lat_f, d.lat_h, d.lat_w, d.patch_t,
                                d.patch_h, d.patch_w, c->stream));
  return WDC_OK;
}

wdc_status dit_forward(wdc_ctx *c, const float *z, double t, const void *cond, const void *text, const void *cam,
                       float *vout) {
  return dit_forward_batch(c, 1, &z, t, &cond, &text, &cam, &vout);
}

// ---------------------------------------------------------------- surrogate / risk (host float64)
double cosine(const double *a, const double *b) {
  double ab = 0, aa = 0, bb = 0;
  for (int i = 0; i < S_DIM; ++i) {
    ab += a[i] * b[i];
    aa += a[i] * a[i];
    bb += b[i] * b[i];
  }
  double den = std::sqrt(aa) * std::sqrt(bb);
  return den >= 1e-30 ? ab / den : 0.0;
}

// softmax over the listed entries (max subtracted)
void softmax(const double *x, const std::vector<int> &idx, double *out) {
  double mx = -INFINITY;
  for (int i : idx) mx = std::max(mx, x[i]);
  double s = 0;
  for (int i : idx) s += std::exp(x[i] - mx);
  for (int i : idx) out[i] = std::exp(x[i] - mx) / s;
}

// fill the latent-dependent part of a summary: P_8(nu z) and P_4(nu(z - z_a)).
// segsum_z / segsum_d: per fine segment sums [C*8]; sq_z / sq_d: sums of squares.
void summary_latent(const wdc_state *st, const double *segsum_z, double sq_z, const double *segsum_d, double sq_d,
                    bool has_anchor, double *s) {
  const wdc_ctx *c = st->ctx;
  const int C = c->d.lat_c;
  const double E = (double)c->E, eps = c->p.eps_nu;
  const double rz = std::sqrt(sq_z / E + eps);
  for (int ch = 0; ch < C; ++ch)
    for (int g = 0; g < G8; ++g) s[ch * G8 + g] = segsum_z[ch * G8 + g] / std::sqrt(st->n8[ch * G8 + g]) / rz;
  const int o = C * G8;
  if (!has_anchor) {
    for (int i = 0; i < C * G4; ++i) s[o + i] = 0.0;
    return;
  }
  const double rd = std::sqrt(sq_d / E + eps);
  for (int ch = 0; ch < C; ++ch)
    for (int g = 0; g < G4; ++g) {
      const int a = ch * G8 + 2 * g, b = a + 1;
      s[o + ch * G4 + g] = (segsum_d[a] + segsum_d[b]) / std::sqrt(st->n8[a] + st->n8[b]) / rd;
    }
}

void summary_tail(const wdc_state *st, double *s) {
  const int o = st->ctx->d.lat_c * (G8 + G4);
  for (int i = 0; i < 32; ++i) s[o + i] = st->hsum[i];
  const bool cond = st->ctx->p.lift_condition != 0;
  for (int i = 0; i < GCAM; ++i) s[o + 32 + i] = cond ? st->cam[i] : 0.0;
  for (int i = 0; i < GCAM; ++i) s[o + 48 + i] = 0.0;  // depth: unavailable
}

// Device buffers the statistics kernels write: per-block partial sums and
// their per-segment float64 reductions (the state's own, or the fixed scratch
// of the allocation-free entry point).
struct Scratch {
  float *part;
  double *red;
};
Scratch own_scratch(wdc_state *st) { return Scratch{st->partials, st->d_red}; }

wdc_status fetch(wdc_state *st, int nv, Scratch sc) {
  wdc_ctx *c = st->ctx;
  HIPCHK(c, launch_reduce_partials(st->plan, sc.part, nv, sc.red, c->stream));
  HIPCHK(c, hipMemcpyAsync(st->h_red, sc.red, sizeof(double) * st->plan.nseg() * nv, hipMemcpyDeviceToHost,
                           c->stream));
  HIPCHK(c, hipStreamSynchronize(c->stream));
  return WDC_OK;
}

void log_clear(wdc_step_log *l) {
  std::memset(l, 0, sizeof(*l));
  l->d_cf = NAN;
  l->sim_margin = INFINITY;
  l->margin = INFINITY;
}

// Pass 1 + candidate (Eq. (2)-(5)) for step k; keeps it pending in the state.
// pre: pass-1 statistics of z [nseg, PRE_NV] already at hand, else null (computed here).
// sc: where the statistics kernels put their partial sums.
wdc_status surrogate_step(wdc_state *st, const float *z, int k, int S, float *zhat, wdc_step_log *log,
                          const double *pre, Scratch sc) {
  wdc_ctx *c = st->ctx;
  const auto &p = c->p;
  const int nseg = st->plan.nseg();
  const float *za = st->has_anchor ? st->anchor[st->acur] : nullptr;
  if (!pre) {
    const double bytes = (za ? 8.0 : 4.0) * c->E;
    HIPCHK(c, timed(c, WDC_T_STATS, bytes,
                    [&] { return launch_stats_pre(st->plan, z, za, sc.part, c->stream); }));
    CHK(fetch(st, PRE_NV, sc));
    pre = st->h_red;
  }
  std::vector<double> sz(nseg), sd(nseg);
  double qz = 0, qd = 0, ad = 0, aa = 0;
  for (int i = 0; i < nseg; ++i) {
    const double *r = pre + i * PRE_NV;
    sz[i] = r[0];
    sd[i] = r[1];
    qz += r[2];
    qd += r[3];
    ad += r[4];
    aa += r[5];
  }
  summary_latent(st, sz.data(), qz, sd.data(), qd, st->has_anchor, st->s_phi);
  summary_tail(st, st->s_phi);
  st->rho_cur = std::sqrt(qz / (double)c->E + p.eps_nu);
  const double t = t_at(k, S), tn = t_at(k + 1, S);
  // risk proxy terms that only need pass-1 statistics (Eq. (6))
  double dz = 0, dph = 0;
  if (st->has_anchor) {
    dz = ad / (aa + p.eps);
    dph = std::fabs(t - st->q_a);
  }
  const double dage = (double)(st->n_s + 1) / (double)(p.age_max + 1);
  st->proxy = p.w_z * dz + p.w_age * dage + p.w_phase * dph;  // camera / depth change: static (0)
  st->pend_k = k;
  st->pend_decided = false;
  st->pend_zhat = nullptr;
  st->pend_support = 0;
  st->pend_finite = false;
  st->pend_cand = false;
  log_clear(log);
  log->k = k;
  log->t = t;
  log->d_z = dz;
  log->d_age = dage;
  log->d_phase = dph;
  log->p = st->proxy;
  int nb = 0;
  std::vector<int> slots;
  for (int i = 0; i < p.bank_capacity; ++i)
    if (st->filled[i]) slots.push_back(i);
  nb = (int)slots.size();
  log->bank = nb;
  if (nb == 0) return WDC_OK;
  double sims[WDC_MAX_BANK] = {}, pi[WDC_MAX_BANK] = {}, kap[WDC_MAX_BANK] = {};
  double alpha = 0;
  int support = 0;
  // linear combination zhat = sum_j coef_j * src_j evaluated by the observation kernel
  const float *src[WDC_MAXB];
  float coef[WDC_MAXB];
  int m = 0;
  if (p.surrogate == WDC_SURROGATE_SECANT) {
    // native latent secant: the latest exact transition anchor -> bank[latest]
    const int latest = (st->inserts - 1) % p.bank_capacity;
    alpha = (tn - t) / (st->q_am1 - st->q_a);
    src[0] = z;
    src[1] = st->bank[latest];
    src[2] = za;
    coef[0] = 1.0f;
    coef[1] = (float)alpha;
    coef[2] = (float)-alpha;
    m = 3;
    pi[latest] = 1.0;
    support = 1;
  } else {
    // retrieval (Eq. (3)); without condition information the phase terms drop out
    double logit[WDC_MAX_BANK] = {};
    std::vector<int> supp, all;
    for (int i : slots) {
      sims[i] = cosine(st->s_phi, st->rec[i].s_in);
      const double dq = t - st->rec[i].q_in;
      const bool cond = p.lift_condition != 0;
      logit[i] = (sims[i] - (cond ? p.gamma_q * dq * dq : 0.0)) / p.tau_in;
      if (sims[i] >= p.theta_sim && (!cond || std::fabs(dq) <= p.theta_q)) supp.push_back(i);
      all.push_back(i);
    }
    if (!supp.empty()) softmax(logit, supp, pi);
    support = (int)supp.size();
    // scheduler scaling and lifted evolution (Eq. (4))
    alpha = std::fabs(tn - t) / (std::fabs(st->q_am1 - st->q_a) + p.eps);
    alpha = std::min(std::max(alpha, p.alpha_min), p.alpha_max);
    if (p.observation == WDC_OBS_LINEAR) {
      // rho_t * (nu(z_t) + alpha * sum pi_i (nu(z_i^out) - nu(z_i^in)))
      src[m] = z;
      coef[m++] = 1.0f;
      for (int i : supp) {
        src[m] = st->bank[i];
        coef[m++] = (float)(alpha * pi[i] * st->rho_cur / st->rec[i].rho_out);
        src[m] = st->bank_in[i];
        coef[m++] = (float)(-alpha * pi[i] * st->rho_cur / st->rec[i].rho_in);
      }
    } else {
      // summary-space evolution (s is linear), then kernelized observation over
      // the whole bank (Eq. (5))
      double shat[S_DIM];
      for (int j = 0; j < S_DIM; ++j) {
        double acc = 0;
        for (int i : supp) acc += pi[i] * (st->rec[i].s_out[j] - st->rec[i].s_in[j]);
        shat[j] = st->s_phi[j] + alpha * acc;
      }
      double ks[WDC_MAX_BANK] = {};
      for (int i : slots) ks[i] = cosine(shat, st->rec[i].s_out) / p.tau_obs;
      softmax(ks, all, kap);
      for (int i : slots) {
        src[m] = st->bank[i];
        coef[m++] = (float)kap[i];
      }
    }
  }
  double simm = INFINITY;
  for (int i : slots) simm = std::min(simm, std::fabs(sims[i] - p.theta_sim));
  const double obytes = (4.0 * m + 4.0 + (za ? 4.0 : 0.0)) * c->E;
  HIPCHK(c, timed(c, WDC_T_OBSERVE, obytes,
                  [&] { return launch_observe(st->plan, src, coef, m, za, zhat, sc.part, c->stream); }));
  CHK(fetch(st, OBS_NV, sc));
  double nonfinite = 0;
  st->pre_obs.resize((size_t)nseg * PRE_NV);
  for (int i = 0; i < nseg; ++i) {
    const double *r = st->h_red + i * OBS_NV;
    for (int j = 0; j < PRE_NV; ++j) st->pre_obs[(size_t)i * PRE_NV + j] = r[j];
    nonfinite += r[PRE_NV];
  }
  st->pend_cand = true;
  st->pend_zhat = zhat;
  st->pend_support = support;
  st->pend_finite = nonfinite == 0;
  log->support = st->pend_support;
  log->finite = st->pend_finite;
  log->alpha = alpha;
  log->sim_margin = simm;
  for (int j = 0; j < nb; ++j) {
    log->pi[j] = pi[slots[j]];
    log->kappa[j] = kap[slots[j]];
    log->sims_in[j] = sims[slots[j]];
  }
  return WDC_OK;
}

// Eq. (6), (9), (10) on the pending candidate of step k.
void pre_decision(wdc_state *st, int k, int S, int mode, int forced, wdc_step_log *log) {
  const auto &p = st->ctx->p;
  const double t = t_at(k, S);
  // camera / depth sensitivity: static (0)
  const double w = p.impact_weight ? std::min(2.0, 1.0 + p.a_phase * t) : 1.0;
  st->wgt = w;
  st->d_hat = st->eta * st->proxy;
  st->r_cand = p.lam * st->R + w * st->d_hat;
  int nb = 0;
  for (int i = 0; i < p.bank_capacity; ++i) nb += st->filled[i];
  const bool supported = st->pend_support >= p.n_min || !p.support_constraint;
  const bool avail = nb > 0 && st->n_s <= p.age_max && supported && st->pend_finite && k >= p.k_init &&
                     k <= S - 1 - p.k_ref;
  const double tau = mode == WDC_MODE_ALL_EXACT ? -INFINITY : p.tau_risk;
  bool take;
  if (mode == WDC_MODE_FORCED)
    take = forced && avail;
  else if (mode == WDC_MODE_PERIODIC)
    take = k % p.period != 0 && avail;
  else
    take = avail && st->r_cand <= tau;
  st->pend_avail = avail;
  st->pend_decided = true;
  st->pend_surrogate = take;
  log->w = w;
  log->d_hat = st->d_hat;
  log->r_cand = st->r_cand;
  log->available = avail;
  log->exact = !take;
  log->margin = std::isfinite(tau) ? std::fabs(st->r_cand - tau) / std::max(std::fabs(tau), 1e-12) : INFINITY;
}

// after an exact step: z -> zn (zn computed here from v when v != null)
wdc_status post_exact(wdc_state *st, const float *z, const float *v, float *zn, int k, int S, wdc_step_log *log) {
  wdc_ctx *c = st->ctx;
  const auto &p = c->p;
  const int nseg = st->plan.nseg();
  const int slot = st->inserts % p.bank_capacity;
  const double t = t_at(k, S), tn = t_at(k + 1, S);
  PostArgs a{};
  a.z = z;
  a.v = v;
  a.zn_in = zn;
  a.zn_out = zn;
  a.dt = (float)(tn - t);
  a.za = st->has_anchor ? st->anchor[st->acur] : nullptr;
  a.has_anchor = st->has_anchor;
  a.zhat = st->pend_cand ? st->pend_zhat : nullptr;
  a.has_zhat = st->pend_cand ? 1 : 0;
  a.bank_slot = st->bank[slot];
  a.anchor_out = st->anchor[st->acur ^ 1];
  a.in_slot = st->bank_in[slot];  // null unless the linear observation keeps record inputs
  // z and v (or zn) read, za and zhat read when present; zn, bank slot and anchor copy written
  const double pbytes = 4.0 * c->E * (2 + a.has_anchor + a.has_zhat + (a.v ? 1 : 0) + 2 + (a.in_slot ? 1 : 0));
  HIPCHK(c, timed(c, WDC_T_EXACT_POST, pbytes,
                  [&] { return launch_exact_post(st->plan, a, st->partials, c->stream); }));
  CHK(fetch(st, POST_NV, own_scratch(st)));
  std::vector<double> sn(nseg), sdn(nseg), sdx(nseg);
  double qn = 0, qdn = 0, qdx = 0, acf = 0, an = 0;
  st->pre_post.resize((size_t)nseg * PRE_NV);
  for (int i = 0; i < nseg; ++i) {
    const double *r = st->h_red + i * POST_NV;
    sn[i] = r[0];
    sdn[i] = r[1];
    sdx[i] = r[2];
    qn += r[3];
    qdn += r[4];
    qdx += r[5];
    acf += r[6];
    an += r[7];
    // next step's pass 1: latent zn against the new anchor z
    double *q = &st->pre_post[(size_t)i * PRE_NV];
    q[0] = r[0];
    q[1] = r[2];
    q[2] = r[3];
    q[3] = r[5];
    q[4] = r[8];
    q[5] = r[9];
  }
  const double E = (double)c->E;
  // counterfactual defect (Eq. (7)) and calibration (Eq. (8))
  double dcf = NAN;
  const bool supported = st->pend_support >= p.n_min || !p.support_constraint;
  if (st->pend_cand && supported && st->pend_finite) {
    dcf = (acf / E) / (an / E + p.eps);
    if (p.calibrate) {
      double e = p.beta_d * st->eta + (1.0 - p.beta_d) * dcf / (st->proxy + p.eps);
      st->eta = std::min(std::max(e, p.eta_min), p.eta_max);
    }
  }
  st->R = p.lam * st->R;
  // record: both lifted states under the pre-insertion anchor and history
  Record &r = st->rec[slot];
  std::memcpy(r.s_in, st->s_phi, sizeof(r.s_in));
  summary_latent(st, sn.data(), qn, sdn.data(), qdn, st->has_anchor, r.s_out);
  summary_tail(st, r.s_out);
  r.q_in = t;
  r.q_out = tn;
  r.rho_in = st->rho_cur;
  r.rho_out = std::sqrt(qn / E + p.eps_nu);
  st->filled[slot] = true;
  st->inserts++;
  // history summary h = P_2(nu(zn - z)) of this transition
  const int C = c->d.lat_c;
  const double rx = std::sqrt(qdx / E + p.eps_nu);
  for (int ch = 0; ch < C; ++ch)
    for (int g = 0; g < G2; ++g) {
      double s = 0, n = 0;
      for (int f = 0; f < 4; ++f) {
        s += sdx[ch * G8 + 4 * g + f];
        n += st->n8[ch * G8 + 4 * g + f];
      }
      st->hsum[ch * G2 + g] = s / std::sqrt(n) / rx;
    }
  st->acur ^= 1;
  st->has_anchor = true;
  st->q_a = t;
  st->q_am1 = tn;
  st->n_s = 0;
  st->pend_k = -1;
  if (log) {
    log->d_cf = dcf;
    log->eta = st->eta;
    log->R = st->R;
    log->slot = slot;
  }
  return WDC_OK;
}

void post_surrogate(wdc_state *st, wdc_step_log *log) {
  st->R = st->r_cand;
  st->n_s += 1;
  st->pend_k = -1;
  if (log) {
    log->eta = st->eta;
    log->R = st->R;
    log->slot = -1;
  }
}

void state_reset(wdc_state *st, const float *h_cam) {
  wdc_ctx *c = st->ctx;
  st->acur = 0;
  st->has_anchor = false;
  st->q_a = st->q_am1 = 0;
  for (int i = 0; i < WDC_MAX_BANK; ++i) st->filled[i] = false;
  st->inserts = 0;
  for (double &x : st->hsum) x = 0;
  for (double &x : st->cam) x = 0;
  if (h_cam && c->d.cam_dim > 0) {
    // 16-d descriptor P_16(nu(cam))
    const int L = c->d.cam_dim;
    double ss = 0;
    for (int i = 0; i < L; ++i) ss += (double)h_cam[i] * h_cam[i];
    const double r = std::sqrt(ss / L + c->p.eps_nu);
    double sum[GCAM] = {}, cnt[GCAM] = {};
    for (int i = 0; i < L; ++i) {
      int g = (int)(((int64_t)i * GCAM) / L);
      sum[g] += h_cam[i] / r;
      cnt[g] += 1;
    }
    for (int g = 0; g < GCAM; ++g) st->cam[g] = cnt[g] > 0 ? sum[g] / std::sqrt(cnt[g]) : 0.0;
  }
  st->R = c->p.r0;
  st->eta = c->p.eta0;
  st->n_s = 0;
  st->pend_k = -1;
  st->pend_cand = false;
}

}  // namespace

// ====================================================================== C ABI
extern "C" {

void wdc_params_default(wdc_params *p) {
  if (!p) return;
  std::memset(p, 0, sizeof(*p));
  p->bank_capacity = 4;
  p->age_max = 6;
  p->n_min = 1;
  p->k_init = 1;
  p->k_ref = 0;
  p->theta_sim = 0.25;
  p->theta_q = 0.43;
  p->tau_in = 0.05;
  p->tau_obs = 0.02;
  p->gamma_q = 10.0;
  p->alpha_min = 0.5;
  p->alpha_max = 2.0;
  p->eps = 1e-8;
  p->eps_nu = 1e-6;
  p->w_z = 1.0;
  p->w_age = 0.05;
  p->w_phase = 0.5;
  p->w_cam = 0.5;
  p->w_depth = 0.5;
  p->eta0 = 1.0;
  p->beta_d = 0.8;
  p->eta_min = 0.05;
  p->eta_max = 20.0;
  p->a_cam = 0.5;
  p->a_depth = 0.5;
  p->a_phase = 0.5;
  p->lam = 0.8;
  p->r0 = 0.0;
  p->tau_risk = 0.5;
  p->period = 4;
  p->surrogate = WDC_SURROGATE_LIFTED;
  p->observation = WDC_OBS_KERNEL;
  p->lift_condition = 1;
  p->impact_weight = 1;
  p->calibrate = 1;
  p->support_constraint = 1;
}

const char *wdc_last_error(const wdc_ctx *ctx) { return ctx ? ctx->err.c_str() : g_create_err.c_str(); }

wdc_status wdc_create(const wdc_model_desc *desc, const wdc_params *params, wdc_stream stream, wdc_ctx **out) {
  g_create_err.clear();
  if (!desc || !out) {
    g_create_err = "null argument";
    return WDC_E_ARG;
  }
  const wdc_model_desc &d = *desc;
  if (d.dtype != WDC_F32 && d.dtype != WDC_BF16) {
    g_create_err = "dtype must be WDC_F32 or WDC_BF16";
    return WDC_E_DTYPE;
  }
  if (d.lat_c != 16) {
    g_create_err = "the 256-d summary needs 16 latent channels";
    return WDC_E_UNSUPPORTED;
  }
  if (d.patch_t < 1 || d.patch_h < 1 || d.patch_w < 1 || d.lat_f % d.patch_t || d.lat_h % d.patch_h ||
      d.lat_w % d.patch_w) {
    g_create_err = "latent shape not divisible by the patch";
    return WDC_E_SHAPE;
  }
  const int nblocks = d.n_seq + d.n_dual + d.n_single;
  if (nblocks > 0) {
    if (d.head_dim != 64 && d.head_dim != 128) {
      g_create_err = "head_dim must be 64 or 128";
      return WDC_E_UNSUPPORTED;
    }
    if (d.heads * d.head_dim != d.hidden || d.hidden % 256 != 0 || d.mlp_ratio < 1) {
      g_create_err = "hidden must equal heads*head_dim and be a multiple of 256";
      return WDC_E_SHAPE;
    }
    const int rs = d.rope_t + d.rope_h + d.rope_w;
    if (rs != 0 && (rs != d.head_dim || d.rope_t % 2 || d.rope_h % 2 || d.rope_w % 2)) {
      g_create_err = "rotary dims must be even and sum to head_dim";
      return WDC_E_SHAPE;
    }
    if (d.n_dual > 0 && d.text_tokens <= 0) {
      g_create_err = "dual-stream blocks need text tokens";
      return WDC_E_SHAPE;
    }
  }
  wdc_ctx *c = new wdc_ctx();
  c->d = d;
  if (params)
    c->p = *params;
  else
    wdc_params_default(&c->p);
  if (c->p.bank_capacity < 1 || c->p.bank_capacity > WDC_MAX_BANK) {
    g_create_err = "bank_capacity out of range";
    delete c;
    return WDC_E_ARG;
  }
  if (c->p.period < 1 || (c->p.surrogate != WDC_SURROGATE_LIFTED && c->p.surrogate != WDC_SURROGATE_SECANT) ||
      (c->p.observation != WDC_OBS_KERNEL && c->p.observation != WDC_OBS_LINEAR)) {
    g_create_err = "period, surrogate or observation out of range";
    delete c;
    return WDC_E_ARG;
  }
  if (d.max_batch < 0 || d.max_batch > 64) {
    g_create_err = "max_batch out of range (0..64)";
    delete c;
    return WDC_E_ARG;
  }
  c->mb = d.max_batch > 1 ? d.max_batch : 1;
  c->fuse_qkv = !(getenv("WDC_FUSE_QKV") && atoi(getenv("WDC_FUSE_QKV")) == 0);
  c->fill_tiles = !(getenv("WDC_FILL_TILES") && atoi(getenv("WDC_FILL_TILES")) == 0);
  c->attn_splits = getenv("WDC_ATTN_SPLITS") ? std::max(0, atoi(getenv("WDC_ATTN_SPLITS"))) : 0;
  c->stream = (hipStream_t)stream;
  c->esz = d.dtype == WDC_BF16 ? 2 : 4;
  c->D = d.hidden;
  c->H = d.heads;
  c->hd = d.head_dim;
  c->F = d.mlp_ratio * d.hidden;
  c->P = d.lat_c * d.patch_t * d.patch_h * d.patch_w;
  c->nv = (int64_t)(d.lat_f / d.patch_t) * (d.lat_h / d.patch_h) * (d.lat_w / d.patch_w);
  c->nt = d.text_tokens;
  c->n = c->nv + c->nt;
  c->n_pad = attn_pad(c->n);
  if (nblocks > 0 && d.dtype == WDC_BF16 && !attn_len_ok(c->n, c->hd)) {
    g_create_err = "sequence too long: one head's q, k or v would exceed 2^30 bytes (32-bit offsets)";
    delete c;
    return WDC_E_SHAPE;
  }
  c->T = (int64_t)d.lat_f * d.lat_h * d.lat_w;
  c->E = (int64_t)d.lat_c * c->T;
  if (nblocks > 0) build_layout(c);
  c->ws_need = ws_layout(c).total;
  *out = c;
  return WDC_OK;
}

wdc_status wdc_destroy(wdc_ctx *ctx) {
  if (!ctx) return WDC_E_ARG;
  release_events(ctx);
  delete ctx;
  return WDC_OK;
}

size_t wdc_weights_bytes(const wdc_ctx *ctx) { return ctx ? ctx->wbytes : 0; }
int32_t wdc_weight_count(const wdc_ctx *ctx) { return ctx ? (int32_t)ctx->tensors.size() : 0; }

wdc_status wdc_weight_info(const wdc_ctx *ctx, int32_t i, const char **name, int64_t shape[2], int32_t *ndim,
                           size_t *offset) {
  if (!ctx || i < 0 || i >= (int32_t)ctx->tensors.size()) return WDC_E_ARG;
  const auto &t = ctx->tensors[i];
  if (name) *name = t.name.c_str();
  if (shape) {
    shape[0] = t.shape[0];
    shape[1] = t.shape[1];
  }
  if (ndim) *ndim = t.ndim;
  if (offset) *offset = t.offset;
  return WDC_OK;
}

wdc_status wdc_bind_weights(wdc_ctx *ctx, const void *d_weights, size_t bytes) {
  if (!ctx || !d_weights) return WDC_E_ARG;
  if (!aligned16(d_weights)) {
    set_err(ctx, "weights blob not 16-byte aligned");
    return WDC_E_ALIGN;
  }
  if (bytes < ctx->wbytes) {
    set_err(ctx, "weights blob too small: %zu < %zu", bytes, ctx->wbytes);
    return WDC_E_WORKSPACE;
  }
  ctx->w = (const char *)d_weights;
  return WDC_OK;
}

wdc_status wdc_init_weights_random(wdc_ctx *ctx, void *d_weights, size_t bytes, uint64_t seed, float std) {
  if (!ctx || !d_weights) return WDC_E_ARG;
  if (bytes < ctx->wbytes) {
    set_err(ctx, "weights blob too small");
    return WDC_E_WORKSPACE;
  }
  for (size_t i = 0; i < ctx->tensors.size(); ++i) {
    const auto &t = ctx->tensors[i];
    HIPCHK(ctx, launch_fill_normal(ctx->d.dtype, (char *)d_weights + t.offset, (int64_t)t.numel, seed, (uint64_t)i << 40,
                                   std, ctx->stream));
  }
  return WDC_OK;
}

size_t wdc_workspace_bytes(const wdc_ctx *ctx) { return ctx ? ctx->ws_need : 0; }

wdc_status wdc_bind_workspace(wdc_ctx *ctx, void *d_ws, size_t bytes) {
  if (!ctx || !d_ws) return WDC_E_ARG;
  if (!aligned16(d_ws)) {
    set_err(ctx, "workspace not 16-byte aligned");
    return WDC_E_ALIGN;
  }
  if (bytes < ctx->ws_need) {
    set_err(ctx, "workspace too small: %zu < %zu", bytes, ctx->ws_need);
    return WDC_E_WORKSPACE;
  }
  WsLayout L = ws_layout(ctx);
  char *b = (char *)d_ws;
  ctx->ws = b;
  ctx->ws_bytes = bytes;
  ctx->x = (float *)(b + L.x);
  ctx->h = b + L.h;
  ctx->qkv = b + L.qkv;
  ctx->qkv_bytes = L.cat - L.qkv;
  ctx->cat = b + L.cat;
  ctx->q = b + L.q;
  ctx->k = b + L.k;
  ctx->v = b + L.v;
  ctx->mod = (float *)(b + L.mod);
  ctx->cemb = (float *)(b + L.cemb);
  ctx->tfeat = (float *)(b + L.tfeat);
  ctx->tmp = (float *)(b + L.tmp);
  ctx->cvec = (float *)(b + L.cvec);
  ctx->patches = b + L.patches;
  ctx->tok = (float *)(b + L.tok);
  ctx->rope = (float2 *)(b + L.rope);
  ctx->r_v = (float *)(b + L.rv);
  const auto &d = ctx->d;
  if (d.rope_t + d.rope_h + d.rope_w > 0 && ctx->nv > 0) {
    // rotation table in float64, rounded once: pair j of axis a turns by pos_a * 1e4^(-2j/d_a)
    const int half = ctx->hd / 2;
    const int gf = d.lat_f / d.patch_t, gh = d.lat_h / d.patch_h, gw = d.lat_w / d.patch_w;
    std::vector<float2> tab((size_t)ctx->nv * half);
    const int dims[3] = {d.rope_t, d.rope_h, d.rope_w};
    for (int64_t nidx = 0; nidx < ctx->nv; ++nidx) {
      const int64_t pos[3] = {nidx / ((int64_t)gh * gw), (nidx / gw) % gh, nidx % gw};
      (void)gf;
      int j0 = 0;
      for (int a = 0; a < 3; ++a) {
        for (int j = 0; j < dims[a] / 2; ++j) {
          double ang = (double)pos[a] * std::pow(10000.0, -2.0 * j / dims[a]);
          tab[nidx * half + j0 + j] = make_float2((float)std::cos(ang), (float)std::sin(ang));
        }
        j0 += dims[a] / 2;
      }
    }
    HIPCHK(ctx, hipMemcpy(ctx->rope, tab.data(), tab.size() * sizeof(float2), hipMemcpyHostToDevice));
  }
  return WDC_OK;
}

// anchor double buffer, bank outputs, and bank inputs for the linear observation
static int n_latents(const wdc_ctx *ctx) {
  return 2 + ctx->p.bank_capacity * (ctx->p.observation == WDC_OBS_LINEAR ? 2 : 1);
}

size_t wdc_state_bytes(const wdc_ctx *ctx) {
  if (!ctx) return 0;
  SegPlan pl = make_seg_plan(ctx->d.lat_c, ctx->T, G8);
  size_t lat = (((size_t)ctx->E * 4 + 255) / 256) * 256;
  size_t part = (((size_t)pl.nblocks() * POST_NV * 4 + 255) / 256) * 256;
  size_t red = (((size_t)pl.nseg() * POST_NV * 8 + 255) / 256) * 256;
  return lat * (n_latents(ctx) + 3) + part + red;
}

wdc_status wdc_state_create(wdc_ctx *ctx, void *d_mem, size_t bytes, wdc_state **out) {
  if (!ctx || !d_mem || !out) return WDC_E_ARG;
  if (!aligned16(d_mem)) {
    set_err(ctx, "state memory not 16-byte aligned");
    return WDC_E_ALIGN;
  }
  if (bytes < wdc_state_bytes(ctx)) {
    set_err(ctx, "state memory too small");
    return WDC_E_WORKSPACE;
  }
  wdc_state *st = new wdc_state();
  st->ctx = ctx;
  st->plan = make_seg_plan(ctx->d.lat_c, ctx->T, G8);
  size_t lat = (((size_t)ctx->E * 4 + 255) / 256) * 256;
  char *b = (char *)d_mem;
  st->anchor[0] = (float *)b;
  st->anchor[1] = (float *)(b + lat);
  for (int i = 0; i < ctx->p.bank_capacity; ++i) st->bank[i] = (float *)(b + lat * (2 + i));
  if (ctx->p.observation == WDC_OBS_LINEAR)
    for (int i = 0; i < ctx->p.bank_capacity; ++i)
      st->bank_in[i] = (float *)(b + lat * (2 + ctx->p.bank_capacity + i));
  for (int i = 0; i < 3; ++i) st->rz[i] = (float *)(b + lat * (n_latents(ctx) + i));
  size_t o = lat * (n_latents(ctx) + 3);
  st->partials = (float *)(b + o);
  o += (((size_t)st->plan.nblocks() * POST_NV * 4 + 255) / 256) * 256;
  st->d_red = (double *)(b + o);
  if (hipHostMalloc((void **)&st->h_red, sizeof(double) * st->plan.nseg() * POST_NV, hipHostMallocDefault) !=
      hipSuccess) {
    set_err(ctx, "hipHostMalloc failed");
    delete st;
    return WDC_E_HIP;
  }
  st->n8.resize(st->plan.nseg());
  for (int ch = 0; ch < ctx->d.lat_c; ++ch)
    for (int g = 0; g < G8; ++g) {
      const int64_t T = ctx->T;
      st->n8[ch * G8 + g] = (double)(((g + 1) * T + G8 - 1) / G8 - (g * T + G8 - 1) / G8);
    }
  state_reset(st, nullptr);
  *out = st;
  return WDC_OK;
}

wdc_status wdc_state_reset(wdc_state *st, const float *h_cam) {
  if (!st) return WDC_E_ARG;
  state_reset(st, h_cam);
  return WDC_OK;
}

wdc_status wdc_state_destroy(wdc_state *st) {
  if (!st) return WDC_E_ARG;
  if (st->h_red) (void)hipHostFree(st->h_red);
  delete st;
  return WDC_OK;
}

wdc_status wdc_state_bank_slot(wdc_state *st, int32_t i, float **d_slot, int32_t *inserts) {
  if (!st || i < 0 || i >= st->ctx->p.bank_capacity) return WDC_E_ARG;
  if (d_slot) *d_slot = st->bank[i];
  if (inserts) *inserts = st->inserts;
  return WDC_OK;
}

wdc_status wdc_cond_embed(wdc_ctx *ctx, double t, const void *d_cond, const void *d_cam, float *d_cemb) {
  if (!ctx || !d_cemb) return WDC_E_ARG;
  CHK(need_ws(ctx));
  CHK(need_w(ctx));
  return cond_embed(ctx, t, d_cond, d_cam, d_cemb);
}

wdc_status wdc_dit_block_forward(wdc_ctx *ctx, int32_t block, float *d_x, const float *d_cemb) {
  if (!ctx || !d_x || !d_cemb) return WDC_E_ARG;
  if (block < 0 || block >= ctx->d.n_seq + ctx->d.n_dual + ctx->d.n_single) {
    set_err(ctx, "block index out of range");
    return WDC_E_ARG;
  }
  CHK(need_ws(ctx));
  CHK(need_w(ctx));
  // the block works on the caller's residual stream and conditioning vector in place
  float *x_saved = ctx->x, *c_saved = ctx->cemb;
  ctx->x = d_x;
  ctx->cemb = const_cast<float *>(d_cemb);
  wdc_status s = block_forward(ctx, block);
  ctx->x = x_saved;
  ctx->cemb = c_saved;
  return s;
}

wdc_status wdc_dit_forward(wdc_ctx *ctx, const float *d_z, double t, const void *d_cond, const void *d_text,
                           const void *d_cam, float *d_v) {
  if (!ctx || !d_z || !d_v) return WDC_E_ARG;
  if (ctx->d.n_seq + ctx->d.n_dual + ctx->d.n_single == 0) {
    set_err(ctx, "model has no blocks");
    return WDC_E_STATE;
  }
  return dit_forward(ctx, d_z, t, d_cond, d_text, d_cam, d_v);
}

wdc_status wdc_scheduler_step(wdc_ctx *ctx, const float *d_z, const float *d_v, double t_cur, double t_next,
                              float *d_z_next, int64_t numel) {
  if (!ctx || !d_z || !d_v || !d_z_next || numel < 0) return WDC_E_ARG;
  HIPCHK(ctx, timed(ctx, WDC_T_PSI, 12.0 * numel, [&] { return launch_psi(d_z, d_v, (float)(t_next - t_cur), d_z_next, numel, ctx->stream); }));
  return WDC_OK;
}

wdc_status wdc_surrogate_step(wdc_ctx *ctx, wdc_state *st, const float *d_z, int32_t k, int32_t S, float *d_zhat,
                              wdc_step_log *h_log) {
  if (!ctx || !st || st->ctx != ctx || !d_z || !d_zhat || !h_log || S < 1 || k < 0 || k >= S) return WDC_E_ARG;
  return surrogate_step(st, d_z, k, S, d_zhat, h_log, nullptr, own_scratch(st));
}

wdc_status wdc_surrogate_step_noalloc(wdc_ctx *ctx, wdc_state *st, const float *d_z, int32_t k, int32_t S,
                                      float *d_zhat, wdc_step_log *h_log) {
  if (!ctx || !st || st->ctx != ctx || !d_z || !d_zhat || !h_log || S < 1 || k < 0 || k >= S) return WDC_E_ARG;
  // the statistics kernels write OBS_NV values per block at most (pass 1: PRE_NV)
  const size_t part = (size_t)st->plan.nblocks() * OBS_NV * sizeof(float);
  const size_t red = (size_t)st->plan.nseg() * OBS_NV * sizeof(double);
  if (part > kScratchRedOffset || red > kScratchBytes - kScratchRedOffset) {
    set_err(ctx, "latent needs %zu + %zu bytes of statistics scratch, more than the fixed %zu + %zu", part, red,
            kScratchRedOffset, kScratchBytes - kScratchRedOffset);
    return WDC_E_WORKSPACE;
  }
  void *p = nullptr;
  HIPCHK(ctx, scratch_address(&p));
  const Scratch sc{(float *)p, (double *)((char *)p + kScratchRedOffset)};
  // kernel timing records HIP events, which this entry point does not create
  const bool timing = ctx->timing;
  ctx->timing = false;
  const wdc_status s = surrogate_step(st, d_z, k, S, d_zhat, h_log, nullptr, sc);
  ctx->timing = timing;
  return s;
}

wdc_status wdc_risk_update(wdc_ctx *ctx, wdc_state *st, int32_t phase, int32_t k, int32_t S, const float *d_z_cur,
                           const float *d_z_next, wdc_step_log *h_log) {
  if (!ctx || !st || st->ctx != ctx || !h_log || S < 1 || k < 0 || k >= S) return WDC_E_ARG;
  if (st->pend_k != k) {
    set_err(ctx, "no pending candidate for step %d (call wdc_surrogate_step first)", k);
    return WDC_E_STATE;
  }
  switch (phase) {
    case WDC_PRE_DECISION: pre_decision(st, k, S, WDC_MODE_RISK, 0, h_log); return WDC_OK;
    case WDC_POST_EXACT:
      if (!d_z_cur || !d_z_next) return WDC_E_ARG;
      return post_exact(st, d_z_cur, nullptr, (float *)d_z_next, k, S, h_log);
    case WDC_POST_SURROGATE:
      if (!st->pend_decided || !st->pend_avail) {
        set_err(ctx, "surrogate commit without an available candidate");
        return WDC_E_STATE;
      }
      post_surrogate(st, h_log);
      return WDC_OK;
    default: return WDC_E_ARG;
  }
}

wdc_status wdc_rollout_batch(wdc_ctx *ctx, wdc_state *const *states, int32_t B, float *const *d_z, int32_t S,
                             const void *const *d_cond, const void *const *d_text, const void *const *d_cam,
                             int32_t mode, const uint8_t *h_forced, const float *const *d_replay_v,
                             uint8_t *h_schedule, wdc_step_log *h_log) {
  if (!ctx || !states || !d_z || S < 1 || !h_schedule || B < 1) return WDC_E_ARG;
  if (mode < WDC_MODE_RISK || mode > WDC_MODE_PERIODIC || (mode == WDC_MODE_FORCED && !h_forced)) return WDC_E_ARG;
  if (B > ctx->mb) {
    set_err(ctx, "batch of %d rollouts exceeds max_batch %d", B, ctx->mb);
    return WDC_E_ARG;
  }
  for (int b = 0; b < B; ++b) {
    if (!states[b] || states[b]->ctx != ctx || !d_z[b]) return WDC_E_ARG;
    for (int j = 0; j < b; ++j)
      if (states[j] == states[b]) {
        set_err(ctx, "rollouts of one batch need distinct states");
        return WDC_E_ARG;
      }
    if (d_replay_v && !d_replay_v[b]) return WDC_E_ARG;
  }
  CHK(need_ws(ctx));
  if (!d_replay_v) {
    CHK(need_w(ctx));
    if (ctx->d.n_seq + ctx->d.n_dual + ctx->d.n_single == 0) {
      set_err(ctx, "model has no blocks and no replay velocities were given");
      return WDC_E_STATE;
    }
  }
  const size_t bytes = (size_t)ctx->E * 4;
  struct Sample {
    wdc_state *st;
    float *zc, *zh, *zn;
    std::vector<double> pre;  // pass-1 statistics of zc, emitted by the kernel that wrote it
  };
  std::vector<Sample> sm(B);
  for (int b = 0; b < B; ++b) {
    wdc_state *st = states[b];
    std::vector<float> cam;
    const void *cb = d_cam ? d_cam[b] : nullptr;
    if (cb && ctx->d.cam_dim > 0) {
      cam.resize(ctx->d.cam_dim);
      HIPCHK(ctx, launch_to_f32(ctx->d.dtype, cb, ctx->cvec, ctx->d.cam_dim, ctx->stream));
      HIPCHK(ctx, hipMemcpyAsync(cam.data(), ctx->cvec, cam.size() * 4, hipMemcpyDeviceToHost, ctx->stream));
      HIPCHK(ctx, hipStreamSynchronize(ctx->stream));
    }
    state_reset(st, cam.empty() ? nullptr : cam.data());
    sm[b] = Sample{st, st->rz[0], st->rz[1], st->rz[2], {}};
    HIPCHK(ctx, hipMemcpyAsync(sm[b].zc, d_z[b], bytes, hipMemcpyDeviceToDevice, ctx->stream));
  }
  wdc_step_log tmp;
  std::vector<int> ex;
  std::vector<const float *> zs;
  std::vector<const void *> cs, ts, ms;
  std::vector<float *> vs;
  for (int k = 0; k < S; ++k) {
    ex.clear();
    for (int b = 0; b < B; ++b) {
      Sample &q = sm[b];
      wdc_step_log *lg = h_log ? &h_log[(size_t)b * S + k] : &tmp;
      CHK(surrogate_step(q.st, q.zc, k, S, q.zh, lg, k > 0 ? q.pre.data() : nullptr, own_scratch(q.st)));
      pre_decision(q.st, k, S, mode, h_forced ? h_forced[(size_t)b * S + k] : 0, lg);
      if (q.st->pend_surrogate) {
        post_surrogate(q.st, lg);
        std::swap(q.zc, q.zh);
        q.pre.swap(q.st->pre_obs);
        h_schedule[(size_t)b * S + k] = 1;
      } else {
        ex.push_back(b);
        h_schedule[(size_t)b * S + k] = 0;
      }
    }
    if (ex.empty()) continue;
    // exact subset: one batched F_theta call (or the recorded velocities)
    if (!d_replay_v) {
      zs.clear();
      cs.clear();
      ts.clear();
      ms.clear();
      vs.clear();
      for (size_t j = 0; j < ex.size(); ++j) {
        const int b = ex[j];
        zs.push_back(sm[b].zc);
        cs.push_back(d_cond ? d_cond[b] : nullptr);
        ts.push_back(d_text ? d_text[b] : nullptr);
        ms.push_back(d_cam ? d_cam[b] : nullptr);
        vs.push_back(ctx->r_v + j * ctx->E);
      }
      CHK(dit_forward_batch(ctx, (int)ex.size(), zs.data(), t_at(k, S), cs.data(), ts.data(), ms.data(), vs.data()));
    }
    for (size_t j = 0; j < ex.size(); ++j) {
      const int b = ex[j];
      Sample &q = sm[b];
      wdc_step_log *lg = h_log ? &h_log[(size_t)b * S + k] : &tmp;
      const float *v = d_replay_v ? d_replay_v[b] + (size_t)k * ctx->E : ctx->r_v + j * ctx->E;
      CHK(post_exact(q.st, q.zc, v, q.zn, k, S, lg));
      std::swap(q.zc, q.zn);
      q.pre.swap(q.st->pre_post);
    }
  }
  for (int b = 0; b < B; ++b) HIPCHK(ctx, hipMemcpyAsync(d_z[b], sm[b].zc, bytes, hipMemcpyDeviceToDevice, ctx->stream));
  HIPCHK(ctx, hipStreamSynchronize(ctx->stream));
  return WDC_OK;
}

wdc_status wdc_rollout(wdc_ctx *ctx, wdc_state *st, float *d_z, int32_t S, const void *d_cond, const void *d_text,
                       const void *d_cam, int32_t mode, const uint8_t *h_forced, const float *d_replay_v,
                       uint8_t *h_schedule, wdc_step_log *h_log) {
  if (!ctx || !st || !d_z) return WDC_E_ARG;
  return wdc_rollout_batch(ctx, &st, 1, &d_z, S, d_cond ? &d_cond : nullptr, d_text ? &d_text : nullptr,
                           d_cam ? &d_cam : nullptr, mode, h_forced, d_replay_v ? &d_replay_v : nullptr, h_schedule,
                           h_log);
}

wdc_status wdc_dit_forward_batch(wdc_ctx *ctx, int32_t B, const float *const *d_z, double t,
                                 const void *const *d_cond, const void *const *d_text, const void *const *d_cam,
                                 float *const *d_v) {
  if (!ctx || !d_z || !d_v || B < 1) return WDC_E_ARG;
  for (int b = 0; b < B; ++b)
    if (!d_z[b] || !d_v[b]) return WDC_E_ARG;
  if (ctx->d.n_seq + ctx->d.n_dual + ctx->d.n_single == 0) {
    set_err(ctx, "model has no blocks");
    return WDC_E_STATE;
  }
  return dit_forward_batch(ctx, B, d_z, t, d_cond, d_text, d_cam, d_v);
}

int64_t wdc_attn_pad(int64_t n) { return attn_pad(n); }

wdc_status wdc_attention(wdc_ctx *ctx, const void *d_q, const void *d_k, const void *d_vt, int64_t n, void *d_o,
                         int64_t ldo) {
  if (!ctx || !d_q || !d_k || !d_vt || !d_o || n <= 0) return WDC_E_ARG;
  if (ldo < (int64_t)ctx->H * ctx->hd) return WDC_E_ARG;     // heads would overlap and the last row overrun
  if (ctx->d.dtype == WDC_BF16 && !attn_len_ok(n, ctx->hd)) return WDC_E_SHAPE;
  if (!aligned16(d_q) || !aligned16(d_k) || !aligned16(d_vt)) return WDC_E_ALIGN;
  // bf16 rows leave as 8-byte groups of 4 columns
  if (ctx->d.dtype == WDC_BF16 && ((uintptr_t)d_o % 8 != 0 || ldo % 4 != 0)) return WDC_E_ALIGN;
  AttnArgs a{};
  a.q = d_q;
  a.k = d_k;
  a.v = d_vt;
  a.o = d_o;
  a.n = n;
  a.n_pad = attn_pad(n);
  a.ldo = ldo;
  a.heads = ctx->H;
  a.hd = ctx->hd;
  attn_scratch(ctx, a);
  const double aw = 4.0 * (double)n * (double)n * ctx->hd * ctx->H;
  HIPCHK(ctx, timed(ctx, WDC_T_ATTENTION, aw, [&] { return launch_attention(ctx->d.dtype, a, ctx->stream); }));
  return WDC_OK;
}

wdc_status wdc_attention_plan(const wdc_ctx *ctx, int64_t n, int32_t *qb_main, int32_t *kv_splits) {
  if (!ctx || n <= 0) return WDC_E_ARG;
  AttnArgs a{};
  a.n = n;
  a.n_pad = attn_pad(n);
  a.heads = ctx->H;
  a.hd = ctx->hd;
  attn_scratch(ctx, a);
  if (ctx->d.dtype == WDC_BF16) {
    attn_split_plan(a);
  } else {
    a.qb_main = (int)(a.n_pad / 256);
    a.kv_splits = 1;
  }
  if (qb_main) *qb_main = a.qb_main;
  if (kv_splits) *kv_splits = a.kv_splits;
  return WDC_OK;
}

wdc_status wdc_linear(wdc_ctx *ctx, const void *d_a, int64_t lda, const void *d_w, const void *d_bias, void *d_c,
                      int64_t ldc, int64_t m, int64_t n, int64_t k) {
  if (!ctx || !d_a || !d_w || !d_c || m < 0 || n <= 0 || k <= 0 || lda < k || ldc < n) return WDC_E_ARG;
  return gemm(ctx, d_a, lda, d_w, d_bias, d_c, ldc, m, n, k, EPI_STORE);
}

wdc_status wdc_set_timing(wdc_ctx *ctx, int32_t on) {
  if (!ctx) return WDC_E_ARG;
  ctx->timing = on != 0;
  release_events(ctx);
  for (int i = 0; i < WDC_T_COUNT; ++i) {
    ctx->t_ms[i] = 0;
    ctx->t_cnt[i] = 0;
    ctx->t_work[i] = 0;
  }
  return WDC_OK;
}

wdc_status wdc_timing(wdc_ctx *ctx, double out_ms[WDC_T_COUNT], int64_t out_count[WDC_T_COUNT],
                      double out_work[WDC_T_COUNT]) {
  if (!ctx || !out_ms || !out_count) return WDC_E_ARG;
  HIPCHK(ctx, hipStreamSynchronize(ctx->stream));
  for (auto &e : ctx->events) {
    float ms = 0;
    const hipError_t err = hipEventElapsedTime(&ms, e.a, e.b);
    if (err != hipSuccess) {
      set_err(ctx, "hipEventElapsedTime failed: %s", hipGetErrorString(err));
      release_events(ctx);
      return WDC_E_HIP;
    }
    ctx->t_ms[e.cls] += ms;
    ctx->t_cnt[e.cls] += 1;
  }
  release_events(ctx);
  for (int i = 0; i < WDC_T_COUNT; ++i) {
    out_ms[i] = ctx->t_ms[i];
    out_count[i] = ctx->t_cnt[i];
    if (out_work) out_work[i] = ctx->t_work[i];
  }
  return WDC_OK;
}

}  // extern "C"

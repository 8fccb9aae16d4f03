// Shared device helpers and the internal launcher interface of the WorldDynCache
// rollout library (gfx950 / CDNA4 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string>

#define WDC_MAXB 17  // most latents one observation combine reads: 2 per bank slot (8) + the current one

namespace wdc {

typedef uint16_t bf16_t;  // bfloat16 bit pattern in memory
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;

__device__ __forceinline__ float bf2f(bf16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// float -> bfloat16, round to nearest even (NaN kept quiet).
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

template <typename T> __device__ __forceinline__ float ld(const T *p);
template <> __device__ __forceinline__ float ld<float>(const float *p) { return *p; }
template <> __device__ __forceinline__ float ld<bf16_t>(const bf16_t *p) { return bf2f(*p); }

template <typename T> __device__ __forceinline__ void st(T *p, float v);
template <> __device__ __forceinline__ void st<float>(float *p, float v) { *p = v; }
template <> __device__ __forceinline__ void st<bf16_t>(bf16_t *p, float v) { *p = f2bf(v); }

__device__ __forceinline__ float gelu_tanh(float x) {
  const float k0 = 0.7978845608028654f;  // sqrt(2/pi)
  float u = k0 * (x + 0.044715f * x * x * x);
  return 0.5f * x * (1.f + tanhf(u));
}

__device__ __forceinline__ float silu(float x) { return x / (1.f + expf(-x)); }

__device__ __forceinline__ float warp_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ double warp_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
// Sum over each aligned group of G consecutive lanes (G = 8 or 16) with DPP
// lane moves, no LDS round trip: lane pairs (quad permutation 1 0 3 2), pairs
// of pairs (2 3 0 1), quads (mirror within 8 lanes), halves of 16 (mirror
// within 16). After each step the two partners hold a + b and b + a, the same
// bits, so every lane of a group ends with the same sum.
template <int DPP_CTRL>
__device__ __forceinline__ float dpp_move(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), DPP_CTRL, 0xF, 0xF, false));
}
template <int G>
__device__ __forceinline__ float group_sum(float v) {
  static_assert(G == 8 || G == 16, "group of 8 or 16 lanes");
  v += dpp_move<0xB1>(v);   // quad_perm [1, 0, 3, 2]
  v += dpp_move<0x4E>(v);   // quad_perm [2, 3, 0, 1]
  v += dpp_move<0x141>(v);  // row_half_mirror
  if (G == 16) v += dpp_move<0x140>(v);  // row_mirror
  return v;
}
__device__ __forceinline__ float warp_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Block-wide sum of NV values per thread in a fixed order (deterministic);
// result valid in thread 0. blockDim.x must be a multiple of 64, <= 1024.
template <int NV>
__device__ __forceinline__ void block_sum(float (&v)[NV], float *lds /* >= 16*NV */) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
#pragma unroll
  for (int i = 0; i < NV; ++i) v[i] = warp_sum(v[i]);
  if (lane == 0)
#pragma unroll
    for (int i = 0; i < NV; ++i) lds[w * NV + i] = v[i];
  __syncthreads();
  if (threadIdx.x == 0) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      float s = 0.f;
      for (int j = 0; j < nw; ++j) s += lds[j * NV + i];
      v[i] = s;
    }
  }
  __syncthreads();
}

// ------------------------------------------------------------------ GEMM
enum Epi {
  EPI_STORE = 0,     // c = acc + bias (model dtype)
  EPI_GELU = 1,      // c = gelu_tanh(acc + bias) (model dtype)
  EPI_GATE_RES = 2,  // x (float32) += gate[n] * (acc + bias)
  EPI_STORE_F32 = 3, // c (float32) = acc + bias
  // EPI_GATE_RES with the float32 stream's read-modify-write marked
  // non-temporal; chosen by launch_gemm, not by callers
  EPI_GATE_RES_NT = 4,
  // fused projection of q, k and v (columns [0, d), [d, 2d), [2d, 3d)): the
  // bf16 result goes straight into the attention layouts with per-head
  // RMSNorm and rotary embedding on q and k (GemmArgs::qkv); no c output.
  // Only where gemm_qkv_fusable() holds.
  EPI_QKV = 5
};

// Destination of EPI_QKV. Row r of batch entry z of the product is token
// row0 + r % rps of sample z + r / rps; q and k of sample b, head h, token j at
// ((b * heads + h) * n_pad + j) * hd, v transposed at ((b * heads + h) * hd + e)
// * n_pad + vt(j), vt swapping bits 2 and 3 of j (the key order of the
// attention kernels' V^T operand).
struct QkvOut {
  void *q, *k, *v;
  const float2 *rope;     // [n_video, hd/2] (cos, sin) or null
  int64_t n_pad, n_video, rps, row0;
  int heads, hd, d, qk_norm;
};

struct GemmArgs {
  const void *a;     // [m, lda] model dtype
  const void *w;     // [n, k] model dtype
  const void *bias;  // [n] model dtype (may be null)
  void *c;           // output, see Epi
  const float *gate; // [n] float32 (EPI_GATE_RES)
  int64_t lda, ldc;
  int64_t m, n, k;
  int epi;
  // batch of independent products on grid z: entry z reads a + z*a_bs and
  // writes c + z*c_bs (elements) with gate + z*gate_bs; batch 0 or 1 = one
  int batch;
  int64_t a_bs, c_bs, gate_bs;
  // block-to-tile order of the MFMA kernels, chosen by launch_gemm: 0 groups
  // of 8 M tiles, 1 one 8 x 4 tile rectangle per XCD per dispatch round
  int order;
  int rect_n;        // order 1: N tiles of the rectangle (32 / rect_n M tiles)
  // 1: a product whose 256 x 256 tiles would fill less than one dispatch round
  // (fewer tiles than compute units) runs on 128 x 128 tiles, four times the
  // blocks; 0: the tile size follows the shape alone
  int fill_tiles;
  QkvOut qkv;        // EPI_QKV only
};

// dtype: 0 float32, 1 bfloat16
hipError_t launch_gemm(int dtype, const GemmArgs &g, hipStream_t s);
// Whether launch_gemm runs this product (epi EPI_STORE shape) on the 256 x 256
// kernels, the only ones with the EPI_QKV epilogue.
bool gemm_qkv_fusable(int dtype, const GemmArgs &g);

// compute units of the current device (0 if the query fails)
int device_cus();

// True the first time it is called with this flag array on the current device
// (kernel attributes such as the dynamic LDS limit are set per device). A
// device id outside the array, or a failed query, always answers true.
inline bool first_on_device(bool (&seen)[64]) {
  int d = 0;
  if (hipGetDevice(&d) != hipSuccess || d < 0 || d >= 64) return true;
  if (seen[d]) return false;
  seen[d] = true;
  return true;
}

// ------------------------------------------------------------------ attention
struct AttnArgs {
  const void *q, *k, *v;  // see wdc_attention
  void *o;
  int64_t n, n_pad, ldo;
  int heads, hd;
  int xcd_order;          // 1: blocks of one head run together on one XCD (heads % 8 == 0)
  // heads per sample when several samples share one launch: head index h is
  // (sample h / hpb, head h % hpb), whose rows start at sample * n in o;
  // 0 = one sample
  int hpb;
  // Scratch for splitting the key range of the last, partly filled dispatch
  // round (bf16): part (part_bytes) takes each key range's unnormalised rows,
  // reference maxima and row sums until a second launch combines them. Null:
  // no split.
  float *part;
  size_t part_bytes;
  int force_splits;       // 0: by the cost estimate; 1: never split; s >= 2: s splits whenever a round is partial
  // set by launch_attention: query blocks per head that run over all keys
  // (the rest run as kv_splits key ranges each)
  int qb_main, kv_splits;
};
int64_t attn_pad(int64_t n);
// The bf16 attention kernel addresses one head's padded rows of q, k and v^T
// with 32-bit byte offsets (buffer ranges, tile offsets): keep a head within 2^30 B.
inline bool attn_len_ok(int64_t n, int hd) { return attn_pad(n) * hd * 2 <= (int64_t(1) << 30); }
// Sets qb_main and kv_splits of a bf16 launch (every query block over all
// keys unless the scratch allows and the estimate favours a split).
void attn_split_plan(AttnArgs &a);
hipError_t launch_attention(int dtype, const AttnArgs &a, hipStream_t s);

// ------------------------------------------------------------------ elementwise and small kernels
// h[r, :] = LN(x[r, :]) * (1 + scale) + shift; x float32, h model dtype.
// Rows come in groups of rps (one sample each): logical row i is row
// (i / rps) * sstride + i % rps of x and h, and uses shift/scale + (i / rps) * mstride.
struct LnRows {
  int64_t rows;             // logical rows in total
  int64_t rps, sstride;     // rows per sample, row distance between samples
  int64_t mstride;          // floats between samples' shift/scale vectors
};
hipError_t launch_ln_mod(int dtype, const float *x, int64_t ldx, void *h, int64_t ldh, const LnRows &r, int d,
                         const float *shift, const float *scale, hipStream_t s);

// Split q/k/v from a fused projection output into attention layout; per-head
// RMSNorm on q and k, rotary embedding on video rows.
struct QKVPrepArgs {
  const void *src;        // rows [r0, r1) of the joint sequence, row stride ld (model dtype)
  int64_t ld;
  int64_t row0, rows;     // joint-sequence index of the first source row, number of rows
  int64_t n_video;        // rows with joint index < n_video get RoPE
  int64_t n_pad;
  void *q, *k, *v;        // [H, n_pad, hd]; v transposed [H, hd, n_pad] for bf16
  int heads, hd, d;       // d = heads*hd; q at columns [0,d), k [d,2d), v [2d,3d)
  int qk_norm;
  const float2 *rope;     // [n_video, hd/2] (cos, sin) or null
};
hipError_t launch_qkv_prep(int dtype, const QKVPrepArgs &a, hipStream_t s);
// zero rows [n, n_pad) of q, k and the matching columns of v
hipError_t launch_qkv_pad(int dtype, void *q, void *k, void *v, int heads, int hd, int64_t n, int64_t n_pad,
                          hipStream_t s);

// y[i] = sum_j W[i, j] * act(x[j]) + b[i] (+ y[i] if accumulate); act = SiLU if silu_in.
hipError_t launch_gemv(int dtype, const void *w, const void *b, const float *x, float *y, int n, int k, int silu_in,
                       int accumulate, hipStream_t s);
// sinusoidal timestep features (256) of 1000 t, computed in double
hipError_t launch_timestep_features(double t, float *out, hipStream_t s);
// convert a model-dtype vector to float32
hipError_t launch_to_f32(int dtype, const void *src, float *dst, int64_t n, hipStream_t s);
// z [C,F,H,W] f32 -> patches [Nv, C*pt*ph*pw] model dtype
hipError_t launch_patchify(int dtype, const float *z, void *out, int c, int f, int h, int w, int pt, int ph, int pw,
                           hipStream_t s);
// tokens [Nv, P] f32 -> v [C,F,H,W] f32
hipError_t launch_unpatchify(const float *tok, float *v, int c, int f, int h, int w, int pt, int ph, int pw,
                             hipStream_t s);
hipError_t launch_fill_normal(int dtype, void *dst, int64_t n, uint64_t seed, uint64_t offset, float std,
                              hipStream_t s);
hipError_t launch_copy_rows_f32(const float *src, int64_t lds, float *dst, int64_t ldd, int64_t rows, int64_t cols,
                                hipStream_t s);

// ------------------------------------------------------------------ surrogate / risk kernels
// A latent [C, T] (T = F*H*W) is split into C*G8 segments: segment (c, g) is
// the flat spatial indices j of channel c with floor(j*G8/T) = g.
struct SegPlan {
  int c;
  int64_t t;
  int g;       // chunks per channel (8)
  int splits;  // blocks per segment
  int vec;     // 16-byte vector access (set per launch from the buffers' alignment)
  int nseg() const { return c * g; }
  int nblocks() const { return c * g * splits; }
};
SegPlan make_seg_plan(int c, int64_t t, int g);

// values per block of each stats kernel; the observation kernel emits the
// PRE_NV statistics of zhat (against its anchor) and then a non-finite count
enum { PRE_NV = 6, OBS_NV = PRE_NV + 1, POST_NV = 10 };

// K8: z, optional anchor za -> per block [sum z, sum d, sum z^2, sum d^2, sum|d|, sum|za|], d = z - za
hipError_t launch_stats_pre(const SegPlan &pl, const float *z, const float *za, float *partials, hipStream_t s);
// K9: zhat = sum_j kappa_j out_j (j < m, slot order); per block the K8 statistics
// of zhat against za (za may be null) followed by the count of non-finite zhat values
hipError_t launch_observe(const SegPlan &pl, const float *const *outs, const float *kappa, int m, const float *za,
                          float *zhat, float *partials, hipStream_t s);
// K7: exact-step epilogue. If v: zn = z + dt*v and zn is written to zn_out; else zn is read from zn_in.
// Copies zn to bank_slot and z to anchor_out and in_slot (each when non-null). Per block:
// [sum zn, sum (zn-za), sum (zn-z), sum zn^2, sum (zn-za)^2, sum (zn-z)^2, sum|zn-zhat|, sum|zn|,
//  sum|zn-z|, sum|z|]; entries 0, 2, 3, 5, 8, 9 are the K8 statistics of zn against the anchor z
struct PostArgs {
  const float *z, *v, *zn_in, *za, *zhat;
  float dt;
  float *zn_out, *bank_slot, *anchor_out, *in_slot;
  int has_anchor, has_zhat;
};
hipError_t launch_exact_post(const SegPlan &pl, const PostArgs &a, float *partials, hipStream_t s);
// sum partials over splits in a fixed order: [nseg, splits, nv] -> [nseg, nv] double
hipError_t launch_reduce_partials(const SegPlan &pl, const float *partials, int nv, double *out, hipStream_t s);
hipError_t launch_psi(const float *z, const float *v, float dt, float *zn, int64_t n, hipStream_t s);

// Fixed device scratch of the allocation-free surrogate step (one array per
// device, held until the process ends): per-block partial sums of the
// statistics kernels at offset 0, their per-segment float64 reductions at
// kScratchRedOffset. Sized for the largest plan (16 channels x 8 segments x
// 64 slices, POST_NV values each).
constexpr size_t kScratchRedOffset = (size_t)16 * 8 * 64 * POST_NV * sizeof(float);
constexpr size_t kScratchBytes = kScratchRedOffset + (size_t)16 * 8 * POST_NV * sizeof(double);
// Device address of that array on the current device, looked up once per device.
hipError_t scratch_address(void **out);

}  // namespace wdc

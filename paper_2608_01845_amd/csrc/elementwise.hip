// Memory-bound kernels of the denoiser: LayerNorm + adaLN modulation, q/k/v
// preparation (per-head RMSNorm, 3D rotary embedding, attention layouts),
// conditioning GEMVs, patch (un)folding and seeded initialisation.
#include "common.h"

namespace wdc {

namespace {

// ---------------------------------------------------------------- LayerNorm + modulate
// One 256-thread block per row; the row stays in registers between the two
// passes (mean, then variance of the centred values).
template <typename T, int MAXV>
__global__ __launch_bounds__(256) void k_ln_mod(const float *__restrict__ x, int64_t ldx, T *__restrict__ h,
                                               int64_t ldh, LnRows lr, int d, const float *__restrict__ shift,
                                               const float *__restrict__ scale) {
  __shared__ float red[8];
  const int64_t i = blockIdx.x;
  const int64_t smp = i / lr.rps;
  const int64_t r = smp * lr.sstride + i % lr.rps;
  shift += smp * lr.mstride;
  scale += smp * lr.mstride;
  const float *xr = x + r * ldx;
  float v[MAXV];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    int c = threadIdx.x + i * 256;
    v[i] = c < d ? xr[c] : 0.f;
    s += v[i];
  }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  s = warp_sum(s);
  if (lane == 0) red[w] = s;
  __syncthreads();
  const float mean = (red[0] + red[1] + red[2] + red[3]) / (float)d;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    int c = threadIdx.x + i * 256;
    float t = c < d ? v[i] - mean : 0.f;
    q += t * t;
  }
  q = warp_sum(q);
  if (lane == 0) red[4 + w] = q;
  __syncthreads();
  const float var = (red[4] + red[5] + red[6] + red[7]) / (float)d;
  const float rstd = rsqrtf(var + 1e-6f);
  T *hr = h + r * ldh;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    int c = threadIdx.x + i * 256;
    if (c < d) st<T>(hr + c, (v[i] - mean) * rstd * (1.f + scale[c]) + shift[c]);
  }
}

// ---------------------------------------------------------------- q/k preparation
// One thread per rotary pair (2p, 2p+1) of one head of one row. The hd/2
// threads of a head sit in one wavefront, so the RMS reduction is a shuffle.
template <typename T, int HALF>
__global__ __launch_bounds__(256) void k_qk_prep(QKVPrepArgs a) {
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int p = (int)(gid % HALF);
  const int64_t rh = gid / HALF;
  const int h = (int)(rh % a.heads);
  const int64_t r = rh / a.heads;
  const bool live = r < a.rows;
  const int64_t rr = live ? r : 0;
  const T *src = (const T *)a.src + rr * a.ld + (int64_t)h * a.hd + 2 * p;
  float q0 = ld<T>(src), q1 = ld<T>(src + 1);
  float k0 = ld<T>(src + a.d), k1 = ld<T>(src + a.d + 1);
  if (a.qk_norm) {
    float sq = q0 * q0 + q1 * q1, sk = k0 * k0 + k1 * k1;
#pragma unroll
    for (int o = HALF / 2; o > 0; o >>= 1) {
      sq += __shfl_xor(sq, o, 64);
      sk += __shfl_xor(sk, o, 64);
    }
    const float rq = rsqrtf(sq / (float)a.hd + 1e-6f), rk = rsqrtf(sk / (float)a.hd + 1e-6f);
    q0 *= rq;
    q1 *= rq;
    k0 *= rk;
    k1 *= rk;
  }
  const int64_t j = a.row0 + rr;  // joint-sequence index
  if (a.rope && j < a.n_video) {
    float2 cs = a.rope[j * HALF + p];
    float t0 = q0 * cs.x - q1 * cs.y, t1 = q0 * cs.y + q1 * cs.x;
    q0 = t0;
    q1 = t1;
    t0 = k0 * cs.x - k1 * cs.y;
    t1 = k0 * cs.y + k1 * cs.x;
    k0 = t0;
    k1 = t1;
  }
  if (!live) return;
  const int64_t o = ((int64_t)h * a.n_pad + j) * a.hd + 2 * p;
  st<T>((T *)a.q + o, q0);
  st<T>((T *)a.q + o + 1, q1);
  st<T>((T *)a.k + o, k0);
  st<T>((T *)a.k + o + 1, k1);
}

// v rows -> [H, n_pad, hd] (float32 attention path)
template <typename T>
__global__ __launch_bounds__(256) void k_v_copy(QKVPrepArgs a) {
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int c = (int)(gid % a.d);
  const int64_t r = gid / a.d;
  if (r >= a.rows) return;
  const int h = c / a.hd, e = c % a.hd;
  const T *src = (const T *)a.src + r * a.ld + 2 * a.d + c;
  ((T *)a.v)[((int64_t)h * a.n_pad + a.row0 + r) * a.hd + e] = *src;
}

// Position of key j in a V^T row: inside each aligned group of 16 keys the
// order is 0-3, 8-11, 4-7, 12-15 (bits 2 and 3 of j swapped), which makes the 8
// keys one lane feeds to an O^T = V^T P^T step one 16-byte chunk.
__device__ __forceinline__ int64_t vt_pos(int64_t j) { return (j & ~(int64_t)12) | ((j & 4) << 1) | ((j & 8) >> 1); }

// v rows -> transposed [H, hd, n_pad] through a 64-row LDS tile, so that both
// the reads (rows of the projection output) and the writes (runs of 64 tokens)
// are coalesced.
__global__ __launch_bounds__(256) void k_v_transpose(QKVPrepArgs a) {
  __shared__ bf16_t tile[64][128 + 2];
  const int h = blockIdx.y;
  const int64_t r0 = (int64_t)blockIdx.x * 64;
  for (int idx = threadIdx.x; idx < 64 * a.hd; idx += 256) {
    int rr = idx / a.hd, e = idx % a.hd;
    int64_t r = r0 + rr;
    bf16_t val = 0;
    if (r < a.rows) val = ((const bf16_t *)a.src)[r * a.ld + 2 * a.d + (int64_t)h * a.hd + e];
    tile[rr][e] = val;
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < 64 * a.hd; idx += 256) {
    int e = idx / 64, rr = idx % 64;
    int64_t r = r0 + rr;
    if (r < a.rows) ((bf16_t *)a.v)[((int64_t)h * a.hd + e) * a.n_pad + vt_pos(a.row0 + r)] = tile[rr][e];
  }
}

// bf16 forms of the two kernels above with 16-byte accesses.
// q/k: one thread per 8 consecutive elements (4 rotary pairs) of one head row;
// the HD/8 threads of a head row are consecutive lanes of one wavefront, so the
// RMS reduction is a butterfly over them. Same arithmetic per element as
// k_qk_prep (float32, RMS scale, then rotation, one bf16 rounding).
__device__ __forceinline__ void unpack8(const uint4 &u, float (&x)[8]) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
// eight floats -> bf16 (round to nearest even, four v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint4 pack8(const float (&x)[8]) {
  typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_v;
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    bf16x2_v p;
    p[0] = (__bf16)x[2 * i];
    p[1] = (__bf16)x[2 * i + 1];
    w[i] = __builtin_bit_cast(uint32_t, p);
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// (No fused multiply-adds in the norm and rotation arithmetic, here and in the
// GEMM's fused q/k epilogue, so both give the same bits.)
template <int HD>
__global__ __launch_bounds__(256) void k_qk_prep8(QKVPrepArgs a) {
#pragma clang fp contract(off)
  constexpr int TPH = HD / 8;              // threads per head row
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int c = (int)(gid % TPH);
  const int64_t rh = gid / TPH;
  const int h = (int)(rh % a.heads);
  const int64_t r = rh / a.heads;
  const bool live = r < a.rows;
  const int64_t rr = live ? r : 0;
  const bf16_t *src = (const bf16_t *)a.src + rr * a.ld + (int64_t)h * HD + 8 * c;
  float q[8], k[8];
  unpack8(*(const uint4 *)src, q);
  unpack8(*(const uint4 *)(src + a.d), k);
  if (a.qk_norm) {
    float sq = 0.f, sk = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      sq += q[e] * q[e];
      sk += k[e] * k[e];
    }
    sq = group_sum<TPH>(sq);
    sk = group_sum<TPH>(sk);
    const float rq = rsqrtf(sq / (float)HD + 1e-6f), rk = rsqrtf(sk / (float)HD + 1e-6f);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      q[e] *= rq;
      k[e] *= rk;
    }
  }
  const int64_t j = a.row0 + rr;           // joint-sequence index
  if (a.rope && j < a.n_video) {
    const float4 *cs4 = (const float4 *)(a.rope + j * (HD / 2) + 4 * c);
    const float4 c01 = cs4[0], c23 = cs4[1];
    const float cs[8] = {c01.x, c01.y, c01.z, c01.w, c23.x, c23.y, c23.z, c23.w};
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const float co = cs[2 * p], si = cs[2 * p + 1];
      float t0 = q[2 * p] * co - q[2 * p + 1] * si, t1 = q[2 * p] * si + q[2 * p + 1] * co;
      q[2 * p] = t0;
      q[2 * p + 1] = t1;
      t0 = k[2 * p] * co - k[2 * p + 1] * si;
      t1 = k[2 * p] * si + k[2 * p + 1] * co;
      k[2 * p] = t0;
      k[2 * p + 1] = t1;
    }
  }
  if (!live) return;
  const int64_t o = ((int64_t)h * a.n_pad + j) * HD + 8 * c;
  *(uint4 *)((bf16_t *)a.q + o) = pack8(q);
  *(uint4 *)((bf16_t *)a.k + o) = pack8(k);
}

// V^T through a 64-row LDS tile with 16-byte row reads and 16-byte writes of 8
// consecutive V^T positions. Needs row0 % 16 == 0: then the key order of
// vt_pos permutes tokens only inside each aligned group of 16 of this tile, and
// output position p holds token vt_pos(p) (the permutation is its own
// inverse). Groups of 16 with rows missing are written element by element,
// valid tokens only (their other positions are padding, zeroed separately).
template <int HD>
__global__ __launch_bounds__(256) void k_v_transpose8(QKVPrepArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t tile[64][HD + 8];
  const int h = blockIdx.y;
  const int64_t r0 = (int64_t)blockIdx.x * 64;
  for (int idx = threadIdx.x; idx < 64 * (HD / 8); idx += 256) {
    const int rr = idx / (HD / 8), c = idx % (HD / 8);
    const int64_t r = r0 + rr;
    uint4 val = make_uint4(0, 0, 0, 0);
    if (r < a.rows) val = *(const uint4 *)((const bf16_t *)a.src + r * a.ld + 2 * a.d + (int64_t)h * HD + 8 * c);
    *(uint4 *)&tile[rr][8 * c] = val;
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < HD * 8; idx += 256) {
    const int e = idx / 8, c = idx % 8;    // feature row, 8-position chunk of the tile
    int tok[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) tok[i] = (int)vt_pos(8 * c + i);
    bf16_t *dst = (bf16_t *)a.v + ((int64_t)h * HD + e) * a.n_pad + a.row0 + r0 + 8 * c;
    const int64_t group_end = r0 + (8 * c / 16) * 16 + 16;   // rows this chunk's group needs
    if (group_end <= a.rows) {
      uint32_t w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        w[i] = (uint32_t)tile[tok[2 * i]][e] | ((uint32_t)tile[tok[2 * i + 1]][e] << 16);
      *(uint4 *)dst = make_uint4(w[0], w[1], w[2], w[3]);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (r0 + tok[i] < a.rows) dst[i] = tile[tok[i]][e];
    }
  }
}

template <typename T>
__global__ void k_qkv_pad(T *q, T *k, T *v, int heads, int hd, int64_t n, int64_t n_pad, int v_transposed) {
  const int64_t tail = n_pad - n;
  const int64_t total = (int64_t)heads * tail * hd;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    int e = (int)(i % hd);
    int64_t rt = (i / hd) % tail;
    int h = (int)(i / ((int64_t)hd * tail));
    int64_t row = n + rt;
    int64_t o = ((int64_t)h * n_pad + row) * hd + e;
    q[o] = 0;
    k[o] = 0;
    if (v_transposed)
      v[((int64_t)h * hd + e) * n_pad + vt_pos(row)] = 0;
    else
      v[o] = 0;
  }
}

// ---------------------------------------------------------------- GEMV (conditioning)
// One wavefront per output row; 16-byte loads along the input dimension.
template <typename T>
__global__ __launch_bounds__(256) void k_gemv(const T *__restrict__ w, const T *__restrict__ b,
                                             const float *__restrict__ x, float *__restrict__ y, int n, int k,
                                             int silu_in, int accumulate) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n) return;
  const T *wr = w + (int64_t)row * k;
  float acc = 0.f;
  for (int j = lane; j < k; j += 64) {
    float xv = x[j];
    if (silu_in) xv = silu(xv);
    acc += ld<T>(wr + j) * xv;
  }
  acc = warp_sum(acc);
  if (lane == 0) {
    float out = acc + (b ? ld<T>(b + row) : 0.f);
    y[row] = accumulate ? y[row] + out : out;
  }
}

// 16-byte vectorised bf16 variant for k % 512 == 0
__global__ __launch_bounds__(256) void k_gemv_bf16_v(const bf16_t *__restrict__ w, const bf16_t *__restrict__ b,
                                                    const float *__restrict__ x, float *__restrict__ y, int n, int k,
                                                    int silu_in, int accumulate) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n) return;
  const uint4 *wr = (const uint4 *)(w + (int64_t)row * k);
  float acc = 0.f;
  for (int j = lane; j < k / 8; j += 64) {
    uint4 pk = wr[j];
    const float *xp = x + j * 8;
    uint32_t u[4] = {pk.x, pk.y, pk.z, pk.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float x0 = xp[2 * e], x1 = xp[2 * e + 1];
      if (silu_in) {
        x0 = silu(x0);
        x1 = silu(x1);
      }
      acc += __uint_as_float(u[e] << 16) * x0 + __uint_as_float(u[e] & 0xffff0000u) * x1;
    }
  }
  acc = warp_sum(acc);
  if (lane == 0) {
    float out = acc + (b ? bf2f(b[row]) : 0.f);
    y[row] = accumulate ? y[row] + out : out;
  }
}

__global__ void k_timestep(double t, float *out) {
  int j = threadIdx.x;
  if (j >= 128) return;
  double f = exp(-log(10000.0) * (double)j / 128.0);
  double arg = 1000.0 * t * f;
  out[j] = (float)cos(arg);
  out[128 + j] = (float)sin(arg);
}

template <typename T>
__global__ void k_to_f32(const T *src, float *dst, int64_t n) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = ld<T>(src + i);
}

// ---------------------------------------------------------------- patches
template <typename T>
__global__ void k_patchify(const float *__restrict__ z, T *__restrict__ out, int c, int f, int h, int w, int pt,
                           int ph, int pw) {
  const int fp = f / pt, hp = h / ph, wp = w / pw;
  const int P = c * pt * ph * pw;
  const int64_t total = (int64_t)fp * hp * wp * P;
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  int feat = (int)(i % P);
  int64_t n = i / P;
  int wq = (int)(n % wp), hq = (int)((n / wp) % hp), fq = (int)(n / ((int64_t)wp * hp));
  int jj = feat % pw, ii = (feat / pw) % ph, aa = (feat / (pw * ph)) % pt, cc = feat / (pw * ph * pt);
  int64_t src = (((int64_t)cc * f + (fq * pt + aa)) * h + (hq * ph + ii)) * w + (wq * pw + jj);
  st<T>(out + i, z[src]);
}

__global__ void k_unpatchify(const float *__restrict__ tok, float *__restrict__ v, int c, int f, int h, int w, int pt,
                             int ph, int pw) {
  const int64_t total = (int64_t)c * f * h * w;
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  int x = (int)(i % w), y = (int)((i / w) % h), fr = (int)((i / ((int64_t)w * h)) % f), cc = (int)(i / ((int64_t)w * h * f));
  const int fp = f / pt, hp = h / ph, wp = w / pw;
  (void)fp;
  int64_t n = ((int64_t)(fr / pt) * hp + (y / ph)) * wp + (x / pw);
  int feat = ((cc * pt + fr % pt) * ph + y % ph) * pw + x % pw;
  v[i] = tok[n * (int64_t)(c * pt * ph * pw) + feat];
}

// ---------------------------------------------------------------- seeded normal fill
// splitmix64 of (seed, counter) -> two 32-bit uniforms -> Box-Muller.
__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
  x += 0x9e3779b97f4a7c15ull;
  x = (x ^ (x >> 30)) * 0xbf58476d1ce4e5b9ull;
  x = (x ^ (x >> 27)) * 0x94d049bb133111ebull;
  return x ^ (x >> 31);
}

template <typename T>
__global__ void k_fill_normal(T *dst, int64_t n, uint64_t seed, uint64_t offset, float std) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) {
    uint64_t r = splitmix64(seed * 0x632be59bd9b4e019ull + offset + (uint64_t)i);
    float u1 = ((uint32_t)(r >> 32) + 1.0f) * 2.3283064365386963e-10f;  // (0, 1]
    float u2 = (uint32_t)r * 2.3283064365386963e-10f;
    float g = sqrtf(-2.f * logf(u1)) * cosf(6.283185307179586f * u2);
    st<T>(dst + i, g * std);
  }
}

__global__ void k_copy_rows(const float *src, int64_t lds, float *dst, int64_t ldd, int64_t rows, int64_t cols) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * cols) return;
  int64_t r = i / cols, c = i % cols;
  dst[r * ldd + c] = src[r * lds + c];
}

inline unsigned nblk(int64_t n, int t) { return (unsigned)((n + t - 1) / t); }
}  // namespace

// Vector form (d % 4 == 0, 16-byte aligned rows): thread t owns the float4
// groups t, t + 256, ... of the row; bf16 output goes out as 8-byte groups.
template <typename T>
__device__ __forceinline__ void st4(T *p, float a, float b, float c, float d);
template <>
__device__ __forceinline__ void st4<bf16_t>(bf16_t *p, float a, float b, float c, float d) {
  *(uint2 *)p = make_uint2((uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16), (uint32_t)f2bf(c) | ((uint32_t)f2bf(d) << 16));
}
template <>
__device__ __forceinline__ void st4<float>(float *p, float a, float b, float c, float d) {
  *(float4 *)p = make_float4(a, b, c, d);
}

template <typename T, int NV4>
__global__ __launch_bounds__(256) void k_ln_mod4(const float *__restrict__ x, int64_t ldx, T *__restrict__ h,
                                                int64_t ldh, LnRows lr, int d, const float *__restrict__ shift,
                                                const float *__restrict__ scale) {
  __shared__ float red[8];
  const int64_t i = blockIdx.x;
  const int64_t smp = i / lr.rps;
  const int64_t r = smp * lr.sstride + i % lr.rps;
  shift += smp * lr.mstride;
  scale += smp * lr.mstride;
  const float4 *xr = (const float4 *)(x + r * ldx);
  const int d4 = d >> 2;
  float4 v[NV4];
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < NV4; ++k) {
    const int c = threadIdx.x + k * 256;
    v[k] = c < d4 ? xr[c] : make_float4(0.f, 0.f, 0.f, 0.f);
    s += (v[k].x + v[k].y) + (v[k].z + v[k].w);
  }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  s = warp_sum(s);
  if (lane == 0) red[w] = s;
  __syncthreads();
  const float mean = (red[0] + red[1] + red[2] + red[3]) / (float)d;
  float q = 0.f;
#pragma unroll
  for (int k = 0; k < NV4; ++k) {
    const int c = threadIdx.x + k * 256;
    if (c < d4) {
      const float a = v[k].x - mean, b = v[k].y - mean, e = v[k].z - mean, f = v[k].w - mean;
      q += (a * a + b * b) + (e * e + f * f);
    }
  }
  q = warp_sum(q);
  if (lane == 0) red[4 + w] = q;
  __syncthreads();
  const float var = (red[4] + red[5] + red[6] + red[7]) / (float)d;
  const float rstd = rsqrtf(var + 1e-6f);
  T *hr = h + r * ldh;
#pragma unroll
  for (int k = 0; k < NV4; ++k) {
    const int c = threadIdx.x + k * 256;
    if (c < d4) {
      const float4 sh = ((const float4 *)shift)[c], sc = ((const float4 *)scale)[c];
      st4<T>(hr + 4 * c, (v[k].x - mean) * rstd * (1.f + sc.x) + sh.x, (v[k].y - mean) * rstd * (1.f + sc.y) + sh.y,
             (v[k].z - mean) * rstd * (1.f + sc.z) + sh.z, (v[k].w - mean) * rstd * (1.f + sc.w) + sh.w);
    }
  }
}

hipError_t launch_ln_mod(int dtype, const float *x, int64_t ldx, void *h, int64_t ldh, const LnRows &r, int d,
                         const float *shift, const float *scale, hipStream_t s) {
  if (r.rows <= 0) return hipSuccess;
  if (d > 16 * 256 || r.rps <= 0 || r.sstride < r.rps) return hipErrorInvalidValue;
  dim3 g((unsigned)r.rows), b(256);
  const bool vec = d % 4 == 0 && ldx % 4 == 0 && ldh % 4 == 0 && r.mstride % 4 == 0 && (uintptr_t)x % 16 == 0 &&
                   (uintptr_t)h % 16 == 0 && (uintptr_t)shift % 16 == 0 && (uintptr_t)scale % 16 == 0;
  if (vec) {
    if (dtype == 1) {
      if (d <= 4 * 256)
        hipLaunchKernelGGL((k_ln_mod4<bf16_t, 1>), g, b, 0, s, x, ldx, (bf16_t *)h, ldh, r, d, shift, scale);
      else
        hipLaunchKernelGGL((k_ln_mod4<bf16_t, 4>), g, b, 0, s, x, ldx, (bf16_t *)h, ldh, r, d, shift, scale);
    } else {
      if (d <= 4 * 256)
        hipLaunchKernelGGL((k_ln_mod4<float, 1>), g, b, 0, s, x, ldx, (float *)h, ldh, r, d, shift, scale);
      else
        hipLaunchKernelGGL((k_ln_mod4<float, 4>), g, b, 0, s, x, ldx, (float *)h, ldh, r, d, shift, scale);
    }
    return hipGetLastError();
  }
  if (dtype == 1) {
    if (d <= 4 * 256)
      hipLaunchKernelGGL((k_ln_mod<bf16_t, 4>), g, b, 0, s, x, ldx, (bf16_t *)h, ldh, r, d, shift, scale);
    else
      hipLaunchKernelGGL((k_ln_mod<bf16_t, 16>), g, b, 0, s, x, ldx, (bf16_t *)h, ldh, r, d, shift, scale);
  } else {
    if (d <= 4 * 256)
      hipLaunchKernelGGL((k_ln_mod<float, 4>), g, b, 0, s, x, ldx, (float *)h, ldh, r, d, shift, scale);
    else
      hipLaunchKernelGGL((k_ln_mod<float, 16>), g, b, 0, s, x, ldx, (float *)h, ldh, r, d, shift, scale);
  }
  return hipGetLastError();
}

hipError_t launch_qkv_prep(int dtype, const QKVPrepArgs &a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  if (a.hd != 64 && a.hd != 128) return hipErrorInvalidValue;
  const int64_t threads = a.rows * a.heads * (a.hd / 2);
  dim3 g(nblk(threads, 256)), b(256);
  if (dtype == 1) {
    // 16-byte forms when every row and head start is 16-byte aligned
    const bool vec = (uintptr_t)a.src % 16 == 0 && a.ld % 8 == 0 && a.d % 8 == 0 && (uintptr_t)a.q % 16 == 0 &&
                     (uintptr_t)a.k % 16 == 0 && (uintptr_t)a.v % 16 == 0 && a.n_pad % 8 == 0 &&
                     (a.rope == nullptr || (uintptr_t)a.rope % 16 == 0);
    if (vec) {
      const dim3 g8(nblk(a.rows * a.heads * (a.hd / 8), 256));
      if (a.hd == 64)
        hipLaunchKernelGGL(k_qk_prep8<64>, g8, b, 0, s, a);
      else
        hipLaunchKernelGGL(k_qk_prep8<128>, g8, b, 0, s, a);
    } else if (a.hd == 64) {
      hipLaunchKernelGGL((k_qk_prep<bf16_t, 32>), g, b, 0, s, a);
    } else {
      hipLaunchKernelGGL((k_qk_prep<bf16_t, 64>), g, b, 0, s, a);
    }
    const dim3 gv(nblk(a.rows, 64), a.heads);
    if (vec && a.row0 % 16 == 0) {
      if (a.hd == 64)
        hipLaunchKernelGGL(k_v_transpose8<64>, gv, dim3(256), 0, s, a);
      else
        hipLaunchKernelGGL(k_v_transpose8<128>, gv, dim3(256), 0, s, a);
    } else {
      hipLaunchKernelGGL(k_v_transpose, gv, dim3(256), 0, s, a);
    }
  } else {
    if (a.hd == 64)
      hipLaunchKernelGGL((k_qk_prep<float, 32>), g, b, 0, s, a);
    else
      hipLaunchKernelGGL((k_qk_prep<float, 64>), g, b, 0, s, a);
    hipLaunchKernelGGL((k_v_copy<float>), dim3(nblk(a.rows * a.d, 256)), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_qkv_pad(int dtype, void *q, void *k, void *v, int heads, int hd, int64_t n, int64_t n_pad,
                          hipStream_t s) {
  if (n_pad <= n) return hipSuccess;
  int64_t total = (int64_t)heads * (n_pad - n) * hd;
  unsigned g = nblk(total, 256);
  if (g > 4096) g = 4096;
  if (dtype == 1)
    hipLaunchKernelGGL((k_qkv_pad<bf16_t>), dim3(g), dim3(256), 0, s, (bf16_t *)q, (bf16_t *)k, (bf16_t *)v, heads,
                       hd, n, n_pad, 1);
  else
    hipLaunchKernelGGL((k_qkv_pad<float>), dim3(g), dim3(256), 0, s, (float *)q, (float *)k, (float *)v, heads, hd,
                       n, n_pad, 0);
  return hipGetLastError();
}

hipError_t launch_gemv(int dtype, const void *w, const void *b, const float *x, float *y, int n, int k, int silu_in,
                       int accumulate, hipStream_t s) {
  dim3 g(nblk(n, 4)), bl(256);
  if (dtype == 1) {
    if (k % 512 == 0 && ((uintptr_t)w & 15) == 0)
      hipLaunchKernelGGL(k_gemv_bf16_v, g, bl, 0, s, (const bf16_t *)w, (const bf16_t *)b, x, y, n, k, silu_in,
                         accumulate);
    else
      hipLaunchKernelGGL((k_gemv<bf16_t>), g, bl, 0, s, (const bf16_t *)w, (const bf16_t *)b, x, y, n, k, silu_in,
                         accumulate);
  } else {
    hipLaunchKernelGGL((k_gemv<float>), g, bl, 0, s, (const float *)w, (const float *)b, x, y, n, k, silu_in,
                       accumulate);
  }
  return hipGetLastError();
}

hipError_t launch_timestep_features(double t, float *out, hipStream_t s) {
  hipLaunchKernelGGL(k_timestep, dim3(1), dim3(128), 0, s, t, out);
  return hipGetLastError();
}

hipError_t launch_to_f32(int dtype, const void *src, float *dst, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (dtype == 1)
    hipLaunchKernelGGL((k_to_f32<bf16_t>), dim3(nblk(n, 256)), dim3(256), 0, s, (const bf16_t *)src, dst, n);
  else
    hipLaunchKernelGGL((k_to_f32<float>), dim3(nblk(n, 256)), dim3(256), 0, s, (const float *)src, dst, n);
  return hipGetLastError();
}

hipError_t launch_patchify(int dtype, const float *z, void *out, int c, int f, int h, int w, int pt, int ph, int pw,
                           hipStream_t s) {
  int64_t total = (int64_t)c * f * h * w;
  if (dtype == 1)
    hipLaunchKernelGGL((k_patchify<bf16_t>), dim3(nblk(total, 256)), dim3(256), 0, s, z, (bf16_t *)out, c, f, h, w,
                       pt, ph, pw);
  else
    hipLaunchKernelGGL((k_patchify<float>), dim3(nblk(total, 256)), dim3(256), 0, s, z, (float *)out, c, f, h, w, pt,
                       ph, pw);
  return hipGetLastError();
}

hipError_t launch_unpatchify(const float *tok, float *v, int c, int f, int h, int w, int pt, int ph, int pw,
                             hipStream_t s) {
  int64_t total = (int64_t)c * f * h * w;
  hipLaunchKernelGGL(k_unpatchify, dim3(nblk(total, 256)), dim3(256), 0, s, tok, v, c, f, h, w, pt, ph, pw);
  return hipGetLastError();
}

hipError_t launch_fill_normal(int dtype, void *dst, int64_t n, uint64_t seed, uint64_t offset, float std,
                              hipStream_t s) {
  if (n <= 0) return hipSuccess;
  unsigned g = nblk(n, 256);
  if (g > 65536) g = 65536;
  if (dtype == 1)
    hipLaunchKernelGGL((k_fill_normal<bf16_t>), dim3(g), dim3(256), 0, s, (bf16_t *)dst, n, seed, offset, std);
  else
    hipLaunchKernelGGL((k_fill_normal<float>), dim3(g), dim3(256), 0, s, (float *)dst, n, seed, offset, std);
  return hipGetLastError();
}

hipError_t launch_copy_rows_f32(const float *src, int64_t lds, float *dst, int64_t ldd, int64_t rows, int64_t cols,
                                hipStream_t s) {
  if (rows * cols <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_copy_rows, dim3(nblk(rows * cols, 256)), dim3(256), 0, s, src, lds, dst, ldd, rows, cols);
  return hipGetLastError();
}

}  // namespace wdc

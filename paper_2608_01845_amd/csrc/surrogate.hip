// HBM-bound kernels of the surrogate and the risk controller (Sec. 4.2-4.3).
//
// The latent [C, F, H, W] is processed as C*8 contiguous segments: segment
// (c, g) holds the flat spatial indices j of channel c with floor(8j/T) = g,
// which is the finest chunking the 256-d summary pools over (coarser chunks
// nest: floor(4j/T) = floor(floor(8j/T)/2)). Each block streams one slice of
// one segment, so every per-chunk sum is a plain per-block sum and the grid
// needs no atomics; partial sums are then combined in a fixed order
// (deterministic, bit-reproducible run to run).
//
// Slices are read as 16-byte vectors when every buffer of the launch is
// 16-byte aligned: a slice is split into a scalar head (< 4 elements up to
// the first multiple of 4), a float4 body and a scalar tail.
//
// The observation and exact-step kernels also emit the pass-1 statistics of
// the latent they produce, under the anchor the next step will use, so a
// rollout reads each latent once per step (Eq. (2), (5), (6)).
#include "common.h"

#include <mutex>

// Statistics scratch of the allocation-free surrogate step (layout in common.h).
// Host code must not pass this name to a kernel: it uses the device address
// that scratch_address() looks up per device.
static __device__ __align__(256) unsigned char scratch[wdc::kScratchBytes];

namespace wdc {

namespace {
constexpr int kThreads = 256;
constexpr int64_t kSliceElems = 4096;  // target elements per block

struct SegRange {
  int64_t a, b;  // flat element range [a, b) of this block
};

__device__ __forceinline__ SegRange seg_range(int64_t t, int g, int splits) {
  const int blk = blockIdx.x;
  const int seg = blk / splits, sp = blk % splits;
  const int c = seg / g, gi = seg % g;
  const int64_t s0 = (gi * t + g - 1) / g;        // ceil(gi*T/G)
  const int64_t s1 = ((gi + 1) * t + g - 1) / g;  // ceil((gi+1)*T/G)
  const int64_t len = s1 - s0;
  SegRange r;
  r.a = (int64_t)c * t + s0 + (len * sp) / splits;
  r.b = (int64_t)c * t + s0 + (len * (sp + 1)) / splits;
  return r;
}

template <int W>
struct Vf {
  float x[W];
};

template <int W>
__device__ __forceinline__ Vf<W> ldv(const float *__restrict__ p, int64_t i) {
  Vf<W> o;
  if constexpr (W == 4) {
    const float4 t = *reinterpret_cast<const float4 *>(p + i);
    o.x[0] = t.x;
    o.x[1] = t.y;
    o.x[2] = t.z;
    o.x[3] = t.w;
  } else {
    o.x[0] = p[i];
  }
  return o;
}

template <int W>
__device__ __forceinline__ void stv(float *__restrict__ p, int64_t i, const Vf<W> &v) {
  if constexpr (W == 4) {
    *reinterpret_cast<float4 *>(p + i) = make_float4(v.x[0], v.x[1], v.x[2], v.x[3]);
  } else {
    p[i] = v.x[0];
  }
}

template <int W>
__device__ __forceinline__ Vf<W> zeros() {
  Vf<W> o;
#pragma unroll
  for (int e = 0; e < W; ++e) o.x[e] = 0.f;
  return o;
}

// Streams [a, b) through op.template step<W>(i, acc): W = 4 on aligned
// indices when vec, else W = 1.
template <int NV, class Op>
__device__ __forceinline__ void stream_range(const Op &op, SegRange r, bool vec, float (&acc)[NV]) {
  if (vec) {
    const int64_t a4 = min(r.b, (r.a + 3) & ~(int64_t)3);
    const int64_t b4 = max(a4, r.b & ~(int64_t)3);
    if (r.a + threadIdx.x < a4) op.template step<1>(r.a + threadIdx.x, acc);
#pragma unroll 2
    for (int64_t i = a4 + 4 * (int64_t)threadIdx.x; i < b4; i += 4 * kThreads) op.template step<4>(i, acc);
    if (b4 + threadIdx.x < r.b) op.template step<1>(b4 + threadIdx.x, acc);
  } else {
    for (int64_t i = r.a + threadIdx.x; i < r.b; i += kThreads) op.template step<1>(i, acc);
  }
}

template <int NV>
__device__ __forceinline__ void write_partials(float (&v)[NV], float *lds, float *__restrict__ part) {
  block_sum<NV>(v, lds);
  if (threadIdx.x == 0)
#pragma unroll
    for (int i = 0; i < NV; ++i) part[(int64_t)blockIdx.x * NV + i] = v[i];
}

// pass-1 statistics of z against the anchor za (0 without one):
// [sum z, sum d, sum z^2, sum d^2, sum |d|, sum |za|], d = z - za
template <int W>
__device__ __forceinline__ void acc_pre(const Vf<W> &z, const Vf<W> &za, float (&v)[PRE_NV]) {
#pragma unroll
  for (int e = 0; e < W; ++e) {
    const float x = z.x[e], a = za.x[e], d = x - a;
    v[0] += x;
    v[1] += d;
    v[2] += x * x;
    v[3] += d * d;
    v[4] += fabsf(d);
    v[5] += fabsf(a);
  }
}

struct PreOp {
  const float *z, *za;
  template <int W>
  __device__ __forceinline__ void step(int64_t i, float (&v)[PRE_NV]) const {
    const Vf<W> x = ldv<W>(z, i);
    const Vf<W> a = za ? ldv<W>(za, i) : zeros<W>();
    acc_pre<W>(x, a, v);
  }
};

__global__ __launch_bounds__(kThreads) void k_stats_pre(SegPlan pl, PreOp op, float *__restrict__ part) {
  __shared__ float lds[16 * PRE_NV];
  float v[PRE_NV] = {};
  stream_range<PRE_NV>(op, seg_range(pl.t, pl.g, pl.splits), pl.vec, v);
  write_partials<PRE_NV>(v, lds, part);
}

struct ObsOp {
  const float *outs[WDC_MAXB];
  float kappa[WDC_MAXB];
  int m;
  const float *za;
  float *zhat;
  template <int W>
  __device__ __forceinline__ void step(int64_t i, float (&v)[OBS_NV]) const {
    Vf<W> acc = zeros<W>();
    for (int j = 0; j < m; ++j) {
      const Vf<W> o = ldv<W>(outs[j], i);
#pragma unroll
      for (int e = 0; e < W; ++e) acc.x[e] += kappa[j] * o.x[e];
    }
    stv<W>(zhat, i, acc);
    const Vf<W> a = za ? ldv<W>(za, i) : zeros<W>();
    float pre[PRE_NV] = {};
    acc_pre<W>(acc, a, pre);
#pragma unroll
    for (int q = 0; q < PRE_NV; ++q) v[q] += pre[q];
#pragma unroll
    for (int e = 0; e < W; ++e) v[PRE_NV] += isfinite(acc.x[e]) ? 0.f : 1.f;
  }
};

__global__ __launch_bounds__(kThreads) void k_observe(SegPlan pl, ObsOp op, float *__restrict__ part) {
  __shared__ float lds[16 * OBS_NV];
  float v[OBS_NV] = {};
  stream_range<OBS_NV>(op, seg_range(pl.t, pl.g, pl.splits), pl.vec, v);
  write_partials<OBS_NV>(v, lds, part);
}

struct PostOp {
  PostArgs a;
  template <int W>
  __device__ __forceinline__ void step(int64_t i, float (&v)[POST_NV]) const {
    const Vf<W> x = ldv<W>(a.z, i);
    Vf<W> xn;
    if (a.v) {
      const Vf<W> vv = ldv<W>(a.v, i);
#pragma unroll
      for (int e = 0; e < W; ++e) xn.x[e] = x.x[e] + a.dt * vv.x[e];
      stv<W>(a.zn_out, i, xn);
    } else {
      xn = ldv<W>(a.zn_in, i);
    }
    if (a.bank_slot) stv<W>(a.bank_slot, i, xn);
    if (a.anchor_out) stv<W>(a.anchor_out, i, x);
    if (a.in_slot) stv<W>(a.in_slot, i, x);
    const Vf<W> za = a.has_anchor ? ldv<W>(a.za, i) : zeros<W>();
    const Vf<W> zh = a.has_zhat ? ldv<W>(a.zhat, i) : zeros<W>();
#pragma unroll
    for (int e = 0; e < W; ++e) {
      const float n = xn.x[e], dn = n - za.x[e], dx = n - x.x[e];
      v[0] += n;
      v[1] += dn;
      v[2] += dx;
      v[3] += n * n;
      v[4] += dn * dn;
      v[5] += dx * dx;
      v[6] += a.has_zhat ? fabsf(n - zh.x[e]) : 0.f;
      v[7] += fabsf(n);
      v[8] += fabsf(dx);
      v[9] += fabsf(x.x[e]);
    }
  }
};

__global__ __launch_bounds__(kThreads) void k_exact_post(SegPlan pl, PostOp op, float *__restrict__ part) {
  __shared__ float lds[16 * POST_NV];
  float v[POST_NV] = {};
  stream_range<POST_NV>(op, seg_range(pl.t, pl.g, pl.splits), pl.vec, v);
  write_partials<POST_NV>(v, lds, part);
}

__global__ void k_reduce(const float *__restrict__ part, int nseg, int splits, int nv, double *__restrict__ out) {
  int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= nseg * nv) return;
  int seg = idx / nv, v = idx % nv;
  double s = 0.0;
  for (int sp = 0; sp < splits; ++sp) s += (double)part[((int64_t)seg * splits + sp) * nv + v];
  out[idx] = s;
}

template <int W>
__global__ __launch_bounds__(256) void k_psi(const float *__restrict__ z, const float *__restrict__ v, float dt,
                                             float *__restrict__ zn, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x * W;
  for (int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * W; i < n; i += stride) {
    if (W == 4 && i + 4 <= n) {
      const Vf<4> a = ldv<4>(z, i), b = ldv<4>(v, i);
      Vf<4> o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o.x[e] = a.x[e] + dt * b.x[e];
      stv<4>(zn, i, o);
    } else {
      for (int64_t j = i; j < i + W && j < n; ++j) zn[j] = z[j] + dt * v[j];
    }
  }
}

bool al16(const void *p) { return ((uintptr_t)p & 15) == 0; }
}  // namespace

SegPlan make_seg_plan(int c, int64_t t, int g) {
  SegPlan p;
  p.c = c;
  p.t = t;
  p.g = g;
  p.vec = 1;
  int64_t seglen = (t + g - 1) / g;
  int64_t sp = (seglen + kSliceElems - 1) / kSliceElems;
  p.splits = (int)(sp < 1 ? 1 : (sp > 64 ? 64 : sp));
  return p;
}

hipError_t launch_stats_pre(const SegPlan &pl, const float *z, const float *za, float *partials, hipStream_t s) {
  SegPlan p = pl;
  p.vec = al16(z) && al16(za);
  hipLaunchKernelGGL(k_stats_pre, dim3(p.nblocks()), dim3(kThreads), 0, s, p, PreOp{z, za}, partials);
  return hipGetLastError();
}

hipError_t launch_observe(const SegPlan &pl, const float *const *outs, const float *kappa, int m, const float *za,
                          float *zhat, float *partials, hipStream_t s) {
  if (m < 1 || m > WDC_MAXB) return hipErrorInvalidValue;
  ObsOp op;
  bool vec = al16(zhat) && al16(za);
  for (int j = 0; j < WDC_MAXB; ++j) {
    op.outs[j] = j < m ? outs[j] : nullptr;
    op.kappa[j] = j < m ? kappa[j] : 0.f;
    if (j < m) vec = vec && al16(outs[j]);
  }
  op.m = m;
  op.za = za;
  op.zhat = zhat;
  SegPlan p = pl;
  p.vec = vec;
  hipLaunchKernelGGL(k_observe, dim3(p.nblocks()), dim3(kThreads), 0, s, p, op, partials);
  return hipGetLastError();
}

hipError_t launch_exact_post(const SegPlan &pl, const PostArgs &a, float *partials, hipStream_t s) {
  SegPlan p = pl;
  p.vec = al16(a.z) && al16(a.v) && al16(a.zn_in) && al16(a.za) && al16(a.zhat) && al16(a.zn_out) &&
          al16(a.bank_slot) && al16(a.anchor_out) && al16(a.in_slot);
  hipLaunchKernelGGL(k_exact_post, dim3(p.nblocks()), dim3(kThreads), 0, s, p, PostOp{a}, partials);
  return hipGetLastError();
}

hipError_t launch_reduce_partials(const SegPlan &pl, const float *partials, int nv, double *out, hipStream_t s) {
  int total = pl.nseg() * nv;
  hipLaunchKernelGGL(k_reduce, dim3((total + 127) / 128), dim3(128), 0, s, partials, pl.nseg(), pl.splits, nv, out);
  return hipGetLastError();
}

hipError_t scratch_address(void **out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void *addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *out = addr[dev];
  return hipSuccess;
}

hipError_t launch_psi(const float *z, const float *v, float dt, float *zn, int64_t n, hipStream_t s) {
  const bool vec = al16(z) && al16(v) && al16(zn);
  const int w = vec ? 4 : 1;
  int64_t blocks = (n + 256 * w - 1) / (256 * w);
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  if (vec)
    hipLaunchKernelGGL(k_psi<4>, dim3((unsigned)blocks), dim3(256), 0, s, z, v, dt, zn, n);
  else
    hipLaunchKernelGGL(k_psi<1>, dim3((unsigned)blocks), dim3(256), 0, s, z, v, dt, zn, n);
  return hipGetLastError();
}

}  // namespace wdc

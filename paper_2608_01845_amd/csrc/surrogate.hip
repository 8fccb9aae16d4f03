// HBM-bound kernels of the surrogate and the risk controller (Sec. 4.2-4.3).
//
// The latent [C, F, H, W] is processed as C*8 contiguous segments: segment
// (c, g) holds the flat spatial indices j of channel c with floor(8j/T) = g,
// which is the finest chunking the 256-d summary pools over (coarser chunks
// nest: floor(4j/T) = floor(floor(8j/T)/2)). Each block streams one slice of
// one segment, so every per-chunk sum is a plain per-block sum and the grid
// needs no atomics; partial sums are then combined in a fixed order
// (deterministic, bit-reproducible run to run).
#include "common.h"

namespace wdc {

namespace {
constexpr int kThreads = 256;

struct SegRange {
  int64_t a, b;  // flat element range [a, b) of this block
  int seg;
};

__device__ __forceinline__ SegRange seg_range(int c_, int64_t t, int g, int splits) {
  const int blk = blockIdx.x;
  const int seg = blk / splits, sp = blk % splits;
  const int c = seg / g, gi = seg % g;
  const int64_t s0 = (gi * t + g - 1) / g;            // ceil(gi*T/G)
  const int64_t s1 = ((gi + 1) * t + g - 1) / g;      // ceil((gi+1)*T/G)
  const int64_t len = s1 - s0;
  SegRange r;
  r.a = (int64_t)c * t + s0 + (len * sp) / splits;
  r.b = (int64_t)c * t + s0 + (len * (sp + 1)) / splits;
  r.seg = seg;
  (void)c_;
  return r;
}

__global__ __launch_bounds__(kThreads) void k_stats_pre(SegPlan pl, const float *__restrict__ z,
                                                        const float *__restrict__ za, float *__restrict__ part) {
  __shared__ float lds[16 * PRE_NV];
  SegRange r = seg_range(pl.c, pl.t, pl.g, pl.splits);
  float v[PRE_NV] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int64_t i = r.a + threadIdx.x; i < r.b; i += kThreads) {
    float x = z[i];
    float a = za ? za[i] : 0.f;
    float d = x - a;
    v[0] += x;
    v[1] += d;
    v[2] += x * x;
    v[3] += d * d;
    v[4] += fabsf(d);
    v[5] += fabsf(a);
  }
  block_sum<PRE_NV>(v, lds);
  if (threadIdx.x == 0)
    for (int i = 0; i < PRE_NV; ++i) part[(int64_t)blockIdx.x * PRE_NV + i] = v[i];
}

struct ObsArgs {
  const float *outs[WDC_MAXB];
  float kappa[WDC_MAXB];
  int m;
};

__global__ __launch_bounds__(kThreads) void k_observe(SegPlan pl, ObsArgs oa, float *__restrict__ zhat,
                                                      float *__restrict__ part) {
  __shared__ float lds[16];
  SegRange r = seg_range(pl.c, pl.t, pl.g, pl.splits);
  float v[1] = {0.f};
  for (int64_t i = r.a + threadIdx.x; i < r.b; i += kThreads) {
    float acc = 0.f;
    for (int j = 0; j < oa.m; ++j) acc += oa.kappa[j] * oa.outs[j][i];
    zhat[i] = acc;
    v[0] += isfinite(acc) ? 0.f : 1.f;
  }
  block_sum<1>(v, lds);
  if (threadIdx.x == 0) part[blockIdx.x] = v[0];
}

__global__ __launch_bounds__(kThreads) void k_exact_post(SegPlan pl, PostArgs a, float *__restrict__ part) {
  __shared__ float lds[16 * POST_NV];
  SegRange r = seg_range(pl.c, pl.t, pl.g, pl.splits);
  float v[POST_NV] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int64_t i = r.a + threadIdx.x; i < r.b; i += kThreads) {
    float x = a.z[i];
    float xn;
    if (a.v) {
      xn = x + a.dt * a.v[i];
      a.zn_out[i] = xn;
    } else {
      xn = a.zn_in[i];
    }
    if (a.bank_slot) a.bank_slot[i] = xn;
    if (a.anchor_out) a.anchor_out[i] = x;
    float za = a.has_anchor ? a.za[i] : 0.f;
    float dn = xn - za, dx = xn - x;
    v[0] += xn;
    v[1] += dn;
    v[2] += dx;
    v[3] += xn * xn;
    v[4] += dn * dn;
    v[5] += dx * dx;
    if (a.has_zhat) v[6] += fabsf(xn - a.zhat[i]);
    v[7] += fabsf(xn);
  }
  block_sum<POST_NV>(v, lds);
  if (threadIdx.x == 0)
    for (int i = 0; i < POST_NV; ++i) part[(int64_t)blockIdx.x * POST_NV + i] = v[i];
}

__global__ void k_reduce(const float *__restrict__ part, int nseg, int splits, int nv, double *__restrict__ out) {
  int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= nseg * nv) return;
  int seg = idx / nv, v = idx % nv;
  double s = 0.0;
  for (int sp = 0; sp < splits; ++sp) s += (double)part[((int64_t)seg * splits + sp) * nv + v];
  out[idx] = s;
}

__global__ void k_psi(const float *__restrict__ z, const float *__restrict__ v, float dt, float *__restrict__ zn,
                      int64_t n) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) zn[i] = z[i] + dt * v[i];
}
}  // namespace

SegPlan make_seg_plan(int c, int64_t t, int g) {
  SegPlan p;
  p.c = c;
  p.t = t;
  p.g = g;
  int64_t seglen = (t + g - 1) / g;
  int64_t sp = (seglen + 2047) / 2048;
  p.splits = (int)(sp < 1 ? 1 : (sp > 64 ? 64 : sp));
  return p;
}

hipError_t launch_stats_pre(const SegPlan &pl, const float *z, const float *za, float *partials, hipStream_t s) {
  hipLaunchKernelGGL(k_stats_pre, dim3(pl.nblocks()), dim3(kThreads), 0, s, pl, z, za, partials);
  return hipGetLastError();
}

hipError_t launch_observe(const SegPlan &pl, const float *const *outs, const float *kappa, int m, float *zhat,
                          float *partials, hipStream_t s) {
  if (m < 1 || m > WDC_MAXB) return hipErrorInvalidValue;
  ObsArgs oa;
  for (int j = 0; j < WDC_MAXB; ++j) {
    oa.outs[j] = j < m ? outs[j] : nullptr;
    oa.kappa[j] = j < m ? kappa[j] : 0.f;
  }
  oa.m = m;
  hipLaunchKernelGGL(k_observe, dim3(pl.nblocks()), dim3(kThreads), 0, s, pl, oa, zhat, partials);
  return hipGetLastError();
}

hipError_t launch_exact_post(const SegPlan &pl, const PostArgs &a, float *partials, hipStream_t s) {
  hipLaunchKernelGGL(k_exact_post, dim3(pl.nblocks()), dim3(kThreads), 0, s, pl, a, partials);
  return hipGetLastError();
}

hipError_t launch_reduce_partials(const SegPlan &pl, const float *partials, int nv, double *out, hipStream_t s) {
  int total = pl.nseg() * nv;
  hipLaunchKernelGGL(k_reduce, dim3((total + 127) / 128), dim3(128), 0, s, partials, pl.nseg(), pl.splits, nv, out);
  return hipGetLastError();
}

hipError_t launch_psi(const float *z, const float *v, float dt, float *zn, int64_t n, hipStream_t s) {
  int64_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_psi, dim3((unsigned)blocks), dim3(256), 0, s, z, v, dt, zn, n);
  return hipGetLastError();
}

}  // namespace wdc

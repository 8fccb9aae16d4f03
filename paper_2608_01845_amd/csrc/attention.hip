// Attention of every denoiser block: O = softmax(Q K^T / sqrt(hd)) V over the
// full (non-causal) spatio-temporal + text sequence.
//
// bf16 path (flash attention on the matrix cores, hd = 64 or 128):
//  * 512-thread blocks of 256 queries, 32 per wavefront, two wavefronts per
//    SIMD; K tiles [64 keys][hd] and V^T tiles [hd][64 keys] reach LDS by
//    direct buffer loads, issued three or four tile steps ahead by four of the
//    waves;
//  * S^T = K Q^T with v_mfma_f32_32x32x16_bf16: the accumulator of a 32x32
//    tile gives lane l one query (l % 32) and 16 keys, so a query's row
//    statistics live in one lane and its partner l ^ 32 (one exchange);
//  * O^T = V^T P^T reuses the S^T accumulators directly as the B operand: the
//    8 accumulator values a lane holds for 16 consecutive keys become its 8
//    bf16 k-values, and the V^T operand is read with the same key order, so P
//    never goes through LDS;
//  * softmax in base 2 against a per-row reference max, each step running the
//    vector work of tile t + 1 inside the MFMA stream of tiles t and t + 2
//    (k_attn_bf16_ppr3);
//  * one head's padded q, k and v^T rows are addressed with 32-bit byte
//    offsets (buffer ranges, tile offsets): at most 2^30 B per head, which
//    the library checks before launching (attn_len_ok);
//  * the query blocks of the last, partly filled dispatch round can run as
//    several blocks over disjoint key ranges in the same launch, each leaving
//    its unnormalised rows, reference maxima and row sums in scratch for a
//    second launch that combines them in range order (attn_split_plan).
// float32 path: a plain online-softmax kernel (tiny fp32 workload).
#include "common.h"

#include <algorithm>
#include <numeric>

namespace wdc {

int64_t attn_pad(int64_t n) { return ((n + 255) / 256) * 256; }

namespace {

// ---------------------------------------------------------------- float32 reference-style kernel
// 16 queries per block, 16 threads per query, each thread owns hd/16 dims.
// Output offset of query q of head h: with several samples in one launch, head
// h is head h % hpb of sample h / hpb, whose rows start at sample * n.
__device__ __forceinline__ int64_t out_off(const AttnArgs &a, int h, int64_t q, int hd) {
  if (a.hpb > 0) {
    const int smp = h / a.hpb;
    return ((int64_t)smp * a.n + q) * a.ldo + (int64_t)(h - smp * a.hpb) * hd;
  }
  return q * a.ldo + (int64_t)h * hd;
}

template <int HD>
__global__ __launch_bounds__(256) void k_attn_f32(AttnArgs a) {
  constexpr int PER = HD / 16;
  constexpr int KT = 32;
  __shared__ float Ks[KT][HD + 1];
  __shared__ float Vs[KT][HD + 1];
  const int h = blockIdx.y;
  const int qi = threadIdx.x / 16, part = threadIdx.x % 16;
  const int64_t q = (int64_t)blockIdx.x * 16 + qi;
  const float *Q = (const float *)a.q + (int64_t)h * a.n_pad * HD;
  const float *K = (const float *)a.k + (int64_t)h * a.n_pad * HD;
  const float *V = (const float *)a.v + (int64_t)h * a.n_pad * HD;
  const float scale = rsqrtf((float)HD);
  float qv[PER], o[PER];
  const int64_t qq = q < a.n ? q : 0;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    qv[i] = Q[qq * HD + part * PER + i] * scale;
    o[i] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int64_t k0 = 0; k0 < a.n; k0 += KT) {
    for (int i = threadIdx.x; i < KT * HD; i += 256) {
      int r = i / HD, c = i % HD;
      int64_t kr = k0 + r;
      Ks[r][c] = kr < a.n ? K[kr * HD + c] : 0.f;
      Vs[r][c] = kr < a.n ? V[kr * HD + c] : 0.f;
    }
    __syncthreads();
    const int kn = (int)((a.n - k0) < KT ? (a.n - k0) : KT);
    for (int j = 0; j < kn; ++j) {
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < PER; ++i) s += qv[i] * Ks[j][part * PER + i];
#pragma unroll
      for (int o2 = 8; o2 > 0; o2 >>= 1) s += __shfl_xor(s, o2, 16);
      float mn = fmaxf(m, s);
      float al = expf(m - mn), p = expf(s - mn);
      l = l * al + p;
#pragma unroll
      for (int i = 0; i < PER; ++i) o[i] = o[i] * al + p * Vs[j][part * PER + i];
      m = mn;
    }
    __syncthreads();
  }
  if (q < a.n) {
    float *O = (float *)a.o + out_off(a, h, q, HD) + part * PER;
#pragma unroll
    for (int i = 0; i < PER; ++i) O[i] = o[i] / l;
  }
}

// ---------------------------------------------------------------- bf16 flash attention on MFMA
constexpr int KV = 64;                   // keys per LDS tile
constexpr int RSRC_WORD3 = 0x00020000;   // raw buffer descriptor word 3
constexpr int WAIT_VM0 = 0x0F70;         // s_waitcnt vmcnt(0), other counters untouched

// LDS swizzles: 16 consecutive lanes read 16 different rows at one logical
// chunk; the XOR spreads them over distinct bank groups of the 64 x 4-byte banks.
// K tile: rows of HD bf16 = HD/8 16-byte chunks. hd = 128 (256-byte rows):
// chunk c of row r at c ^ (r & 15); hd = 64 (128-byte rows, two per bank span):
// c ^ ((r >> 1) & 7).
template <int HD>
__device__ __forceinline__ int kswz(int r, int c) {
  return HD == 128 ? (r * 16 + (c ^ (r & 15))) * 16 : (r * 8 + (c ^ ((r >> 1) & 7))) * 16;
}
// V^T tile: rows of 64 keys (128 B) = 8 16-byte slots. Within 16-key group j,
// slot 2j holds keys 16j+[0,4) and 16j+8+[0,4), slot 2j+1 keys 16j+4+[0,4) and
// 16j+12+[0,4): exactly the 8 keys lane group 0 / 1 feeds to one 32x32x16 step
// of O^T = V^T P^T (the key order of the S^T accumulator), so each A operand is
// one 16-byte read. Slot p of row r lives at p ^ ((r >> 1) & 7).
__device__ __forceinline__ int vslot(int r, int p) { return (r * 8 + (p ^ ((r >> 1) & 7))) * 16; }

// Direct global -> LDS tile loads (buffer_load_dwordx4 ... lds): lane L of a
// wavefront's load writes its 16 bytes at LDS base + 16 L, so the swizzles above
// are applied by choosing which global chunk each lane fetches. Wave w of 4
// fills 1 KB stripes w, w+4, w+8, ... of each tile:
//   K tile:   stripe holds rows [r0, r0 + 1024/(2 HD)) of 2 HD bytes;
//   V^T tile: stripe holds 8 rows of 128 bytes (the global V^T rows are stored
//             with the slot key order already applied, see k_v_transpose).
// Stripe i of wave w starts at LDS byte w*1024 + i*4096 in both tiles; the row
// swizzle keys are the same for every stripe of a wave, so one VGPR offset per
// tile kind plus a uniform SGPR offset per stripe addresses the global side.
typedef __attribute__((address_space(3))) void lds_void;
// (kept out of line of the kernel templates: called directly from a template
// kernel body the builtin makes the host pass drop the kernel's launch stub)
__device__ __forceinline__ void lds_load16(__amdgpu_buffer_rsrc_t r, char *lds, int voff, int soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void *)lds, 16, voff, soff, 0, 0);
}
template <int HD>
struct TileLoad {
  static constexpr int K_ROWS = 1024 / (2 * HD);   // K rows per 1 KB stripe (4 or 8)
  static constexpr int K_STRIPES = 16 / K_ROWS;    // stripes per wave per K tile (4 or 2)
  static constexpr int V_STRIPES = HD / 32;        // stripes per wave per V^T tile (4 or 2)
  int kvo, vvo;                                    // per-lane global byte offsets (stripe 0, tile 0)
  __device__ __forceinline__ TileLoad(int w, int lane, int64_t n_pad) {
    const int kr0 = w * K_ROWS + lane / (HD / 8), kps = lane % (HD / 8);
    const int kc = HD == 128 ? (kps ^ (kr0 & 15)) : (kps ^ ((kr0 >> 1) & 7));
    kvo = kr0 * HD * 2 + kc * 16;
    const int vr0 = 8 * w + lane / 8, vps = lane % 8;
    vvo = vr0 * (int)n_pad * 2 + (vps ^ ((vr0 >> 1) & 7)) * 16;
  }
};

template <int HD>
__device__ __forceinline__ void pp_wait4(int n_outstanding) {
  constexpr int KS = TileLoad<HD>::K_STRIPES, VS = TileLoad<HD>::V_STRIPES;
  static_assert(KS + VS < 16, "vmcnt immediate");
  if (n_outstanding == KS + VS)
    __builtin_amdgcn_s_waitcnt(WAIT_VM0 | (KS + VS));
  else if (n_outstanding == VS)
    __builtin_amdgcn_s_waitcnt(WAIT_VM0 | VS);
  else
    __builtin_amdgcn_s_waitcnt(WAIT_VM0);
}

// Vector phase: Q is scaled by sc = log2(e)/sqrt(HD) once, and -m is the
// accumulator input of the first Q K MFMA of each 32-key half (a lane holds one
// query, so the tile is -m in all 16 values), so the matrix phase hands over
// S' = sc Q K^T - m and the vector phase is P = exp2(S'), its bf16 conversion
// and the row sum of those bf16 values (the weights the PV product uses). m is
// a reference, not a running max: the first tile's row max, moved to a row's
// true max only when a lane's P sum over a tile exceeds 2^64 (then O and l are
// rescaled and P recomputed). Any reference gives the same normalised result,
// and P <= 2^64 keeps O and l far from float overflow.
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;
constexpr float PPR_LIMIT = 0x1p64f;

// accumulator tile that starts a row's Q K contraction at -m
__device__ __forceinline__ f32x16 ppr_mtile(float m) {
  f32x16 t;
#pragma unroll
  for (int e = 0; e < 16; ++e) t[e] = -m;
  return t;
}

template <int HD>
__device__ __forceinline__ void ppr_qk(f32x16 (&S)[2], const char *k, const bf16x8 (&qf)[HD / 16],
                                       const int (&kro)[HD / 16], const f32x16 &mi) {
#pragma unroll
  for (int st_ = 0; st_ < HD / 16; ++st_)
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const bf16x8 kf = *(const bf16x8 *)(k + kro[st_] + kt * 32 * HD * 2);
      S[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[st_], st_ == 0 ? mi : S[kt], 0, 0, 0);
    }
}

// row max over the tile's 64 keys (32 per lane, the rest in lane l ^ 32)
__device__ __forceinline__ float ppr_rowmax(const f32x16 (&S)[2]) {
  float mx = fmaxf(S[0][0], S[1][0]);
#pragma unroll
  for (int e = 1; e < 16; ++e) mx = fmaxf(mx, fmaxf(S[0][e], S[1][e]));
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float ppr_exp(const f32x16 (&S)[2], bf16x8 (&pf)[4]) {
  const bf16x2_t one2 = {(__bf16)1.f, (__bf16)1.f};
  float ls = 0.f;
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int e = 0; e < 16; ++e) pf[2 * kt + e / 8][e % 8] = (__bf16)__builtin_amdgcn_exp2f(S[kt][e]);
#pragma unroll
  for (int q = 0; q < 16; ++q)
    ls = __builtin_amdgcn_fdot2_f32_bf16(bf16x2_t{pf[q / 4][2 * (q % 4)], pf[q / 4][2 * (q % 4) + 1]}, one2, ls,
                                         false);
  return ls;
}

// End of a key-range block (block j of the split round: head h, query block
// qb_main + qt, range sp, in that nesting): its unnormalised rows O (float32),
// reference maxima m and row sums l go to slot (j * 256 + query) of the
// scratch: O at part + slot * HD, (m, l) at part + slots * HD + 2 slot.
template <int HD>
__device__ __forceinline__ void attn_split_store(const AttnArgs &a, const f32x16 (&o)[HD / 32], float m, float lt,
                                                 int j) {
  const int lane = threadIdx.x & 63, lr = lane & 31, lg = lane >> 5, wid = threadIdx.x >> 6;
  const int tail = (int)(a.n_pad / 256) - a.qb_main;
  const int64_t slots = (int64_t)a.heads * tail * a.kv_splits * 256;
  const int64_t slot = (int64_t)j * 256 + wid * 32 + lr;
  float *po = a.part + slot * HD;
#pragma unroll
  for (int i = 0; i < HD / 32; ++i)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4)
      *(float4 *)(po + 32 * i + 8 * g4 + 4 * lg) =
          make_float4(o[i][4 * g4], o[i][4 * g4 + 1], o[i][4 * g4 + 2], o[i][4 * g4 + 3]);
  if (lg == 0) *(float2 *)(a.part + slots * HD + 2 * slot) = make_float2(m, lt);
}

// Combine of the split round, after the attention launch: for each of its
// queries (thread: one query, eight columns) the key ranges in range order,
//   O = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s,  M = max_s m_s
// (m in log2 units), rounded to bf16 once.
template <int HD>
__global__ __launch_bounds__(256) void k_attn_combine(AttnArgs a) {
  constexpr int C8 = HD / 8;
  const int ns = a.kv_splits, tail = (int)(a.n_pad / 256) - a.qb_main;
  const int64_t slots = (int64_t)a.heads * tail * ns * 256;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (gid >= (int64_t)a.heads * tail * 256 * C8) return;
  const int c8 = (int)(gid % C8);
  const int64_t qt = gid / C8;                   // (head, tail query block, query)
  const int qi = (int)(qt % 256);
  const int64_t hb = qt / 256;                   // head * tail + tail query block
  const int h = (int)(hb / tail), qb = a.qb_main + (int)(hb % tail);
  const int64_t q = (int64_t)qb * 256 + qi;
  if (q >= a.n) return;
  const int64_t s0 = hb * ns * 256 + qi;         // slot of range 0; range r at s0 + 256 r
  const float *pml = a.part + slots * HD;
  float mx = -INFINITY;
  for (int r = 0; r < ns; ++r) mx = fmaxf(mx, pml[2 * (s0 + 256 * r)]);
  float den = 0.f, acc[8] = {};
  for (int r = 0; r < ns; ++r) {
    const int64_t sl = s0 + 256 * r;
    const float w = __builtin_amdgcn_exp2f(pml[2 * sl] - mx);
    den += w * pml[2 * sl + 1];
    const float4 v0 = *(const float4 *)(a.part + sl * HD + 8 * c8);
    const float4 v1 = *(const float4 *)(a.part + sl * HD + 8 * c8 + 4);
    acc[0] += w * v0.x;
    acc[1] += w * v0.y;
    acc[2] += w * v0.z;
    acc[3] += w * v0.w;
    acc[4] += w * v1.x;
    acc[5] += w * v1.y;
    acc[6] += w * v1.z;
    acc[7] += w * v1.w;
  }
  const float inv = 1.f / den;
  bf16_t *O = (bf16_t *)a.o + out_off(a, h, q, HD) + 8 * c8;
  *(uint2 *)O = make_uint2((uint32_t)f2bf(acc[0] * inv) | ((uint32_t)f2bf(acc[1] * inv) << 16),
                           (uint32_t)f2bf(acc[2] * inv) | ((uint32_t)f2bf(acc[3] * inv) << 16));
  *(uint2 *)(O + 4) = make_uint2((uint32_t)f2bf(acc[4] * inv) | ((uint32_t)f2bf(acc[5] * inv) << 16),
                                 (uint32_t)f2bf(acc[6] * inv) | ((uint32_t)f2bf(acc[7] * inv) << 16));
}

// bf16 flash attention. 8 wavefronts per block (two per SIMD), 32 queries each
// (256 per block); K tiles of 64 keys and V^T tiles reach four K and four V^T
// LDS slots by direct buffer loads issued by waves 0-3; one block barrier per
// tile step. Step t runs the P V MFMAs of
// tile t and the Q K MFMAs of tile t + 2 with the vector phase of tile t + 1
// (P = exp2(S'), its bf16 conversion and row sum) interleaved into the same
// instruction stream, so a wave's VALU work executes under its own MFMAs
// instead of in a separate phase that the two waves of a SIMD run together.
// S and P are double-buffered (S of t + 1 and t + 2, P of t and t + 1). Tile j
// sits in slot j % 4: step t reads K_{t+2} and V_t, loads K_{t+4} into the
// slot of K_t (last read in step t - 2, or by the prologue for t = 0, hence
// one more barrier there) and V_{t+3} into the slot of V_{t-1} (last read in
// step t - 1, and waited for before the barrier that ends it); the first four
// reads of V_{t+1} go out at the end of step t.
template <int HD>
__global__ __launch_bounds__(512, 1) void k_attn_bf16_ppr3(AttnArgs a) {
  constexpr int QB = 256;                  // 8 waves x 32 queries
  constexpr int NB = 4;                    // K buffers and V^T buffers
  constexpr int K_BYTES = KV * HD * 2;
  constexpr int V_BASE = NB * K_BYTES;     // V^T buffers follow the K buffers
  using TL = TileLoad<HD>;
  extern __shared__ __attribute__((aligned(16))) char smem[];

  // Block b < heads x qb_main: query block qb < qb_main of head h over all
  // keys (with the XCD order, each XCD runs whole heads: blocks go to the XCDs
  // round robin); the rest: query block qb >= qb_main of head h, key range sp
  // of kv_splits, in (head, query block, range) order.
  const int ns = a.kv_splits > 1 ? a.kv_splits : 1;
  const int nqb = (int)(a.n_pad / QB), tail = nqb - a.qb_main;
  const int bid = blockIdx.x, main_blocks = a.heads * a.qb_main;
  int h, qb, sp = 0, nr = 1;                  // key range sp of nr
  if (bid < main_blocks) {
    if (a.xcd_order) {
      const int li = bid >> 3;
      h = (bid & 7) + 8 * (li / a.qb_main);
      qb = li % a.qb_main;
    } else {
      h = bid / a.qb_main;
      qb = bid % a.qb_main;
    }
  } else {
    const int j = bid - main_blocks;
    h = j / (tail * ns);
    qb = a.qb_main + (j % (tail * ns)) / ns;
    sp = j % ns;
    nr = ns;
  }

  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool grp_a = wid < 4;
  const int lr = lane & 31, lg = lane >> 5;
  const int64_t qbase = (int64_t)qb * QB + wid * 32;
  const bf16_t *Q = (const bf16_t *)a.q + (int64_t)h * a.n_pad * HD;

  const float sc = 1.4426950408889634f * rsqrtf((float)HD);
  bf16x8 qf[HD / 16];                      // Q^T scaled by sc: scores in log2 units
#pragma unroll
  for (int s = 0; s < HD / 16; ++s) {
    const bf16x8 raw = *(const bf16x8 *)(Q + (qbase + lr) * HD + 16 * s + 8 * lg);
#pragma unroll
    for (int j = 0; j < 8; ++j) qf[s][j] = (__bf16)((float)raw[j] * sc);
  }

  // key tiles [t_first, t_first + ntiles) of tiles_all (all of them outside
  // the split round); only the range that ends the sequence holds the partial
  // last tile. The K and V^T buffer ranges start at the range's first key, so
  // the tile loads address tiles relative to the range.
  const int tiles_all = (int)((a.n + KV - 1) / KV);
  const int t_first = (int)((int64_t)sp * tiles_all / nr);
  const int t_end = (int)((int64_t)(sp + 1) * tiles_all / nr);
  const int ntiles = t_end - t_first;
  const int last_valid = t_end == tiles_all ? (int)(a.n - (int64_t)(tiles_all - 1) * KV) : KV;
  const int64_t key0 = (int64_t)t_first * KV;
  const __amdgpu_buffer_rsrc_t kdesc = __builtin_amdgcn_make_buffer_rsrc(
      (void *)((const bf16_t *)a.k + ((int64_t)h * a.n_pad + key0) * HD), (short)0,
      (int)((a.n_pad - key0) * HD * 2), RSRC_WORD3);
  const __amdgpu_buffer_rsrc_t vdesc = __builtin_amdgcn_make_buffer_rsrc(
      (void *)((const bf16_t *)a.v + (int64_t)h * HD * a.n_pad + key0), (short)0,
      (int)((a.n_pad * HD - key0) * 2), RSRC_WORD3);
  const int lw = wid & 3;
  const TileLoad<HD> tl(lw, lane, a.n_pad);
  int kro[HD / 16];
#pragma unroll
  for (int s = 0; s < HD / 16; ++s) kro[s] = kswz<HD>(lr, 2 * s + lg);
  int vro[4];                              // V^T fragment offsets, V region base folded in
#pragma unroll
  for (int j = 0; j < 4; ++j) vro[j] = V_BASE + vslot(lr, 2 * j + lg);

  auto load_k = [&](int b, int tile) {
#pragma unroll
    for (int i = 0; i < TL::K_STRIPES; ++i)
      lds_load16(kdesc, smem + b * K_BYTES + lw * 1024 + i * 4096, tl.kvo, tile * KV * HD * 2 + i * 4096);
  };
  auto load_v = [&](int b, int tile) {
#pragma unroll
    for (int i = 0; i < TL::V_STRIPES; ++i)
      lds_load16(vdesc, smem + V_BASE + b * K_BYTES + lw * 1024 + i * 4096, tl.vvo,
                 tile * KV * 2 + i * 32 * (int)a.n_pad * 2);
  };

  if (grp_a) {                             // K_0..K_3, V_0..V_2
#pragma unroll
    for (int j = 0; j < NB; ++j)
      if (j < ntiles) load_k(j, j);
    load_v(0, 0);
    if (ntiles > 1) load_v(1, 1);
    if (ntiles > 2) load_v(2, 2);
    __builtin_amdgcn_s_waitcnt(WAIT_VM0);
  }
  __syncthreads();

  f32x16 o[HD / 32];
#pragma unroll
  for (int i = 0; i < HD / 32; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[i][e] = 0.f;
  float m = 0.f, l = 0.f;
  f32x16 mi = ppr_mtile(m);
  f32x16 S[2][2];                          // S' of tiles t + 1 and t + 2 (index tile & 1)
  bf16x8 pf[2][4];                         // P of tiles t and t + 1 (index tile & 1)
  ppr_qk<HD>(S[0], smem, qf, kro, mi);
  {                                        // m = the first tile's row max
    const int v0 = ntiles == 1 ? last_valid : KV;
    if (v0 < KV) {
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (32 * kt + 8 * (e / 4) + 4 * lg + (e % 4) >= v0) S[0][kt][e] = -1e30f;
    }
    m = ppr_rowmax(S[0]);
    mi = ppr_mtile(m);
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) S[0][kt][e] -= m;
    l = ppr_exp(S[0], pf[0]);
  }
  if (ntiles > 1) ppr_qk<HD>(S[1], smem + K_BYTES, qf, kro, mi);
  // step 0 refills the slot of K_0, which every wave has just read
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");

  constexpr int NMF = 4 * (HD / 32) + 2 * (HD / 16);   // fragment reads per step
  static_assert(NMF == 16 || NMF == 32, "hd 64 or 128");
  constexpr int NPV = NMF / 2;             // P V reads (and MFMAs) per step; as many Q K
  constexpr int EPM = 32 / NMF;            // exponentials after each MFMA (32 per step)
  // V^T tiles are loaded three steps ahead, so the tile of step t + 1 is
  // published by the barrier that ends step t - 1 and step t issues its first
  // four fragment reads after its own MFMA stream: the next step's first MFMA
  // finds its operand in registers instead of waiting on LDS after the barrier.
  const bf16x2_t one2_ = {(__bf16)1.f, (__bf16)1.f};
  // fragment read r of a step from V^T slot vb and K slot kb: r < NPV V^T (k-step
  // r / (HD/32), O tile r % (HD/32)), then K (hd step (r-NPV) / 2, key half (r-NPV) % 2)
#define WDC_PPR3_READ(r, vb, kb)                                                                 \
  {                                                                                              \
    if ((r) < NPV)                                                                               \
      fr_[(r)] = *(const bf16x8 *)((vb) + ((r) % (HD / 32)) * 32 * KV * 2 + vro[(r) / (HD / 32)]);\
    else                                                                                         \
      fr_[(r)] = *(const bf16x8 *)((kb) + kro[((r) >= NPV ? (r) - NPV : 0) / 2] +                \
                                   (((r) >= NPV ? (r) - NPV : 0) % 2) * 32 * HD * 2);            \
  }
  bf16x8 fr_[NMF];
#pragma unroll
  for (int r_ = 0; r_ < 4; ++r_) WDC_PPR3_READ(r_, smem, smem);   // step 0's first reads (V^T of tile 0)
  // One tile step with compile-time slot P = t % NB; c = (t + 1) & 1 indexes
  // S' of tile t + 1 and the P it becomes, n = t & 1 the S' of tile t + 2 and
  // the P of tile t.
#define WDC_PPR3_STEP(P)                                                                         \
  {                                                                                              \
    constexpr int c = ((P) + 1) & 1, n = (P) & 1;                                                \
    const int t = t0 + (P);                                                                      \
    int issued = 0;                                                                              \
    if (grp_a) {                                                                                 \
      if (t + 4 < ntiles) {                                                                      \
        load_k((P), t + 4);                                                                      \
        issued += TL::K_STRIPES;                                                                 \
      }                                                                                          \
      if (t + 3 < ntiles) {                                                                      \
        load_v(((P) + 3) % NB, t + 3);                                                           \
        issued += TL::V_STRIPES;                                                                 \
      }                                                                                          \
    }                                                                                            \
    const bool soft = t + 1 < ntiles;                                                            \
    if (t + 2 == ntiles && last_valid < KV) {  /* tile t + 1 is the partial last one */          \
      asm volatile("" ::: "memory");                                                             \
      _Pragma("unroll") for (int kt = 0; kt < 2; ++kt)                                           \
      _Pragma("unroll") for (int e = 0; e < 16; ++e)                                             \
        if (32 * kt + 8 * (e / 4) + 4 * lg + (e % 4) >= last_valid) S[c][kt][e] = -1e30f;        \
    }                                                                                            \
    __builtin_amdgcn_sched_barrier(0);                                                           \
    /* One fixed-order stream (unconditional: past the end the Q K reads a stale */              \
    /* K slot and the exponentials a stale S', and neither result is used). MFMA */              \
    /* q: 0-15 P V (k-step j = q / (HD/32), O tile i = q % (HD/32)), 16-31 Q K (hd */            \
    /* step (q-16) / 2, key half q % 2; hd step 0 starts from the -m tile); */                   \
    /* fragment read q goes out four reads ahead of its MFMA (reads 0-3 in the */                \
    /* previous step); after MFMA q comes exponential q of S'_{t+1}, after every */              \
    /* second one the bf16 pair and its row-sum dot product. */                                  \
    const char *vb_ = smem + (P) * K_BYTES, *kb_ = smem + (((P) + 2) % NB) * K_BYTES;            \
    const char *vn_ = smem + (((P) + 1) % NB) * K_BYTES;   /* V^T slot of tile t + 1 */          \
    float ls = 0.f;                                                                              \
    _Pragma("unroll") for (int q_ = 0; q_ < NMF; ++q_) {                                         \
      if (q_ < NPV) {                                                                            \
        constexpr int NI = HD / 32;                                                              \
        o[q_ % NI] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr_[q_], pf[n][q_ / NI], o[q_ % NI], 0, 0, 0);\
      } else {                                                                                   \
        const int g_ = q_ >= NPV ? q_ - NPV : 0;                                                 \
        S[n][g_ % 2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr_[q_], qf[g_ / 2],              \
                                                               g_ < 2 ? mi : S[n][g_ % 2], 0, 0, 0);\
      }                                                                                          \
      __builtin_amdgcn_sched_barrier(0);                                                         \
      if (q_ + 4 < NMF)                                                                          \
        WDC_PPR3_READ(q_ + 4, vb_, kb_)                                                          \
      else  /* the next step's first reads: V^T of tile t + 1, published by the last barrier */  \
        WDC_PPR3_READ(q_ + 4 - NMF, vn_, kb_)                                                    \
      /* hd 64: the read goes out before the pair (0.8% faster than after it) */                 \
      if constexpr (EPM == 2) __builtin_amdgcn_sched_barrier(0);                                  \
      if constexpr (EPM == 2) {                                                                  \
        /* both exponentials of a pair, converted together; the empty asm pins */                \
        /* the pair under this MFMA (left free, the compiler sinks all of them */                \
        /* past the stream, where they no longer overlap the matrix cores) */                    \
        const int ei_ = 2 * q_, kt_ = ei_ / 16, e_ = ei_ % 16;                                   \
        const bf16x2_t pr_ = {(__bf16)__builtin_amdgcn_exp2f(S[c][kt_][e_]),                     \
                              (__bf16)__builtin_amdgcn_exp2f(S[c][kt_][e_ + 1])};                \
        uint32_t u_ = __builtin_bit_cast(uint32_t, pr_);                                         \
        asm volatile("" : "+v"(u_));                                                             \
        u32x4_t w_ = __builtin_bit_cast(u32x4_t, pf[c][2 * kt_ + e_ / 8]);                        \
        w_[(e_ % 8) / 2] = u_;                                                                   \
        pf[c][2 * kt_ + e_ / 8] = __builtin_bit_cast(bf16x8, w_);                                \
        ls = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, u_), one2_, ls, false); \
      } else {                                                                                   \
        _Pragma("unroll") for (int x_ = 0; x_ < EPM; ++x_) {                                     \
          const int ei_ = q_ * EPM + x_, kt_ = ei_ / 16, e_ = ei_ % 16;                          \
          pf[c][2 * kt_ + e_ / 8][e_ % 8] = (__bf16)__builtin_amdgcn_exp2f(S[c][kt_][e_]);       \
          if (ei_ & 1)                                                                           \
            ls = __builtin_amdgcn_fdot2_f32_bf16(                                                \
                bf16x2_t{pf[c][2 * kt_ + e_ / 8][(e_ - 1) % 8], pf[c][2 * kt_ + e_ / 8][e_ % 8]}, one2_, ls, false);\
        }                                                                                        \
      }                                                                                          \
      __builtin_amdgcn_sched_barrier(0);                                                         \
    }                                                                                            \
    __builtin_amdgcn_sched_barrier(0);                                                           \
    if (soft) {                                                                                  \
      if (__any(ls > PPR_LIMIT)) {                                                               \
        const float mx = ppr_rowmax(S[c]);                                                       \
        const float mn = m + (mx > 8.f ? mx : 0.f);                                              \
        mi = ppr_mtile(mn);                                                                      \
        const float d = mn - m, alpha = __builtin_amdgcn_exp2f(-d);                              \
        m = mn;                                                                                  \
        l *= alpha;                                                                              \
        _Pragma("unroll") for (int i = 0; i < HD / 32; ++i)                                      \
        _Pragma("unroll") for (int e = 0; e < 16; ++e) o[i][e] *= alpha;                         \
        _Pragma("unroll") for (int kt = 0; kt < 2; ++kt)                                         \
        _Pragma("unroll") for (int e = 0; e < 16; ++e) {                                         \
          S[c][kt][e] -= d;                                                                      \
          S[n][kt][e] -= d;                                                                      \
        }                                                                                        \
        ls = ppr_exp(S[c], pf[c]);                                                               \
      }                                                                                          \
      l += ls;                                                                                   \
    }                                                                                            \
    if (grp_a) pp_wait4<HD>(issued);                                                             \
    /* every older read is done; the four just issued read a slot no load of */                  \
    /* the next step writes */                                                                   \
    asm volatile("s_waitcnt lgkmcnt(4)\n\ts_barrier" ::: "memory");                              \
  }
  for (int t0 = 0; t0 < ntiles; t0 += NB) {
    WDC_PPR3_STEP(0)
    if (t0 + 1 >= ntiles) break;
    WDC_PPR3_STEP(1)
    if (t0 + 2 >= ntiles) break;
    WDC_PPR3_STEP(2)
    if (t0 + 3 >= ntiles) break;
    WDC_PPR3_STEP(3)
  }
#undef WDC_PPR3_STEP
#undef WDC_PPR3_READ

  const float lt = l + __shfl_xor(l, 32, 64);
  if (bid >= main_blocks && ns > 1) {
    attn_split_store<HD>(a, o, m, lt, bid - main_blocks);
    return;
  }
  const float inv = 1.f / lt;
  const int64_t q = qbase + lr;
  if (q < a.n) {
    bf16_t *O = (bf16_t *)a.o + out_off(a, h, q, HD);
#pragma unroll
    for (int i = 0; i < HD / 32; ++i)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int d0 = 32 * i + 8 * g4 + 4 * lg;
        uint32_t w0 = (uint32_t)f2bf(o[i][4 * g4 + 0] * inv) | ((uint32_t)f2bf(o[i][4 * g4 + 1] * inv) << 16);
        uint32_t w1 = (uint32_t)f2bf(o[i][4 * g4 + 2] * inv) | ((uint32_t)f2bf(o[i][4 * g4 + 3] * inv) << 16);
        *(uint2 *)(O + d0) = make_uint2(w0, w1);
      }
  }
}

template <int HD>
hipError_t launch_bf16_ppr3(const AttnArgs &a, hipStream_t s) {
  constexpr int LDS = 2 * 4 * KV * HD * 2;     // four K tiles, four V^T tiles
  static bool seen[64] = {};
  if (first_on_device(seen)) {
    const hipError_t e = hipFuncSetAttribute((const void *)k_attn_bf16_ppr3<HD>, hipFuncAttributeMaxDynamicSharedMemorySize, LDS);
    if (e != hipSuccess) return e;
  }
  AttnArgs b = a;
  attn_split_plan(b);
  const int nqb = (int)(b.n_pad / 256);
  const int64_t blocks = (int64_t)b.heads * b.qb_main + (int64_t)b.heads * (nqb - b.qb_main) * b.kv_splits;
  hipLaunchKernelGGL((k_attn_bf16_ppr3<HD>), dim3((unsigned)blocks), dim3(512), LDS, s, b);
  if (b.kv_splits > 1) {
    const int64_t items = (int64_t)b.heads * (nqb - b.qb_main) * 256 * (HD / 8);
    hipLaunchKernelGGL((k_attn_combine<HD>), dim3((unsigned)((items + 255) / 256)), dim3(256), 0, s, b);
  }
  return hipGetLastError();
}

}  // namespace

// Key-range split of the last dispatch round. Query blocks [0, qb_main) of
// every head fill whole rounds (heads x qb_main a multiple of the compute
// units); the other heads x (nqb - qb_main) blocks would leave CUs idle in a
// partial round, so each runs as s blocks over s disjoint key ranges when the
// estimate says so: ceil(tail s / CUs) / s rounds of a block's time, against
// ceil(tail / CUs), plus the scratch traffic (written once, read once). A
// block's time is taken at about half the bf16 peak of one CU; at least 8
// key tiles per range.
void attn_split_plan(AttnArgs &b) {
  const int nqb = (int)(b.n_pad / 256);
  b.qb_main = nqb;
  b.kv_splits = 1;
  const int cus = device_cus();
  if (!b.part || b.force_splits == 1 || cus <= 0) return;
  const int g = cus / std::gcd(cus, b.heads);    // heads x g blocks fill whole rounds
  const int qb_main = nqb / g * g, tail = nqb - qb_main;
  const int64_t tb = (int64_t)b.heads * tail;
  if (tail == 0) return;
  const int tiles = (int)((b.n + 63) / 64);
  auto bytes = [&](int s) { return (size_t)(tb * s * 256) * (size_t)(b.hd + 2) * sizeof(float); };
  int best_s = 1;
  if (b.force_splits >= 2) {
    best_s = std::min(b.force_splits, tiles);
    if (bytes(best_s) > b.part_bytes) return;
  } else {
    const double t_blk = 1024.0 * (double)b.n * b.hd / 4.9e12;
    const double base = (double)((tb + cus - 1) / cus) * t_blk;
    double best = base;
    for (int s = 2; s <= 8 && tiles >= 8 * s && bytes(s) <= b.part_bytes; ++s) {
      const double t = (double)((tb * s + cus - 1) / cus) / s * t_blk + 2.0 * (double)bytes(s) / 4e12;
      if (t < best) {
        best = t;
        best_s = s;
      }
    }
    if (best >= 0.9 * base) best_s = 1;
  }
  if (best_s < 2) return;
  b.qb_main = qb_main;
  b.kv_splits = best_s;
}

hipError_t launch_attention(int dtype, const AttnArgs &a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  if (a.n_pad != attn_pad(a.n)) return hipErrorInvalidValue;
  if (dtype == 1) {
    // heads grouped per XCD when the head count allows it (every real workload)
    AttnArgs b = a;
    b.xcd_order = a.heads % 8 == 0 ? 1 : 0;
    if (a.hd == 128) return launch_bf16_ppr3<128>(b, s);
    if (a.hd == 64) return launch_bf16_ppr3<64>(b, s);
    return hipErrorInvalidValue;
  }
  dim3 grid((unsigned)((a.n + 15) / 16), (unsigned)a.heads);
  if (a.hd == 64)
    hipLaunchKernelGGL(k_attn_f32<64>, grid, dim3(256), 0, s, a);
  else if (a.hd == 128)
    hipLaunchKernelGGL(k_attn_f32<128>, grid, dim3(256), 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace wdc

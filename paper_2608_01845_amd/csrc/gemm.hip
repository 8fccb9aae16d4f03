// GEMMs of the denoiser: c[m, n] = sum_k a[m, k] * w[n, k] + bias[n] with a
// fused epilogue (store, GELU-tanh, gated residual into the float32 stream,
// float32 store). Both operands are K-contiguous ("NT"), which is the layout
// the MFMA operand registers want: every lane loads 8 consecutive bf16.
//
// bf16 path: v_mfma_f32_32x32x16_bf16 tiles, BMxBN block tile (256 x 256 in 8
// waves of 128 x 64 for the large products), BK = 64, double-buffered LDS with
// an XOR swizzle of the 16-byte chunks of each 128-byte row (conflict-free
// fragment reads). K stages go straight from HBM into LDS (buffer loads with the
// LDS flag) two stages ahead; each wave reads its fragments one k-step ahead,
// one read at a time between its MFMAs, and the stage barrier sits before a
// stage's last k-step so the matrix cores never drain at it. Large single
// products take an XCD-aware block order, and long-K ones whose last dispatch
// round would be thin run their last rows as a second launch of 128 x 128 tiles;
// products too small to fill one dispatch round of 256 x 256 tiles run on
// 128 x 128 tiles throughout (128 x 64 when even those would not fill it).
// float32 path (tiny fp32 workload, and shapes the MFMA tiles do not cover):
// a plain LDS-tiled FMA kernel.
#include "common.h"

namespace wdc {

// compute units of the current device (the rectangle order needs exactly 256)
int device_cus() {
  static int cus[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (!cus[dev] && hipDeviceGetAttribute(&cus[dev], hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    cus[dev] = 0;
  return cus[dev];
}

namespace {

template <typename T>
__device__ __forceinline__ void epilogue(const GemmArgs &g, int epi, int64_t row, int64_t col, float acc) {
  float v = acc + (g.bias ? ld<T>((const T *)g.bias + col) : 0.f);
  int64_t o = row * g.ldc + col;
  switch (epi) {
    case EPI_STORE: st<T>((T *)g.c + o, v); break;
    case EPI_GELU: st<T>((T *)g.c + o, gelu_tanh(v)); break;
    case EPI_GATE_RES:
    case EPI_GATE_RES_NT: ((float *)g.c)[o] += g.gate[col] * v; break;
    default: ((float *)g.c)[o] = v; break;
  }
}

// ---------------------------------------------------------------- generic tiled kernel
// Batch entry blockIdx.z of a batched product: shifted operand and output pointers.
template <typename T>
__device__ __forceinline__ GemmArgs batch_entry(const GemmArgs &g0) {
  GemmArgs g = g0;
  const int64_t z = blockIdx.z;
  if (z) {
    const bool c16 = (g0.epi == EPI_STORE || g0.epi == EPI_GELU) && sizeof(T) == 2;
    g.a = (const T *)g0.a + z * g0.a_bs;
    g.c = c16 ? (void *)((T *)g0.c + z * g0.c_bs) : (void *)((float *)g0.c + z * g0.c_bs);
    if (g0.gate) g.gate = g0.gate + z * g0.gate_bs;
  }
  return g;
}

template <typename T>
__global__ __launch_bounds__(256) void k_gemm_simple(GemmArgs g0) {
  const GemmArgs g = batch_entry<T>(g0);
  __shared__ float As[16][64 + 4];
  __shared__ float Bs[16][64 + 4];
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  const int64_t m0 = (int64_t)blockIdx.y * 64, n0 = (int64_t)blockIdx.x * 64;
  const T *A = (const T *)g.a, *W = (const T *)g.w;
  float acc[4][4] = {};
  for (int64_t k0 = 0; k0 < g.k; k0 += 16) {
    for (int i = threadIdx.x; i < 64 * 16; i += 256) {
      int r = i / 16, kk = i % 16;
      int64_t gr = m0 + r, gk = k0 + kk;
      As[kk][r] = (gr < g.m && gk < g.k) ? ld<T>(A + gr * g.lda + gk) : 0.f;
      int64_t gn = n0 + r;
      Bs[kk][r] = (gn < g.n && gk < g.k) ? ld<T>(W + gn * g.k + gk) : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = As[kk][ty * 4 + i];
        b[i] = Bs[kk][tx * 4 + i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int64_t r = m0 + ty * 4 + i, c = n0 + tx * 4 + j;
      if (r < g.m && c < g.n) epilogue<T>(g, g.epi, r, c, acc[i][j]);
    }
}

// ---------------------------------------------------------------- bf16 MFMA kernel
constexpr int BK = 64;  // K per LDS stage: one 128-byte row of bf16 per tile row
constexpr int RSRC_WORD3 = 0x00020000;  // raw buffer: 32-bit data format, no swizzle
constexpr int WAIT_VM0 = 0x0F70;        // s_waitcnt vmcnt(0), other counters untouched
constexpr int WAIT_LGKM0 = 0xC07F;      // s_waitcnt lgkmcnt(0), other counters untouched
// s_waitcnt vmcnt(n) with the other counters untouched; n above the counter's
// 6-bit range is clamped (a wave never has more than 63 operations pending)
__host__ __device__ constexpr int vm_wait(int n) {
  return n > 63 ? vm_wait(63) : (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8);
}

typedef __attribute__((address_space(3))) void lds_void;
// 16 bytes per lane from a buffer straight into LDS (lane L at lds + 16 L); kept
// out of the kernel templates, where the builtin makes the host pass drop stubs
__device__ __forceinline__ void lds_load16(__amdgpu_buffer_rsrc_t r, char *lds, int voff, int soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void *)lds, 16, voff, soff, 0, 0);
}

template <int BM, int BN, int WM, int WN>
struct Cfg {
  static constexpr int NT = 64 * WM * WN;       // threads
  static constexpr int TM = BM / WM / 32;       // 32x32 tiles per wave along M
  static constexpr int TN = BN / WN / 32;       // along N
  // the first LW waves (one per SIMD) issue the tile loads: with all 16 waves
  // loading, the 16-wave kernel was 2-5% slower on the 13B products
  static constexpr int LW = NT / 64 >= 4 ? 4 : NT / 64;
  static constexpr int A_CHUNKS = BM * 8 / (64 * LW);  // 1 KB stripes per loading wave per stage
  static constexpr int B_CHUNKS = BN * 8 / (64 * LW);
  static constexpr int LDS_BYTES = 2 * (BM + BN) * BK * 2;
};

// Each tile row is 8 chunks of 16 bytes (128 B, two rows per 256-byte span of
// the 64 LDS banks). Chunk c of row r lives at c ^ ((r >> 1) & 7), so the 16
// rows read by 16 consecutive lanes land on 16 distinct 16-byte bank groups.
__device__ __forceinline__ int swz(int row, int chunk) { return (row * 8 + (chunk ^ ((row >> 1) & 7))) * 16; }

template <int EPI>
__device__ __forceinline__ float epi_act(float v) {
  if (EPI == EPI_GELU) {
    // 0.5 v (1 + tanh(u)) = v * sigmoid(2u), u = sqrt(2/pi) (v + 0.044715 v^3);
    // the hardware exp2 and reciprocal (about 1 ulp each) replace exp and the
    // IEEE division: the result is rounded to bfloat16 (8 significant bits)
    // exp(-2u) = exp2(v (A + B v^2)), A = -2 sqrt(2/pi) log2(e), B = 0.044715 A
    constexpr float A = -2.f * 0.7978845608028654f * 1.4426950408889634f, B = 0.044715f * A;
    return v * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(v * fmaf(B, v * v, A)));
  }
  return v;
}

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
// two floats -> packed bfloat16 pair (one v_cvt_pk_bf16_f32: round to nearest
// even, NaN stays NaN), low half first
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  bf16x2_t p;
  p[0] = (__bf16)lo;
  p[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, p);
}

// ---------------------------------------------------------------- fused q/k/v epilogue (EPI_QKV)
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
// V^T position of token j (and token of position j): bits 2 and 3 swapped
__device__ __forceinline__ int64_t vt_swap(int64_t j) { return (j & ~(int64_t)12) | ((j & 4) << 1) | ((j & 8) >> 1); }

// The block's 256 x 256 bf16 tile (bias added, rounded once) sits in LDS as the
// staged epilogue leaves it: wave (wm, wn) of 2 x 4 holds rows 128 wm.., columns
// 64 wn.. as 128-byte rows, 16-byte chunk c of row r at c ^ (r & 7). The tile
// lies inside the q, k or v columns (d is a multiple of 256).
__device__ __forceinline__ const char *qkv_chunk(const char *smem, int row, int cc) {
  const int slice = (row >> 7) * 4 + (cc >> 3), r = row & 127;
  return smem + slice * (128 * 128) + r * 128 + (((cc & 7) ^ (r & 7)) * 16);
}

// q or k: per head row the RMSNorm (float32, eps 1e-6) and the rotation of the
// video tokens' pairs (2p, 2p + 1), one more bf16 rounding, 16-byte stores of
// whole head rows. HD / 8 consecutive lanes hold one head row. The arithmetic
// is that of the separate preparation kernel (k_qk_prep8), without fused
// multiply-adds in either, so both give the same bits.
template <int HD, bool ROPE>
__device__ __forceinline__ void qk_scatter(const GemmArgs &g, const char *smem, int64_t m0, int h0, bf16_t *dst) {
#pragma clang fp contract(off)
  const QkvOut &o = g.qkv;
  constexpr int TPH = HD / 8;
  // Iteration it handles tile row 16 it + threadIdx.x / 32; the thread's chunk
  // of the row (threadIdx.x % 32: head hh, eight columns from 8 c) is the same
  // in every iteration. The sample and token advance incrementally (no
  // division per row). With a rotation table (ROPE: a table and video rows)
  // its entries go out four rows at a time, one group of four ahead, and
  // unconditionally (rows that take no rotation read table row 0), so the
  // stores of a group never stand between a table read and its use.
  const int cc = threadIdx.x & 31, hh = cc / TPH, c = cc % TPH;
  const int64_t r_first = m0 + (threadIdx.x >> 5);
  int64_t b = (int64_t)blockIdx.z + r_first / o.rps, jr = r_first % o.rps;
  int64_t bsv[2][4], jv[2][4];   // group g4 in slot g4 & 1
  float4 cs4v[2][4][2];
  auto rotates = [&](int it, int64_t jt) { return ROPE && jt < o.n_video && m0 + 16 * it + (threadIdx.x >> 5) < g.m; };
  auto coords = [&](int64_t (&bs4)[4], int64_t (&j4)[4]) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      bs4[u] = b;
      j4[u] = o.row0 + jr;
      jr += 16;
      while (jr >= o.rps) {
        jr -= o.rps;
        ++b;
      }
    }
  };
  auto fetch = [&](int g4, const int64_t (&js)[4], float4 (&dst4)[4][2]) {
    if (!ROPE) return;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t jt = rotates(4 * g4 + u, js[u]) ? js[u] : 0;
      const float4 *cs4 = (const float4 *)(o.rope + jt * (HD / 2) + 4 * c);
      dst4[u][0] = cs4[0];
      dst4[u][1] = cs4[1];
    }
  };
  coords(bsv[0], jv[0]);
  fetch(0, jv[0], cs4v[0]);
#pragma unroll
  for (int g4 = 0; g4 < 4; ++g4) {
    const int sl = g4 & 1;
    if (g4 + 1 < 4) {
      coords(bsv[sl ^ 1], jv[sl ^ 1]);
      fetch(g4 + 1, jv[sl ^ 1], cs4v[sl ^ 1]);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int it = 4 * g4 + u, row = 16 * it + (threadIdx.x >> 5);
      float x[8];
      unpack8(*(const uint4 *)qkv_chunk(smem, row, cc), x);
      if (o.qk_norm) {
        float sq = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) sq += x[e] * x[e];
        sq = group_sum<TPH>(sq);
        const float rs = rsqrtf(sq / (float)HD + 1e-6f);
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] *= rs;
      }
      if (m0 + row >= g.m) continue;
      if (rotates(it, jv[sl][u])) {
        const float4 c01 = cs4v[sl][u][0], c23 = cs4v[sl][u][1];
        const float cs[8] = {c01.x, c01.y, c01.z, c01.w, c23.x, c23.y, c23.z, c23.w};
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          const float co = cs[2 * p], si = cs[2 * p + 1];
          const float t0 = x[2 * p] * co - x[2 * p + 1] * si, t1 = x[2 * p] * si + x[2 * p + 1] * co;
          x[2 * p] = t0;
          x[2 * p + 1] = t1;
        }
      }
      *(uint4 *)(dst + ((bsv[sl][u] * o.heads + h0 + hh) * o.n_pad + jv[sl][u]) * HD + 8 * c) = pack8(x);
    }
  }
}

// v: transposed into [heads, hd, n_pad] in the V^T key order. A tile whose
// first token is 16-aligned and whose rows all belong to one sample writes 8
// consecutive positions (one 16-byte store) per lane for every group of 16
// tokens it holds whole; partial groups and other tiles go element by element
// (positions of missing tokens are padding, zeroed separately).
template <int HD>
__device__ __forceinline__ void v_scatter(const GemmArgs &g, const char *smem, int64_t m0, int h0) {
  const QkvOut &o = g.qkv;
  bf16_t *v = (bf16_t *)o.v;
  auto at = [&](int row, int col) -> uint32_t {
    return *(const bf16_t *)(qkv_chunk(smem, row, col >> 3) + 2 * (col & 7));
  };
  const int64_t mr = m0 % o.rps;
  const bool clean = (o.row0 + mr) % 16 == 0 && mr + 256 <= o.rps;
  static_assert(HD == 64 || HD == 128, "head size");
  if (clean) {
    // a wavefront's lanes take 64 consecutive columns at one chunk of 8
    // positions: every LDS read of the wave hits one 128-byte tile row segment
    // (columns of a fixed token are contiguous; tokens of a fixed column 16
    // apart would all fall on one bank)
    const int64_t b = (int64_t)blockIdx.z + m0 / o.rps, j0 = o.row0 + mr;
#pragma unroll 2
    for (int it = 0; it < 16; ++it) {
      const int col = threadIdx.x & 255, p8 = 2 * it + (threadIdx.x >> 8);
      const int hh = col / HD, e = col % HD, grp = 16 * (p8 >> 1), half = p8 & 1;
      bf16_t *dst = v + ((b * o.heads + h0 + hh) * HD + e) * o.n_pad + j0;
      if (m0 + grp + 16 <= g.m) {
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t0 = grp + (int)vt_swap(8 * half + 2 * i), t1 = grp + (int)vt_swap(8 * half + 2 * i + 1);
          w[i] = at(t0, col) | (at(t1, col) << 16);
        }
        *(uint4 *)(dst + 8 * p8) = make_uint4(w[0], w[1], w[2], w[3]);
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int t = grp + (int)vt_swap(8 * half + i);
          if (m0 + t < g.m) dst[8 * p8 + i] = (bf16_t)at(t, col);
        }
      }
    }
  } else {
    // element by element: the thread's column is fixed, its row steps by 2
    const int col = threadIdx.x & 255, hh = col / HD, e = col % HD;
    const int64_t r_first = m0 + (threadIdx.x >> 8);
    int64_t b = (int64_t)blockIdx.z + r_first / o.rps, jr = r_first % o.rps;
    for (int it = 0; it < 128; ++it) {
      const int row = 2 * it + (threadIdx.x >> 8);
      const int64_t bs = b, j = o.row0 + jr;
      jr += 2;
      while (jr >= o.rps) {
        jr -= o.rps;
        ++b;
      }
      if (m0 + row >= g.m) break;
      v[((bs * o.heads + h0 + hh) * HD + e) * o.n_pad + vt_swap(j)] = (bf16_t)at(row, col);
    }
  }
}

template <int BM, int BN, int WM, int WN, int EPI>
__global__ __launch_bounds__(64 * WM * WN) void k_gemm_mfma(GemmArgs g0) {
  using C = Cfg<BM, BN, WM, WN>;
  // bf16 outputs: compute C^T tiles (weight fragment as the MFMA A operand) so a
  // lane holds 4 consecutive columns of one row (8-byte stores); float32 outputs
  // keep C tiles, whose lanes cover 32 consecutive columns of two rows (a full
  // 128-byte line per read-modify-write instruction)
  constexpr bool TR = EPI == EPI_STORE || EPI == EPI_GELU || EPI == EPI_QKV;
  static_assert(EPI != EPI_QKV || (BM == 256 && BN == 256 && WM == 2 && WN == 4), "EPI_QKV: 256 x 256, 8 waves");
  constexpr bool RES = EPI == EPI_GATE_RES || EPI == EPI_GATE_RES_NT;   // gated residual into the float32 stream
  constexpr bool STAGE_OUT = BM == 256;   // bf16 output through LDS, whole-line non-temporal stores
  const GemmArgs g = batch_entry<bf16_t>(g0);
  extern __shared__ __attribute__((aligned(16))) char smem[];
  char *sA = smem;                      // [2][BM][128 B]
  char *sB = smem + 2 * BM * BK * 2;    // [2][BN][128 B]

  // Tile order: a group of 8 consecutive M tiles walks all N tiles, so blocks
  // running at once share A rows and the weight panel in L2.
  const int n_tiles = (int)(g.n / BN);
  const int m_tiles = (int)((g.m + BM - 1) / BM);
  const int bid = blockIdx.x;
  const int group = 8;
  const int per_group = group * n_tiles;
  const int gidx = bid / per_group;
  const int first_m = gidx * group;
  const int gsize = min(m_tiles - first_m, group);
  int mt, nt;
  if (g.order == 1) {
    // Dispatch rounds of 256 blocks, one per CU; block id % 8 is its XCD. Round
    // r gives XCD x chunk 8r + x: a (32 / rect_n) (M) x rect_n (N) rectangle of
    // tiles (8 x 4 or 2 x 16), one per block, so the 32 blocks an XCD runs
    // together start together and share their A and weight slices in its L2.
    // Blocks past the last tile exit.
    const int r = bid / 256, x = bid % 8, l = (bid / 8) % 32;
    const int rn = g.rect_n, rm = 32 / rn;
    const int chunk = 8 * r + x, cpb = n_tiles / rn;
    mt = rm * (chunk / cpb) + l % rm;
    nt = rn * (chunk % cpb) + l / rm;
    if (mt >= m_tiles) return;
  } else if (gsize == group && n_tiles >= 24) {
    // Workgroups go to the 8 XCDs round robin (id % 8). Give each XCD a
    // contiguous run of n_tiles tiles of the group in (nt, mt) order: an
    // 8-row by n_tiles/8-column rectangle, so the ~32 blocks one XCD runs at
    // once share 8 A slices and a few B slices in its L2 (+5.6% at N = 12,288,
    // K = 3,072). Narrow products (N = 3,072, long K) keep one row tile per XCD
    // against every column tile, which measured 3% faster for them.
    const int b = bid % per_group;
    const int idx = (b % 8) * n_tiles + b / 8;
    mt = first_m + idx % group;
    nt = idx / group;
  } else {
    mt = first_m + (bid % per_group) % gsize;
    nt = (bid % per_group) / gsize;
  }
  const int64_t m0 = (int64_t)mt * BM, n0 = (int64_t)nt * BN;

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm = wid / WN, wn = wid % WN;
  const int lr = lane & 31, lg = lane >> 5;

  // Tiles go straight from HBM to LDS (buffer_load_dwordx4 ... lds: lane L of a
  // wavefront's load writes 16 bytes at LDS base + 16 L). Stripe s = 1 KB = 8
  // tile rows; loading wave w (of NW) loads stripes w, w + NW, w + 2 NW, ... so each lane fetches
  // row 8s + lane/8 and the logical chunk that the swizzle puts at physical
  // chunk lane%8 (the swizzle key (row >> 1) & 7 is the same for every stripe
  // of a wave since NW is even).
  // The A descriptor spans only this block's valid rows and every stripe's row
  // is in the VGPR offset, which the buffer range check covers: rows past m are
  // read as zero (the K offset rides in the SGPR offset and is always in range).
  constexpr int NW = C::LW;
  static_assert(NW % 2 == 0, "stripe swizzle assumes an even wave count");
  const int64_t rows_a = min((int64_t)BM, g.m - m0);
  const __amdgpu_buffer_rsrc_t a_desc = __builtin_amdgcn_make_buffer_rsrc(
      (void *)((const bf16_t *)g.a + m0 * g.lda), (short)0, (int)(rows_a * g.lda * 2), RSRC_WORD3);
  const __amdgpu_buffer_rsrc_t b_desc = __builtin_amdgcn_make_buffer_rsrc(
      (void *)((const bf16_t *)g.w + n0 * g.k), (short)0, (int)(BN * g.k * 2), RSRC_WORD3);
  const int wu = __builtin_amdgcn_readfirstlane(wid);
  const int lch = (lane & 7) ^ ((4 * (wu & 1) + (lane >> 4)) & 7);
  const int row0 = 8 * wu + (lane >> 3);
  // A stripe i is row0 + 8 NW i: its offset steps by a_step from stripe to
  // stripe, added in the load sequence itself (an asm add the compiler cannot
  // hoist) so the loop does not keep A_CHUNKS offsets live in VGPRs
  const int va0 = row0 * (int)g.lda * 2 + lch * 16;
  const int a_step = 8 * NW * (int)g.lda * 2;
  const int vb = row0 * (int)g.k * 2 + lch * 16;

  // fragment read offsets: row wm*(BM/WM) + 32i + lr, chunk 2s + lg; the
  // swizzle key depends on the row only, so k-step s reads at offset(0) ^ 32 s
  const int ra0 = swz(wm * (BM / WM) + lr, lg), rb0 = swz(wn * (BN / WN) + lr, lg);

#define WDC_GEMM_LOAD(buf, kt)                                                                     \
  {                                                                                                \
    const int kb_ = (kt) * BK * 2;                                                                 \
    if (wu < NW) {                                                                                 \
      int v_ = va0;                                                                                \
      _Pragma("unroll") for (int i = 0; i < C::A_CHUNKS; ++i) {                                     \
        lds_load16(a_desc, sA + (buf) * BM * 128 + (i * NW + wu) * 1024, v_, kb_);                  \
        if (i + 1 < C::A_CHUNKS) asm volatile("v_add_u32 %0, %0, %1" : "+v"(v_) : "s"(a_step));     \
      }                                                                                            \
      _Pragma("unroll") for (int i = 0; i < C::B_CHUNKS; ++i)                                       \
          lds_load16(b_desc, sB + (buf) * BN * 128 + (i * NW + wu) * 1024, vb, i * 8 * NW * (int)g.k * 2 + kb_); \
    }                                                                                              \
  }

  // k-step s of the stage in buffer buf: the wave's TM A and TN B fragments
#define WDC_GEMM_READ(fa, fb, buf, s)                                                               \
  {                                                                                                \
    const char *a_ = sA + (buf) * BM * 128, *b_ = sB + (buf) * BN * 128;                           \
    const int oa_ = ra0 ^ (32 * (s)), ob_ = rb0 ^ (32 * (s));                                      \
    _Pragma("unroll") for (int i = 0; i < C::TM; ++i) fa[i] = *(const bf16x8 *)(a_ + oa_ + i * 32 * 128); \
    _Pragma("unroll") for (int j = 0; j < C::TN; ++j) fb[j] = *(const bf16x8 *)(b_ + ob_ + j * 32 * 128); \
  }
  // Workgroup barrier after this wave's LDS reads complete, without the memory
  // fence of __syncthreads (whose vmcnt(0) would also wait for a stage still
  // in flight). The wait is the builtin rather than asm so that the compiler's
  // own wait tracking sees the fragment reads as complete.
#define WDC_GEMM_BARRIER()                                                                         \
  {                                                                                                \
    __builtin_amdgcn_s_waitcnt(WAIT_LGKM0);                                                        \
    __builtin_amdgcn_s_barrier();                                                                  \
  }

  constexpr int S = BK / 16;                              // k-steps per stage
  constexpr int SL = C::A_CHUNKS + C::B_CHUNKS;           // load instructions per loading wave per stage
  const int nk = (int)(g.k / BK);
  // Stages 0 and 1 fill both buffers; stage 0 is complete once no more than
  // stage 1's loads are pending (a wave's memory operations complete in issue
  // order).
  WDC_GEMM_LOAD(0, 0);
  if (nk > 1) WDC_GEMM_LOAD(1, 1);
  if (wu < NW) {
    if (nk > 1) __builtin_amdgcn_s_waitcnt(vm_wait(SL));
    else __builtin_amdgcn_s_waitcnt(WAIT_VM0);
  }
  WDC_GEMM_BARRIER();

  f32x16 acc[C::TM][C::TN];
#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  // Software pipeline over two fragment sets x and y: the fragments of k-step
  // s+1 are read while the MFMAs of step s run. The stage barrier sits before
  // the last k-step, whose fragments are already in registers: after it the
  // stage two ahead goes into the buffer just consumed and the next stage's
  // first fragments are read, both under the last step's MFMAs, so the matrix
  // cores do not drain at the barrier. Within a step the reads and loads are
  // interleaved one by one with the MFMAs in a fixed order (a scheduling
  // barrier after each), so they issue while the wave's MFMAs execute; the
  // reads go in the order the next step's MFMAs use them (A0, every B, then
  // the other A fragments).
  static_assert(S == 4, "the x/y alternation assumes four k-steps per stage");
  constexpr int NQ = C::TM * C::TN, NR = C::TM + C::TN;
#define WDC_GEMM_MFMA1(fa, fb, q)                                                                   \
  {                                                                                                \
    const int i_ = (q) / C::TN, j_ = (q) % C::TN;                                                  \
    acc[i_][j_] = TR ? __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[j_], fa[i_], acc[i_][j_], 0, 0, 0) \
                     : __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i_], fb[j_], acc[i_][j_], 0, 0, 0); \
  }
  // read number r of a step: 0 -> A0, 1..TN -> B0..B(TN-1), then A1..A(TM-1)
#define WDC_GEMM_READ1(fa, fb, buf, s, r)                                                          \
  {                                                                                                \
    const bool isb_ = (r) >= 1 && (r) <= C::TN;                                                    \
    const int ia_ = (r) == 0 ? 0 : (r) - C::TN, jb_ = (r) - 1;                                     \
    if (isb_)                                                                                      \
      fb[isb_ ? jb_ : 0] = *(const bf16x8 *)(sB + (buf) * BN * 128 + (rb0 ^ (32 * (s))) + (isb_ ? jb_ : 0) * 32 * 128); \
    else                                                                                           \
      fa[isb_ ? 0 : ia_] = *(const bf16x8 *)(sA + (buf) * BM * 128 + (ra0 ^ (32 * (s))) + (isb_ ? 0 : ia_) * 32 * 128); \
  }
  // load number l of a stage (A stripes first, then B); v_ steps through the A stripes
#define WDC_GEMM_LOAD1(buf, kt, l)                                                                 \
  {                                                                                                \
    if ((l) < C::A_CHUNKS) {                                                                       \
      lds_load16(a_desc, sA + (buf) * BM * 128 + ((l) * NW + wu) * 1024, v_, (kt) * BK * 2);       \
      if ((l) + 1 < C::A_CHUNKS) asm volatile("v_add_u32 %0, %0, %1" : "+v"(v_) : "s"(a_step));     \
    } else {                                                                                       \
      const int lb_ = (l) - C::A_CHUNKS;                                                           \
      lds_load16(b_desc, sB + (buf) * BN * 128 + (lb_ * NW + wu) * 1024, vb,                       \
                 lb_ * 8 * NW * (int)g.k * 2 + (kt) * BK * 2);                                     \
    }                                                                                              \
  }
  // one k-step: the MFMAs on (ca, cb); if READS, the reads of step rs of buffer
  // rbuf into (na, nb); if LOADS (a uniform condition), the loads of stage lkt
  // into buffer lbuf
#define WDC_GEMM_STEP(ca, cb, na, nb, rbuf, rs, READS, lbuf, lkt, LOADS)                           \
  {                                                                                                \
    int v_ = va0;                                                                                  \
    _Pragma("unroll") for (int q = 0; q < NQ; ++q) {                                               \
      WDC_GEMM_MFMA1(ca, cb, q);                                                                   \
      __builtin_amdgcn_sched_barrier(0);                                                           \
      /* load l goes after MFMA l NQ / SL, read r after MFMA r NQ / NR (constant bounds, */     \
      /* so the loops unroll fully and every register index is a constant) */                      \
      /* (LOADS is a run-time condition: the branch holds loads only, so the */                   \
      /* accumulators never meet at a join) */                                                     \
      if (LOADS) {                                                                                 \
        _Pragma("unroll") for (int l = 0; l < SL; ++l) {                                           \
          if (l * NQ / SL == q) {                                                                  \
            WDC_GEMM_LOAD1(lbuf, lkt, l);                                                          \
          }                                                                                        \
        }                                                                                          \
      }                                                                                            \
      __builtin_amdgcn_sched_barrier(0);                                                           \
      if (READS) {                                                                                 \
        _Pragma("unroll") for (int r = 0; r < NR; ++r) {                                           \
          if (r * NQ / NR == q) {                                                                  \
            WDC_GEMM_READ1(na, nb, rbuf, rs, r);                                                   \
            __builtin_amdgcn_sched_barrier(0);                                                     \
          }                                                                                        \
        }                                                                                          \
      }                                                                                            \
    }                                                                                              \
    (void)v_;                                                                                      \
  }
  bf16x8 xa[C::TM], xb[C::TN], ya[C::TM], yb[C::TN];
  WDC_GEMM_READ(xa, xb, 0, 0);
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    WDC_GEMM_STEP(xa, xb, ya, yb, buf, 1, true, 0, 0, false);
    WDC_GEMM_STEP(ya, yb, xa, xb, buf, 2, true, 0, 0, false);
    WDC_GEMM_STEP(xa, xb, ya, yb, buf, 3, true, 0, 0, false);
    // stage kt+1 was requested a stage ago; after the barrier every wave's
    // reads of buffer buf are complete. The last stage's step also reads the
    // other buffer's first fragments: stale data, never used.
    if (wu < NW) __builtin_amdgcn_s_waitcnt(WAIT_VM0);
    WDC_GEMM_BARRIER();
    const bool ld = kt + 2 < nk && wu < NW;
    WDC_GEMM_STEP(ya, yb, xa, xb, buf ^ 1, 0, true, buf, kt + 2, ld);
  }
#undef WDC_GEMM_STEP
#undef WDC_GEMM_LOAD1
#undef WDC_GEMM_READ1
#undef WDC_GEMM_MFMA1

  const bf16_t *bias = (const bf16_t *)g.bias;
  if (TR && STAGE_OUT) {
    // bf16 output staged through LDS (free once the last K stage is consumed:
    // every read that matters completed before the last stage barrier): each
    // wave writes its BM/WM x BN/WN tile into its own slice, row-major with the
    // 16-byte chunk index XOR (row & 7), then reads it back so that every store
    // instruction writes whole 128-byte row segments, marked non-temporal.
    constexpr int RB = BN / WN * 2, CPR = RB / 16, RPI = 1024 / RB, WR = BM / WM;
    static_assert(WR * RB * C::NT / 64 <= C::LDS_BYTES, "staging slices exceed LDS");
    char *wl = smem + wid * (WR * RB);
    uint2 bw[C::TN][4];
#pragma unroll
    for (int j = 0; j < C::TN; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        bw[j][q] = bias ? *(const uint2 *)(bias + n0 + wn * (BN / WN) + j * 32 + 4 * lg + 8 * q) : make_uint2(0, 0);
#pragma unroll
    for (int j = 0; j < C::TN; ++j) {
#pragma unroll
      for (int i = 0; i < C::TM; ++i) {
        const int r = i * 32 + lr;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float b0 = bf2f((bf16_t)(bw[j][q].x & 0xffff)), b1 = bf2f((bf16_t)(bw[j][q].x >> 16));
          const float b2 = bf2f((bf16_t)(bw[j][q].y & 0xffff)), b3 = bf2f((bf16_t)(bw[j][q].y >> 16));
          const uint32_t w0 = pack_bf16(epi_act<EPI>(acc[i][j][4 * q + 0] + b0), epi_act<EPI>(acc[i][j][4 * q + 1] + b1));
          const uint32_t w1 = pack_bf16(epi_act<EPI>(acc[i][j][4 * q + 2] + b2), epi_act<EPI>(acc[i][j][4 * q + 3] + b3));
          *(uint2 *)(wl + r * RB + (((4 * j + q) ^ (r & 7)) * 16) + 8 * lg) = make_uint2(w0, w1);
        }
      }
    }
    if constexpr (EPI == EPI_QKV) {
      __syncthreads();                      // every wave's slice is written
      const int region = (int)(n0 / g.qkv.d), h0 = (int)((n0 % g.qkv.d) / g.qkv.hd);
      if (region < 2) {
        bf16_t *dst = (bf16_t *)(region == 0 ? g.qkv.q : g.qkv.k);
        const bool rope = g.qkv.rope && g.qkv.n_video > 0;
        if (g.qkv.hd == 128) {
          if (rope) qk_scatter<128, true>(g, smem, m0, h0, dst);
          else qk_scatter<128, false>(g, smem, m0, h0, dst);
        } else {
          if (rope) qk_scatter<64, true>(g, smem, m0, h0, dst);
          else qk_scatter<64, false>(g, smem, m0, h0, dst);
        }
      } else if (g.qkv.hd == 128) {
        v_scatter<128>(g, smem, m0, h0);
      } else {
        v_scatter<64>(g, smem, m0, h0);
      }
      return;
    }
    typedef __attribute__((ext_vector_type(4))) unsigned u32x4_t;
#pragma unroll
    for (int s = 0; s < WR / RPI; ++s) {
      const int r = s * RPI + lane / CPR, ch = lane % CPR;
      const u32x4_t v = *(const u32x4_t *)(wl + r * RB + ((ch ^ (r & 7)) * 16));
      const int64_t row = m0 + wm * WR + r;
      if (row < g.m)
        __builtin_nontemporal_store(v, (u32x4_t *)((bf16_t *)g.c + row * g.ldc + n0 + wn * (BN / WN) + ch * 8));
    }
  } else if constexpr (TR) {
    // bf16 output: lane (lr, lg) of tile (i, j) holds row lr of the 32x32 output
    // tile and, in accumulator entries 4q..4q+3, the four consecutive columns
    // 8q + 4lg + 0..3, stored as one 8-byte group. The bias of all the lane's
    // columns is read before the first store, so one wait covers every read.
    uint2 bw[C::TN][4];
#pragma unroll
    for (int j = 0; j < C::TN; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        bw[j][q] = bias ? *(const uint2 *)(bias + n0 + wn * (BN / WN) + j * 32 + 4 * lg + 8 * q) : make_uint2(0, 0);
#pragma unroll
    for (int j = 0; j < C::TN; ++j) {
      const int64_t cb = n0 + wn * (BN / WN) + j * 32 + 4 * lg;   // column of group q: cb + 8 q
      float bq[4][4];                                               // bias of the lane's 16 columns
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        bq[q][0] = bf2f((bf16_t)(bw[j][q].x & 0xffff));
        bq[q][1] = bf2f((bf16_t)(bw[j][q].x >> 16));
        bq[q][2] = bf2f((bf16_t)(bw[j][q].y & 0xffff));
        bq[q][3] = bf2f((bf16_t)(bw[j][q].y >> 16));
      }
#pragma unroll
      for (int i = 0; i < C::TM; ++i) {
        const int64_t row = m0 + wm * (BM / WM) + i * 32 + lr;
        if (row >= g.m) continue;
        bf16_t *out = (bf16_t *)g.c + row * g.ldc + cb;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t w0 = pack_bf16(epi_act<EPI>(acc[i][j][4 * q + 0] + bq[q][0]),
                                        epi_act<EPI>(acc[i][j][4 * q + 1] + bq[q][1]));
          const uint32_t w1 = pack_bf16(epi_act<EPI>(acc[i][j][4 * q + 2] + bq[q][2]),
                                        epi_act<EPI>(acc[i][j][4 * q + 3] + bq[q][3]));
          *(uint2 *)(out + 8 * q) = make_uint2(w0, w1);
        }
      }
    }
  } else {
    // float32 output: lane holds column lr of each 32x32 tile, rows
    // 8 (e / 4) + 4 lg + e % 4; 32 lanes cover one 128-byte line per row
    float bvs[C::TN], gvs[C::TN];
#pragma unroll
    for (int j = 0; j < C::TN; ++j) {
      const int64_t col = n0 + wn * (BN / WN) + j * 32 + lr;
      bvs[j] = bias ? bf2f(bias[col]) : 0.f;
      gvs[j] = RES ? g.gate[col] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < C::TN; ++j) {
      const int64_t col = n0 + wn * (BN / WN) + j * 32 + lr;
      const float bv = bvs[j], gv = gvs[j];
#pragma unroll
      for (int i = 0; i < C::TM; ++i) {
        const int64_t rb = m0 + wm * (BM / WM) + i * 32 + 4 * lg;   // row of element e: rb + 8 (e / 4) + e % 4
        float *xc = (float *)g.c + rb * g.ldc + col;
        if (m0 + wm * (BM / WM) + i * 32 + 32 <= g.m) {
          // whole 32-row tile inside m (uniform per wave): no per-element guard, so
          // the residual reads go out together (vmcnt also counts stores, and a
          // guarded store per element would serialise every read-modify-write)
          if constexpr (RES) {
            float xr[16];
            if constexpr (EPI == EPI_GATE_RES_NT) {
#pragma unroll
              for (int e = 0; e < 16; ++e) xr[e] = __builtin_nontemporal_load(&xc[(8 * (e / 4) + (e % 4)) * g.ldc]);
#pragma unroll
              for (int e = 0; e < 16; ++e)
                __builtin_nontemporal_store(xr[e] + gv * (acc[i][j][e] + bv), &xc[(8 * (e / 4) + (e % 4)) * g.ldc]);
            } else {
#pragma unroll
              for (int e = 0; e < 16; ++e) xr[e] = xc[(8 * (e / 4) + (e % 4)) * g.ldc];
#pragma unroll
              for (int e = 0; e < 16; ++e) xc[(8 * (e / 4) + (e % 4)) * g.ldc] = xr[e] + gv * (acc[i][j][e] + bv);
            }
          } else {
#pragma unroll
            for (int e = 0; e < 16; ++e) xc[(8 * (e / 4) + (e % 4)) * g.ldc] = acc[i][j][e] + bv;
          }
          continue;
        }
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int64_t row = rb + 8 * (e / 4) + (e % 4);
          if (row >= g.m) continue;
          float *x = (float *)g.c + row * g.ldc + col;
          if (RES)
            *x += gv * (acc[i][j][e] + bv);
          else
            *x = acc[i][j][e] + bv;
        }
      }
    }
  }
#undef WDC_GEMM_READ
#undef WDC_GEMM_BARRIER
#undef WDC_GEMM_LOAD
}

template <int BM, int BN, int WM, int WN>
hipError_t launch_mfma(const GemmArgs &g0, hipStream_t s) {
  using C = Cfg<BM, BN, WM, WN>;
  GemmArgs g = g0;
  const int m_tiles = (int)((g.m + BM - 1) / BM), n_tiles = (int)(g.n / BN);
  // The rectangle order pays on large single products; a z-batch would put every
  // slice's rectangles on the same XCDs, and with fewer than 8 dispatch rounds
  // the partly filled last round costs more than the L2 reuse gains (a batched
  // rollout of 8 mid-size samples ran 40% slower with it).
  // 8 x 4 rectangles. 2 x 16 ones (A panels, larger than the last-level cache,
  // re-read once per rectangle column; weight panels, which fit it, once per
  // rectangle row) made the N = 12,288 product 2.5-3% faster alone but the
  // whole 13B forward's GEMMs 1% slower (same-box A/B), so they are not used;
  // nor 2 x 16 for that product alone (1.1% slower over the forward) or 16 x 2
  // for the N = 3,072 ones (1.8% slower).
  g.rect_n = 4;
  const int chunks = n_tiles % g.rect_n == 0 ? (m_tiles + 32 / g.rect_n - 1) / (32 / g.rect_n) * (n_tiles / g.rect_n) : 0;
  g.order = (BM == 256 && chunks >= 64 && g.batch <= 1 && device_cus() == 256) ? 1 : 0;
  int blocks = m_tiles * n_tiles;
  if (g.order == 1) blocks = (chunks + 7) / 8 * 256;
  dim3 grid(blocks, 1, g.batch > 1 ? g.batch : 1), block(C::NT);
  switch (g.epi) {
    case EPI_STORE: hipLaunchKernelGGL((k_gemm_mfma<BM, BN, WM, WN, EPI_STORE>), grid, block, C::LDS_BYTES, s, g); break;
    case EPI_GELU: hipLaunchKernelGGL((k_gemm_mfma<BM, BN, WM, WN, EPI_GELU>), grid, block, C::LDS_BYTES, s, g); break;
    case EPI_GATE_RES: hipLaunchKernelGGL((k_gemm_mfma<BM, BN, WM, WN, EPI_GATE_RES>), grid, block, C::LDS_BYTES, s, g); break;
    case EPI_GATE_RES_NT: hipLaunchKernelGGL((k_gemm_mfma<BM, BN, WM, WN, EPI_GATE_RES_NT>), grid, block, C::LDS_BYTES, s, g); break;
    case EPI_QKV:
      if constexpr (BM == 256 && BN == 256 && WM == 2 && WN == 4) {
        hipLaunchKernelGGL((k_gemm_mfma<BM, BN, WM, WN, EPI_QKV>), grid, block, C::LDS_BYTES, s, g);
        break;
      } else {
        return hipErrorInvalidValue;
      }
    default: hipLaunchKernelGGL((k_gemm_mfma<BM, BN, WM, WN, EPI_STORE_F32>), grid, block, C::LDS_BYTES, s, g); break;
  }
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN>
hipError_t set_lds_limit() {
  using C = Cfg<BM, BN, WM, WN>;
  const void *k[5] = {(const void *)k_gemm_mfma<BM, BN, WM, WN, EPI_STORE>,
                      (const void *)k_gemm_mfma<BM, BN, WM, WN, EPI_GELU>,
                      (const void *)k_gemm_mfma<BM, BN, WM, WN, EPI_GATE_RES>,
                      (const void *)k_gemm_mfma<BM, BN, WM, WN, EPI_GATE_RES_NT>,
                      (const void *)k_gemm_mfma<BM, BN, WM, WN, EPI_STORE_F32>};
  for (const void *f : k) {
    const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS_BYTES);
    if (e != hipSuccess) return e;
  }
  if constexpr (BM == 256 && BN == 256 && WM == 2 && WN == 4)
    return hipFuncSetAttribute((const void *)k_gemm_mfma<BM, BN, WM, WN, EPI_QKV>,
                               hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS_BYTES);
  return hipSuccess;
}

bool operands_aligned(const GemmArgs &g) {
  return ((uintptr_t)g.a % 16 == 0) && ((uintptr_t)g.w % 16 == 0) && g.lda % 8 == 0 && g.k % BK == 0 &&
         (uintptr_t)g.c % 16 == 0 && g.ldc % 4 == 0 && (uintptr_t)g.bias % 8 == 0 && (uintptr_t)g.gate % 16 == 0 &&
         (g.batch <= 1 || (g.a_bs % 8 == 0 && g.c_bs % 4 == 0 && g.gate_bs % 4 == 0));
}

// products on fewer 256 x 256 tiles than the device has compute units take
// 128 x 128 tiles when the caller allows it (GemmArgs::fill_tiles)
bool small_product(const GemmArgs &g) {
  const int64_t tiles = (g.m + 255) / 256 * (g.n / 256) * (g.batch > 1 ? g.batch : 1);
  return g.fill_tiles && g.n % 128 == 0 && tiles < device_cus();
}
}  // namespace

bool gemm_qkv_fusable(int dtype, const GemmArgs &g) {
  const QkvOut &o = g.qkv;
  return dtype == 1 && operands_aligned(g) && g.n % 256 == 0 && g.m >= 512 && g.k < 8192 && !small_product(g) &&
         (o.hd == 64 || o.hd == 128) && o.d % 256 == 0 && g.n == 3 * (int64_t)o.d && o.rps > 0 &&
         o.n_pad % 8 == 0 && (uintptr_t)o.q % 16 == 0 && (uintptr_t)o.k % 16 == 0 && (uintptr_t)o.v % 16 == 0 &&
         (uintptr_t)o.rope % 16 == 0;
}

hipError_t launch_gemm(int dtype, const GemmArgs &g_in, hipStream_t s) {
  GemmArgs g = g_in;
  if (g.m <= 0 || g.n <= 0) return hipSuccess;
  if (g.epi == EPI_GATE_RES_NT) return hipErrorInvalidValue;   // internal, chosen below
  if (g.epi == EPI_QKV && !gemm_qkv_fusable(dtype, g)) return hipErrorInvalidValue;
  // the MFMA kernels read 16-byte operand chunks and write 4-column output groups
  const bool aligned = operands_aligned(g);
  if (dtype == 1 && aligned) {
    static bool seen[64] = {};
    if (first_on_device(seen)) {
      hipError_t e = set_lds_limit<256, 256, 2, 4>();
      if (e == hipSuccess) e = set_lds_limit<128, 128, 2, 2>();
      if (e == hipSuccess) e = set_lds_limit<128, 64, 2, 2>();
      if (e != hipSuccess) return e;
    }
    // 256 x 256 block tiles: 8 waves of 128 x 64 (two per SIMD). With the reads
    // and loads interleaved into the MFMA stream they were 0.3-1.5% faster than
    // 16 waves of 64 x 64 on the 13B products and read a quarter fewer LDS
    // bytes per MFMA (the chip is power-limited under this load).
    // Gated residual of a long-K product: the float32 stream's read-modify-write
    // goes past the caches (non-temporal), which then keep the A and weight
    // tiles: +7.5% at K = 12,288, +2% at K = 15,360; at K = 3,072 it was 1.5%
    // slower, so shorter products keep cached accesses.
    if (g.epi == EPI_GATE_RES && g.k >= 8192) g.epi = EPI_GATE_RES_NT;
    auto big = [&](const GemmArgs &gg) { return launch_mfma<256, 256, 2, 4>(gg, s); };
    // the 256 x 256 kernels stage bf16 outputs through LDS and store whole
    // 16-byte row chunks: they need 16-byte-aligned output rows (other bf16
    // outputs take the 128 x 128 kernels, which store 8-byte groups)
    const bool c16 = g.epi == EPI_STORE || g.epi == EPI_GELU;
    const bool out16 = !c16 || ((uintptr_t)g.c % 16 == 0 && g.ldc % 8 == 0 && (g.batch <= 1 || g.c_bs % 8 == 0));
    if (g.epi == EPI_QKV) return launch_mfma<256, 256, 2, 4>(g, s);
    // A product that would leave compute units idle in its only dispatch round
    // (the mid-size model's products: 44 to 176 tiles of 256 x 256) runs four
    // times the blocks on 128 x 128 tiles: 17% off the mid-size forward, whose
    // q/k/v projection then takes the separate preparation kernels. One that
    // would still leave CUs idle on 128 x 128 tiles (its N = 1,024 products:
    // 168 tiles) runs on 128 x 64 tiles, up to two blocks per CU: 5.7% off the
    // mid-size forward's products. Every output is summed over K in the same
    // order on any tile shape, so the results are the same bits.
    if (small_product(g)) {
      const int64_t t128 = (g.m + 127) / 128 * (g.n / 128) * (g.batch > 1 ? g.batch : 1);
      if (t128 < device_cus()) return launch_mfma<128, 64, 2, 2>(g, s);
      return launch_mfma<128, 128, 2, 2>(g, s);
    }
    if (g.n % 256 == 0 && g.m >= 512 && out16) {
      // Tail split for a single large long-K product on a 256-CU device: the
      // rows whose 256 x 256 tiles fill whole dispatch rounds (m1 tiles, a
      // multiple of 256 / gcd(n_tiles, 256)) run as above; the remaining rows,
      // which would leave most CUs idle in a last round at most half full, run
      // as 128 x 128 tiles (two blocks per CU). At M = 67,576 and N = 3,072 that
      // turns 12.375 rounds into 12 plus 2,040 rows: +1.5% at K = 12,288, +2% at
      // K = 15,360; at K = 3,072 the small tiles' lower efficiency costs more
      // than the idle CUs (-1.3%), so short products keep one launch.
      const int64_t m_tiles = (g.m + 255) / 256, n_tiles = g.n / 256;
      int64_t gcd = n_tiles, r = 256;
      while (r) { const int64_t t = gcd % r; gcd = r; r = t; }
      const int64_t m1 = m_tiles / (256 / gcd) * (256 / gcd) * 256;   // rows in whole rounds
      const bool thin_tail = (m_tiles * n_tiles) % 256 != 0 && (m_tiles * n_tiles) % 256 <= 128;
      if (g.batch <= 1 && g.k >= 8192 && thin_tail && device_cus() == 256 && m1 > 0 && m1 < g.m) {
        GemmArgs g1 = g, g2 = g;
        g1.m = m1;
        g2.m = g.m - m1;
        g2.a = (const bf16_t *)g.a + m1 * g.lda;
        g2.c = c16 ? (void *)((bf16_t *)g.c + m1 * g.ldc) : (void *)((float *)g.c + m1 * g.ldc);
        hipError_t e = big(g1);
        if (e != hipSuccess) return e;
        return launch_mfma<128, 128, 2, 2>(g2, s);
      }
      return big(g);
    }
    if (g.n % 128 == 0) return launch_mfma<128, 128, 2, 2>(g, s);
    // narrow outputs (the output head: n = 64 latent values per token)
    if (g.n % 64 == 0) return launch_mfma<128, 64, 2, 2>(g, s);
  }
  dim3 grid((unsigned)((g.n + 63) / 64), (unsigned)((g.m + 63) / 64), g.batch > 1 ? g.batch : 1), block(256);
  if (dtype == 1)
    hipLaunchKernelGGL(k_gemm_simple<bf16_t>, grid, block, 0, s, g);
  else
    hipLaunchKernelGGL(k_gemm_simple<float>, grid, block, 0, s, g);
  return hipGetLastError();
}

}  // namespace wdc

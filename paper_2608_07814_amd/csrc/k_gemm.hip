// Grouped GEMMs of the forward: every projection is C = A * W^T over the rows
// of one tree level, tile by tile, where a tile's rows all use the weights of
// one node (W in nn.Linear layout [N][K], K contiguous).
//
// bf16 path (gfx950 MFMA, v_mfma_f32_32x32x16_bf16):
//   * 128 x 128 output tile per 256-thread workgroup, 4 wavefronts of 64 x 64,
//     2 x 2 MFMA 32x32 blocks each, K staged through LDS 64 at a time;
//   * A rows may be gathered through an index map (activations per (token,
//     node) row), so no gathered copy of x is ever written;
//   * A may be bf16 (activations) or fp32 (intermediates). fp32 A is split
//     on the fly into hi = bf16(a) and lo = bf16(a - hi); both are multiplied
//     with the same weight fragment, which keeps about 16 bits of the
//     intermediate's mantissa at the cost of a second MFMA per fragment;
//   * LDS rows of 64 bf16 (128 B) are stored with the 16-byte chunk index
//     XOR-swizzled by the row so fragment reads of 32 consecutive rows hit
//     distinct banks;
//   * double-buffered LDS with register prefetch: the next K-slab is loaded
//     from HBM while the current one is multiplied.
// fp32 path: a plain LDS-tiled VALU kernel (fp32 layers are small).
#include "lx_internal.h"

namespace lx {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint16_t u16;

constexpr int BM = 128, BN = 128, BK = 64, NTHR = 256;
static_assert((BM & (BM - 1)) == 0, "tile heights are powers of two (bucketing shifts)");

__device__ __forceinline__ int swz(int row) { return (row ^ (row >> 3)) & 7; }
__device__ __forceinline__ int lds_off(int row, int kc) { return row * BK + ((kc ^ swz(row)) << 3); }

__device__ __forceinline__ void split_hilo(const float4& a, const float4& b, uint4& hi, uint4& lo) {
  const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  bf16x8 h, l;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const __bf16 hb = (__bf16)v[i];
    h[i] = hb;
    l[i] = (__bf16)(v[i] - (float)hb);
  }
  hi = __builtin_bit_cast(uint4, h);
  lo = __builtin_bit_cast(uint4, l);
}

template <int AMODE>
__global__ __launch_bounds__(NTHR) void k_gemm_bf16(GemmArgs p) {
  if ((int)blockIdx.x >= *p.n_tiles) return;
  const TileEntry te = p.tiles[blockIdx.x];
  const int ntp0 = (p.ncols[0] + BN - 1) / BN;
  const int part = (int)blockIdx.y < ntp0 ? 0 : 1;
  const int n0 = ((int)blockIdx.y - (part ? ntp0 : 0)) * BN;
  const int ncol = p.ncols[part];
  const int K = p.K;
  const int akoff = p.a_koff[part];
  const u16* __restrict__ Bw = (const u16*)p.B[part] + (int64_t)te.widx * p.b_stride[part];

  constexpr bool HILO = AMODE == A_F32_HILO;
  __shared__ __attribute__((aligned(16))) u16 sA[2][BM * BK];
  __shared__ __attribute__((aligned(16))) u16 sB[2][BN * BK];
  __shared__ __attribute__((aligned(16))) u16 sAl[HILO ? 2 : 1][HILO ? BM * BK : 8];

  const int tid = threadIdx.x;
  const int lrow = tid >> 3;   // 0..31
  const int lkc = tid & 7;     // 16-byte chunk within a 64-wide K slab

  // Rows this thread stages: lrow + 32*i. Invalid rows/columns read nothing
  // and stage zeros; their offsets are clamped to row 0 so no address is
  // ever formed outside the operands.
  int64_t aoff[4], boff[4];
  unsigned amask = 0, bmask = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = lrow + 32 * i;
    const bool av = r < te.nrows;
    const int64_t src = !av ? 0 : (p.a_rows ? (int64_t)p.a_rows[te.row0 + r] : (int64_t)(te.row0 + r));
    aoff[i] = src * p.lda + akoff;
    amask |= av ? (1u << i) : 0u;
    const int n = n0 + r;
    boff[i] = n < ncol ? (int64_t)n * K : 0;
    bmask |= n < ncol ? (1u << i) : 0u;
  }
  const u16* __restrict__ Ab = (const u16*)p.A;
  const float* __restrict__ Af = (const float*)p.A;

  uint4 ra0, ra1, ra2, ra3, rb0, rb1, rb2, rb3;
  float4 rf0a, rf0b, rf1a, rf1b, rf2a, rf2b, rf3a, rf3b;
  const uint4 z4 = make_uint4(0, 0, 0, 0);
  const float4 zf = make_float4(0.f, 0.f, 0.f, 0.f);

// Loads are unconditional from clamped, in-bounds addresses (row 0, column
// 0 for masked lanes); masking selects the loaded value, never the address.
// The four staged rows are written out explicitly so every staging register
// has a fixed name (no dynamically indexed arrays).
#define LX_LD1(i)                                                                 \
  do {                                                                            \
    const bool av = kin && ((amask >> i) & 1u);                                   \
    if (HILO) {                                                                   \
      const float4* q = (const float4*)(Af + aoff[i] + kcl);                      \
      const float4 v0 = q[0], v1 = q[1];                                          \
      rf##i##a = av ? v0 : zf;                                                    \
      rf##i##b = av ? v1 : zf;                                                    \
    } else {                                                                      \
      const uint4 v = *(const uint4*)(Ab + aoff[i] + kcl);                        \
      ra##i = av ? v : z4;                                                        \
    }                                                                             \
    const uint4 w = *(const uint4*)(Bw + boff[i] + kcl);                          \
    rb##i = (kin && ((bmask >> i) & 1u)) ? w : z4;                                \
  } while (0)
#define LX_GLOAD(K0)                                                              \
  do {                                                                            \
    const int kk = (K0) + lkc * 8;                                                \
    const bool kin = kk < K;                                                      \
    const int kcl = kin ? kk : 0;                                                 \
    LX_LD1(0);                                                                    \
    LX_LD1(1);                                                                    \
    LX_LD1(2);                                                                    \
    LX_LD1(3);                                                                    \
  } while (0)
#define LX_ST1(BUF, i)                                                            \
  do {                                                                            \
    const int off = lds_off(lrow + 32 * i, lkc);                                  \
    if (HILO) {                                                                   \
      uint4 hi, lo;                                                               \
      split_hilo(rf##i##a, rf##i##b, hi, lo);                                     \
      *(uint4*)&sA[BUF][off] = hi;                                                \
      *(uint4*)&sAl[BUF][off] = lo;                                               \
    } else {                                                                      \
      *(uint4*)&sA[BUF][off] = ra##i;                                             \
    }                                                                             \
    *(uint4*)&sB[BUF][off] = rb##i;                                               \
  } while (0)
#define LX_SSTORE(BUF)                                                            \
  do {                                                                            \
    LX_ST1(BUF, 0);                                                               \
    LX_ST1(BUF, 1);                                                               \
    LX_ST1(BUF, 2);                                                               \
    LX_ST1(BUF, 3);                                                               \
  } while (0)

  f32x16 acc[2][2];
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[mi][ni][i] = 0.f;

  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave >> 1, wn = wave & 1;
  const int nk = (K + BK - 1) / BK;

  LX_GLOAD(0);
  LX_SSTORE(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) LX_GLOAD((kt + 1) * BK);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int kc = ks * 2 + (lane >> 5);
      bf16x8 af[2], al[2], bw[2];
#pragma unroll
      for (int mi = 0; mi < 2; ++mi) {
        const int off = lds_off(wm * 64 + mi * 32 + (lane & 31), kc);
        af[mi] = *(const bf16x8*)&sA[cur][off];
        if (HILO) al[mi] = *(const bf16x8*)&sAl[cur][off];
      }
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
        bw[ni] = *(const bf16x8*)&sB[cur][lds_off(wn * 64 + ni * 32 + (lane & 31), kc)];
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) {
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mi], bw[ni], acc[mi][ni], 0, 0, 0);
          if (HILO)
            acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al[mi], bw[ni], acc[mi][ni], 0, 0, 0);
        }
    }
    if (kt + 1 < nk) LX_SSTORE(cur ^ 1);
    __syncthreads();
  }

#undef LX_LD1
#undef LX_GLOAD
#undef LX_ST1
#undef LX_SSTORE

  // 32x32 accumulator layout: lane holds column (lane & 31) and rows
  // 8*(i/4) + 4*(lane/32) + (i%4) for i = 0..15.
  float* __restrict__ C = p.C + p.c_coloff[part] + n0;
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
      const int c = wn * 64 + ni * 32 + (lane & 31);
      if (n0 + c >= ncol) continue;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int r = wm * 64 + mi * 32 + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
        if (r < te.nrows) C[(int64_t)(te.row0 + r) * p.ldc + c] = acc[mi][ni][i];
      }
    }
}

// ------------------------------------------------------------------ fp32 path
constexpr int FBM = 64, FBN = 64, FBK = 16;
static_assert((FBM & (FBM - 1)) == 0, "tile heights are powers of two (bucketing shifts)");

__global__ __launch_bounds__(256) void k_gemm_f32(GemmArgs p) {
  if ((int)blockIdx.x >= *p.n_tiles) return;
  const TileEntry te = p.tiles[blockIdx.x];
  const int ntp0 = (p.ncols[0] + FBN - 1) / FBN;
  const int part = (int)blockIdx.y < ntp0 ? 0 : 1;
  const int n0 = ((int)blockIdx.y - (part ? ntp0 : 0)) * FBN;
  const int ncol = p.ncols[part];
  const int K = p.K;
  const float* __restrict__ Bw = (const float*)p.B[part] + (int64_t)te.widx * p.b_stride[part];
  const float* __restrict__ Af = (const float*)p.A;

  __shared__ float sA[FBK][FBM + 4];
  __shared__ float sB[FBK][FBN + 4];
  const int tid = threadIdx.x;
  const int ty = tid >> 4, tx = tid & 15;
  const int lk = tid & 15, lr = tid >> 4;  // loader: row lr + 16*e, column lk

  const float* arow[4];
  const float* brow[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int r = lr + 16 * e;
    if (r < te.nrows) {
      const int64_t src = p.a_rows ? (int64_t)p.a_rows[te.row0 + r] : (int64_t)(te.row0 + r);
      arow[e] = Af + src * p.lda + p.a_koff[part];
    } else {
      arow[e] = nullptr;
    }
    brow[e] = (n0 + r < ncol) ? Bw + (int64_t)(n0 + r) * K : nullptr;
  }

  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;

  for (int k0 = 0; k0 < K; k0 += FBK) {
    const int kk = k0 + lk;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = lr + 16 * e;
      sA[lk][r] = (arow[e] && kk < K) ? arow[e][kk] : 0.f;
      sB[lk][r] = (brow[e] && kk < K) ? brow[e][kk] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < FBK; ++q) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = sA[q][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = sB[q][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
  float* __restrict__ C = p.C + p.c_coloff[part] + n0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = ty * 4 + i;
    if (r >= te.nrows) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = tx * 4 + j;
      if (n0 + c < ncol) C[(int64_t)(te.row0 + r) * p.ldc + c] = acc[i][j];
    }
  }
}

}  // namespace

int gemm_bm(lx_dtype dt) { return dt == LX_BF16 ? BM : FBM; }
int gemm_bn(lx_dtype dt) { return dt == LX_BF16 ? BN : FBN; }

hipError_t launch_gemm(const GemmArgs& g, lx_dtype dt, AMode am, int grid_x, hipStream_t s) {
  const int bn = gemm_bn(dt);
  const int gy = (g.ncols[0] + bn - 1) / bn + (g.ncols[1] + bn - 1) / bn;
  if (grid_x <= 0 || gy <= 0) return hipSuccess;
  const dim3 grid(grid_x, gy);
  if (dt == LX_F32) {
    hipLaunchKernelGGL(k_gemm_f32, grid, dim3(256), 0, s, g);
  } else if (am == A_BF16) {
    hipLaunchKernelGGL(k_gemm_bf16<A_BF16>, grid, dim3(NTHR), 0, s, g);
  } else {
    hipLaunchKernelGGL(k_gemm_bf16<A_F32_HILO>, grid, dim3(NTHR), 0, s, g);
  }
  return hipGetLastError();
}

}  // namespace lx

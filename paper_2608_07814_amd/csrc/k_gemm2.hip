// Large-tile grouped GEMM for gfx950: C = A * W^T over the rows of one tree
// level, for operands whose K is a multiple of 64 and whose A is bf16.
//
//   * 256 x BN output tile (BN = 256 or 128) per 256-thread workgroup; each of
//     the 4 wavefronts owns 128 x BN/2 (4 x BN/64 MFMA 32x32x16 blocks, the
//     accumulators live in AGPRs);
//   * both operands go HBM -> LDS with global_load_lds_dwordx4 (16 B per lane,
//     no staging registers); a 2-stage LDS ring lets the next K-slab stream in
//     while the current one feeds the MFMAs;
//   * the LDS image is the same XOR-swizzled 128-byte-row layout as the
//     register-staged kernel: since a direct load writes lane-contiguous LDS,
//     each lane picks the global chunk that belongs at its LDS slot;
//   * rows past the tile's end and weight rows past N are clamped to valid
//     addresses (their results are never stored), so every load is in bounds;
//   * XCD-aware order: workgroups are dispatched round-robin over the 8 XCDs;
//     the kernel renumbers them so each XCD receives a contiguous range of
//     (tile, n-tile) work, i.e. neighbours that share A rows and weight slabs
//     share one L2.
#include "lx_internal.h"

namespace lx {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint16_t u16;
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) const void gbl_void_t;

constexpr int BM2 = 256, BK2 = 64, NTHR2 = 256, NXCD = 8;

__device__ __forceinline__ int swz2(int row) { return (row ^ (row >> 3)) & 7; }
__device__ __forceinline__ int lds_off2(int row, int kc) { return row * BK2 + ((kc ^ swz2(row)) << 3); }

// One 16-byte direct HBM -> LDS load per lane: lane i writes LDS bytes
// [lds_base + 16 i, lds_base + 16 i + 16). lds_base must be wave-uniform. The
// load is issued through inline asm so that the only waits on it are the
// explicit per-stage vmcnt waits below (the compiler's own tracking of LDS
// DMA would otherwise serialize consecutive loads). M0 is written here only;
// nothing else in these kernels uses it.
__device__ __forceinline__ void load_lds16(const void* gptr, const void* lds_dst) {
  const uint32_t lds = (uint32_t)(uintptr_t)(lds_void_t*)lds_dst;
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(gptr), "s"(__builtin_amdgcn_readfirstlane(lds))
               : "memory");
}

// s_waitcnt with only the vector-memory counter constrained to <= n (n < 64).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

template <int BN>
__global__ __launch_bounds__(NTHR2, 1) void k_gemm_big(GemmArgs p, int ntn) {
  constexpr int WN = BN / 2;              // columns per wavefront
  constexpr int NI = WN / 32;             // MFMA blocks along N per wavefront
  constexpr int A_ROUNDS = BM2 * 8 / NTHR2;  // 16-byte chunks per thread for A (8)
  constexpr int B_ROUNDS = BN * 8 / NTHR2;   // ... for B (8 or 4)

  // ---- which (tile, n-tile) this workgroup computes (XCD-contiguous order)
  const int real = *p.n_tiles * ntn;
  const int P = blockIdx.x;
  if (P >= real) return;
  const int q = real / NXCD, rmd = real % NXCD;
  const int x = P % NXCD, idx = P / NXCD;
  const int Lg = x * q + (x < rmd ? x : rmd) + idx;
  const int ti = Lg / ntn, nt = Lg % ntn;

  // The two weight parts form one column range [0, ncol): column n < ncols[0]
  // is row n of part 0, otherwise row n - ncols[0] of part 1.
  const TileEntry te = p.tiles[ti];
  const int n0 = nt * BN;
  const int ncol = p.ncols[0] + p.ncols[1];
  const int K = p.K;
  const int Kb = p.Kb > 0 ? p.Kb : K;
  const int akoff = p.a_koff[0];
  const u16* __restrict__ Bw0 = (const u16*)p.B[0] + (int64_t)te.widx * p.b_stride[0];
  const u16* __restrict__ Bw1 = (const u16*)p.B[1] + (int64_t)te.widx * p.b_stride[1];
  const u16* __restrict__ Ab = (const u16*)p.A;

  __shared__ __attribute__((aligned(1024))) u16 sA0[BM2 * BK2];
  __shared__ __attribute__((aligned(1024))) u16 sA1[BM2 * BK2];
  __shared__ __attribute__((aligned(1024))) u16 sB0[BN * BK2];
  __shared__ __attribute__((aligned(1024))) u16 sB1[BN * BK2];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;

  // Per-thread source offsets (elements, chunk offset folded in) for each
  // 16-byte chunk it loads. LDS slot P = round*256 + tid holds row P>>3,
  // physical chunk P&7, i.e. logical chunk (P&7) ^ swz(row). 32-bit offsets:
  // the host routes operands whose element counts reach 2^31 elsewhere.
  uint32_t aoff[A_ROUNDS];
#pragma unroll
  for (int j = 0; j < A_ROUNDS; ++j) {
    const int Ps = j * NTHR2 + tid;
    const int row = Ps >> 3;
    const int c = (Ps & 7) ^ swz2(row);
    const int r = row < te.nrows ? row : te.nrows - 1;
    const int src = p.a_rows ? p.a_rows[te.row0 + r] : te.row0 + r;
    aoff[j] = (uint32_t)src * (uint32_t)p.lda + (uint32_t)(akoff + c * 8);
  }
  const u16* bptr[B_ROUNDS];
#pragma unroll
  for (int j = 0; j < B_ROUNDS; ++j) {
    const int Ps = j * NTHR2 + tid;
    const int row = Ps >> 3;
    const int c = (Ps & 7) ^ swz2(row);
    const int n = n0 + row < ncol ? n0 + row : ncol - 1;
    bptr[j] = (n < p.ncols[0] ? Bw0 + (int64_t)n * Kb : Bw1 + (int64_t)(n - p.ncols[0]) * Kb) + c * 8;
  }

#define LX_ISSUE(SA, SB, K0)                                                        \
  do {                                                                              \
    const int kb_ = (K0) % Kb;                                                      \
    _Pragma("unroll") for (int j = 0; j < A_ROUNDS; ++j)                            \
        load_lds16(Ab + (aoff[j] + (uint32_t)(K0)), &SA[(j * NTHR2 + wave * 64) * 8]); \
    _Pragma("unroll") for (int j = 0; j < B_ROUNDS; ++j)                            \
        load_lds16(bptr[j] + kb_, &SB[(j * NTHR2 + wave * 64) * 8]);                \
  } while (0)

  f32x16 acc[4][NI];
#pragma unroll
  for (int mi = 0; mi < 4; ++mi)
#pragma unroll
    for (int ni = 0; ni < NI; ++ni)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[mi][ni][i] = 0.f;

  const int wm = wave >> 1, wn = wave & 1;
  const int nk = K / BK2;

  // One K-slab of MFMAs from stage (SA, SB).
#define LX_COMPUTE(SA, SB)                                                          \
  do {                                                                              \
    _Pragma("unroll") for (int ks = 0; ks < BK2 / 16; ++ks) {                       \
      const int kc = ks * 2 + (lane >> 5);                                          \
      bf16x8 af[4], bw[NI];                                                         \
      _Pragma("unroll") for (int mi = 0; mi < 4; ++mi)                              \
        af[mi] = *(const bf16x8*)&SA[lds_off2(wm * 128 + mi * 32 + (lane & 31), kc)]; \
      _Pragma("unroll") for (int ni = 0; ni < NI; ++ni)                             \
        bw[ni] = *(const bf16x8*)&SB[lds_off2(wn * WN + ni * 32 + (lane & 31), kc)]; \
      _Pragma("unroll") for (int mi = 0; mi < 4; ++mi)                              \
        _Pragma("unroll") for (int ni = 0; ni < NI; ++ni)                           \
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mi], bw[ni], acc[mi][ni], 0, 0, 0); \
    }                                                                               \
  } while (0)
  // Barrier without a memory fence: the fence of __syncthreads() would drain
  // the next slab's in-flight loads. Each wavefront first waits for its own
  // loads of the slab (vmcnt), so after the barrier the whole slab is in LDS.
  // The empty asm keeps the compiler from moving LDS accesses across it.
  auto barrier = []() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  LX_ISSUE(sA0, sB0, 0);
  if (nk > 1) LX_ISSUE(sA1, sB1, BK2);
  int kt = 0;
  // Slabs kt (stage 0) and kt + 1 (stage 1) are in flight at the top of
  // every iteration; one loop exit keeps the accumulators in place.
  for (; kt + 1 < nk; kt += 2) {
    wait_vmcnt<A_ROUNDS + B_ROUNDS>();
    barrier();
    LX_COMPUTE(sA0, sB0);
    barrier();
    const bool more0 = kt + 2 < nk;
    if (more0) LX_ISSUE(sA0, sB0, (kt + 2) * BK2);
    if (more0)
      wait_vmcnt<A_ROUNDS + B_ROUNDS>();
    else
      wait_vmcnt<0>();
    barrier();
    LX_COMPUTE(sA1, sB1);
    barrier();
    if (kt + 3 < nk) LX_ISSUE(sA1, sB1, (kt + 3) * BK2);
  }
  if (kt < nk) {  // odd slab count: the last slab is in stage 0
    wait_vmcnt<0>();
    barrier();
    LX_COMPUTE(sA0, sB0);
  }

#undef LX_ISSUE
#undef LX_COMPUTE

  float* __restrict__ C = p.C + n0;
#pragma unroll
  for (int mi = 0; mi < 4; ++mi)
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) {
      const int c = wn * WN + ni * 32 + (lane & 31);
      if (n0 + c >= ncol) continue;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int r = wm * 128 + mi * 32 + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
        if (r < te.nrows) C[(int64_t)(te.row0 + r) * p.ldc + c] = acc[mi][ni][i];
      }
    }
}

}  // namespace

int gemm_big_bm() { return BM2; }

bool gemm_big_ok(const GemmArgs& g, int64_t a_rows_total) {
  const int Kb = g.Kb > 0 ? g.Kb : g.K;
  if (g.K <= 0 || g.K % BK2 || Kb % BK2 || g.K % Kb) return false;
  if (g.ncols[1] > 0 && (g.a_koff[0] != g.a_koff[1] || g.c_coloff[1] != g.ncols[0])) return false;
  if (g.c_coloff[0] != 0) return false;
  return a_rows_total * g.lda < ((int64_t)1 << 31);
}

hipError_t launch_gemm_big(const GemmArgs& g, int bn, int grid_tiles, hipStream_t s) {
  const int ntn = (g.ncols[0] + g.ncols[1] + bn - 1) / bn;
  const int grid = grid_tiles * ntn;
  if (grid <= 0) return hipSuccess;
  if (bn == 256)
    hipLaunchKernelGGL(k_gemm_big<256>, dim3(grid), dim3(NTHR2), 0, s, g, ntn);
  else
    hipLaunchKernelGGL(k_gemm_big<128>, dim3(grid), dim3(NTHR2), 0, s, g, ntn);
  return hipGetLastError();
}

}  // namespace lx

// Large-tile grouped GEMM for gfx950: C = A * W^T over the rows of one tree
// level, for bf16 A whose K is a multiple of 64.
//
//   * BM x BN output tile (BM = 128 or 256, BN = 64, 128 or 256) per
//     256-thread workgroup; the 4 wavefronts form a 2 x 2 grid, each owning
//     (BM/2) x (BN/2) as MFMA 32x32x16 blocks (accumulators in AGPRs);
//   * both operands go HBM -> LDS with global_load_lds_dwordx4 (16 B per lane,
//     no staging registers) into a 2-stage LDS ring, so the next K-slab
//     streams in while the current one feeds the MFMAs; inside a slab the
//     fragments of k-step s+1 are read from LDS while the MFMAs of step s run;
//   * the LDS image uses 128-byte rows with the 16-byte chunk index XOR-
//     swizzled by the row (no bank conflicts on fragment reads); since a direct
//     load writes lane-contiguous LDS, each lane fetches the global chunk that
//     belongs at its LDS slot;
//   * rows past the tile's end and weight rows past N are clamped to valid
//     addresses (their results are never stored), so every load is in bounds;
//   * the two weight parts (e.g. gate and up) form one column range; when a
//     tile lies inside one part, that part's A column offset is used, so the
//     parts may read different A columns;
//   * K may be a multiple of the weights' row length Kb: A = [A_hi | A_lo]
//     against the same W, i.e. C = (A_hi + A_lo) W^T, which keeps ~16 bits of
//     an fp32 intermediate at bf16 MFMA rate;
//   * output either fp32, or a bf16 (hi, lo) pair ready to feed the next GEMM
//     as its two K-halves;
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

constexpr int BK2 = 64, NTHR2 = 256, NXCD = 8;

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

// s_waitcnt with only the vector-memory counter constrained to <= N.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Barrier without a memory fence: the fence of __syncthreads() would drain
// the next slab's in-flight loads. Each wavefront first waits for its own
// loads of the slab (vmcnt), so after the barrier the whole slab is in LDS.
// The empty asm keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void bar() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <int BM, int BN, bool OUT_HILO>
__global__ __launch_bounds__(NTHR2, 1) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_gemm_big(GemmArgs p, int ntn) {
  constexpr int MI = BM / 64;              // 32-row MFMA blocks per wavefront
  constexpr int NI = BN / 64;              // 32-column MFMA blocks per wavefront
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int A_ROUNDS = BM * 8 / NTHR2;  // 16-byte chunks per thread per slab
  constexpr int B_ROUNDS = BN * 8 / NTHR2;
  constexpr int ROUNDS = A_ROUNDS + B_ROUNDS;

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
  const int tpart = n0 < p.ncols[0] ? 0 : 1;
  const int akoff = p.a_koff[tpart];
  const u16* __restrict__ Bw0 = (const u16*)p.B[0] + (int64_t)te.widx * p.b_stride[0];
  const u16* __restrict__ Bw1 = (const u16*)p.B[1] + (int64_t)te.widx * p.b_stride[1];
  const u16* __restrict__ Ab = (const u16*)p.A;

  __shared__ __attribute__((aligned(1024))) u16 sA0[BM * BK2];
  __shared__ __attribute__((aligned(1024))) u16 sA1[BM * BK2];
  __shared__ __attribute__((aligned(1024))) u16 sB0[BN * BK2];
  __shared__ __attribute__((aligned(1024))) u16 sB1[BN * BK2];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;

  // Per-thread source offsets (elements, chunk offset folded in) for each
  // 16-byte chunk it loads. LDS slot P = round*256 + tid holds row P>>3,
  // physical chunk P&7, i.e. logical chunk (P&7) ^ swz(row). 32-bit A
  // offsets: the host routes A operands with 2^31 or more elements elsewhere.
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

  f32x16 acc[MI][NI];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int ni = 0; ni < NI; ++ni)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[mi][ni][i] = 0.f;

  const int wm = wave >> 1, wn = wave & 1;
  const int nk = K / BK2;

  // One K-slab of MFMAs from stage (SA, SB), fragments double-buffered in
  // registers: the LDS reads of k-step s+1 are issued before the MFMAs of
  // step s (pinned by scheduling fences).
  bf16x8 fa0[MI], fb0[NI], fa1[MI], fb1[NI];
#define LX_FRAG(SA, SB, KS, FA, FB)                                                 \
  do {                                                                              \
    const int kc_ = (KS) * 2 + (lane >> 5);                                         \
    _Pragma("unroll") for (int mi = 0; mi < MI; ++mi)                               \
      FA[mi] = *(const bf16x8*)&SA[lds_off2(wm * WM + mi * 32 + (lane & 31), kc_)]; \
    _Pragma("unroll") for (int ni = 0; ni < NI; ++ni)                               \
      FB[ni] = *(const bf16x8*)&SB[lds_off2(wn * WN + ni * 32 + (lane & 31), kc_)]; \
  } while (0)
#define LX_MFMAS(FA, FB)                                                            \
  do {                                                                              \
    _Pragma("unroll") for (int mi = 0; mi < MI; ++mi)                               \
      _Pragma("unroll") for (int ni = 0; ni < NI; ++ni)                             \
        acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(FA[mi], FB[ni], acc[mi][ni], 0, 0, 0); \
  } while (0)
#define LX_COMPUTE(SA, SB)                                                          \
  do {                                                                              \
    LX_FRAG(SA, SB, 0, fa0, fb0);                                                   \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_FRAG(SA, SB, 1, fa1, fb1);                                                   \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_MFMAS(fa0, fb0);                                                             \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_FRAG(SA, SB, 2, fa0, fb0);                                                   \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_MFMAS(fa1, fb1);                                                             \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_FRAG(SA, SB, 3, fa1, fb1);                                                   \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_MFMAS(fa0, fb0);                                                             \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_MFMAS(fa1, fb1);                                                             \
  } while (0)

  LX_ISSUE(sA0, sB0, 0);
  if (nk > 1) LX_ISSUE(sA1, sB1, BK2);
  int kt = 0;
  // Slabs kt (stage 0) and kt + 1 (stage 1) are in flight at the top of
  // every iteration; one loop exit keeps the accumulators in place.
  for (; kt + 1 < nk; kt += 2) {
    wait_vmcnt<ROUNDS>();
    bar();
    LX_COMPUTE(sA0, sB0);
    bar();
    const bool more0 = kt + 2 < nk;
    if (more0) LX_ISSUE(sA0, sB0, (kt + 2) * BK2);
    if (more0)
      wait_vmcnt<ROUNDS>();
    else
      wait_vmcnt<0>();
    bar();
    LX_COMPUTE(sA1, sB1);
    bar();
    if (kt + 3 < nk) LX_ISSUE(sA1, sB1, (kt + 3) * BK2);
  }
  if (kt < nk) {  // odd slab count: the last slab is in stage 0
    wait_vmcnt<0>();
    bar();
    LX_COMPUTE(sA0, sB0);
  }
#undef LX_ISSUE
#undef LX_COMPUTE
#undef LX_FRAG
#undef LX_MFMAS

  // 32x32 accumulator layout: lane holds column (lane & 31) and rows
  // 8*(i/4) + 4*(lane/32) + (i%4) for i = 0..15.
#pragma unroll
  for (int ni = 0; ni < NI; ++ni) {
    const int col = n0 + wn * WN + ni * 32 + (lane & 31);
    if (col >= ncol) continue;
    if (OUT_HILO) {
      // part p, local column c -> hi at base_p + c, lo at base_p + ncols[p] + c
      const int pp = col < p.ncols[0] ? 0 : 1;
      const int c = pp ? col - p.ncols[0] : col;
      const int hi_col = (pp ? 2 * p.ncols[0] : 0) + c;
      const int lo_col = hi_col + p.ncols[pp];
      __bf16* __restrict__ C = (__bf16*)p.C;
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int r = wm * WM + mi * 32 + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
          if (r < te.nrows) {
            const float v = acc[mi][ni][i];
            const __bf16 h = (__bf16)v;
            __bf16* rowp = C + (int64_t)(te.row0 + r) * p.ldc;
            rowp[hi_col] = h;
            rowp[lo_col] = (__bf16)(v - (float)h);
          }
        }
    } else {
      float* __restrict__ C = p.C + col;
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int r = wm * WM + mi * 32 + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
          if (r < te.nrows) C[(int64_t)(te.row0 + r) * p.ldc] = acc[mi][ni][i];
        }
    }
  }
}

template <int BM, int BN>
hipError_t launch_bn(const GemmArgs& g, bool hilo, int grid, int ntn, hipStream_t s) {
  if (hilo)
    hipLaunchKernelGGL((k_gemm_big<BM, BN, true>), dim3(grid), dim3(NTHR2), 0, s, g, ntn);
  else
    hipLaunchKernelGGL((k_gemm_big<BM, BN, false>), dim3(grid), dim3(NTHR2), 0, s, g, ntn);
  return hipGetLastError();
}

}  // namespace

bool gemm_big_ok(const GemmArgs& g, int bn, int64_t a_rows_total) {
  const int Kb = g.Kb > 0 ? g.Kb : g.K;
  // every 64-wide K-slab must map to 64 consecutive weight columns of a row
  if (g.K <= 0 || g.K % BK2 || Kb % BK2 || g.K % Kb) return false;
  if (g.a_koff[0] + g.K > g.lda || (g.ncols[1] > 0 && g.a_koff[1] + g.K > g.lda)) return false;
  if (g.ncols[1] > 0 && g.a_koff[0] != g.a_koff[1] && g.ncols[0] % bn) return false;
  return a_rows_total * g.lda < ((int64_t)1 << 31);
}

hipError_t launch_gemm_big(const GemmArgs& g, int bm, int bn, bool out_hilo, int grid_tiles, hipStream_t s) {
  const int ntn = (g.ncols[0] + g.ncols[1] + bn - 1) / bn;
  const int grid = grid_tiles * ntn;
  if (grid <= 0) return hipSuccess;
  if (bm == 256) {
    if (bn == 256) return launch_bn<256, 256>(g, out_hilo, grid, ntn, s);
    if (bn == 128) return launch_bn<256, 128>(g, out_hilo, grid, ntn, s);
    return launch_bn<256, 64>(g, out_hilo, grid, ntn, s);
  }
  if (bn == 256) return launch_bn<128, 256>(g, out_hilo, grid, ntn, s);
  if (bn == 128) return launch_bn<128, 128>(g, out_hilo, grid, ntn, s);
  return launch_bn<128, 64>(g, out_hilo, grid, ntn, s);
}

}  // namespace lx

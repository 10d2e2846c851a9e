// Large-tile grouped GEMM for gfx950: C = A * W^T over the rows of one tree
// level, for bf16 A whose K is a multiple of 64.
//
//   * BM x BN output tile (BM = 128 or 256, BN = 64, 128 or 256); 256x256
//     tiles use 8 wavefronts (2 x 4 grid of 128x64 blocks, two per SIMD),
//     256x128 tiles 8 (4 x 2 grid of 64x64 blocks), the others 4 (2 x 2
//     grid), each block as MFMA 32x32x16 sub-blocks;
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
//   * output fp32, a bf16 (hi, lo) pair ready to feed the next GEMM as its
//     two K-halves, or x16 (rows read back only by the elementwise kernels);
//   * persistent: the grid is at most one workgroup per compute unit and each
//     workgroup loops over (tile, n-tile) work items, so the epilogue of one
//     item and the prologue loads of the next are not separated by a
//     workgroup launch;
//   * XCD-aware order: workgroups are dispatched round-robin over the 8 XCDs;
//     each XCD's workgroups take a contiguous range of work items, i.e.
//     neighbours that share A rows and weight slabs share one L2;
//   * epilogue through LDS: each wavefront transposes its accumulator block
//     so that every lane stores 4 consecutive columns of one row (16-byte
//     fp32 or 8-byte bf16 stores), 8 for x16 outputs (one 16-byte group).
#include "lx_internal.h"

#include <algorithm>
#include <mutex>
#include <type_traits>

namespace lx {
namespace {
int grid_cap();  // defined below

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint16_t u16;
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int BK2 = 64, NXCD = 8;

__device__ __forceinline__ int swz2(int row) { return (row ^ (row >> 3)) & 7; }
__device__ __forceinline__ int lds_off2(int row, int kc) { return row * BK2 + ((kc ^ swz2(row)) << 3); }
// Large-tile swizzle: rows r and r + 1 share a 256-byte bank window, so the
// 16 lanes a ds_read_b128 serves together (rows r..r+15, one chunk) land on
// 16 distinct 16-byte bank groups when the chunk is XORed with (row / 2) % 8.
// Every fragment row of a lane (row = 32 * i + (lane % 32) + a multiple of 64)
// has the same swizzle, so a lane's k-step offsets are shared by all its
// fragments and the row steps become immediate offsets.
__device__ __forceinline__ int swzb(int row) { return (row >> 1) & 7; }
__device__ __forceinline__ int lds_offb(int row, int kc) { return row * BK2 + ((kc ^ swzb(row)) << 3); }

// One 16-byte direct HBM -> LDS load per lane: lane i writes LDS bytes
// [lds_base + 16 i, lds_base + 16 i + 16). lds_base must be wave-uniform. The
// load is issued through inline asm so that the only waits on it are the
// explicit per-stage vmcnt waits below (the compiler's own tracking of LDS
// DMA would otherwise serialize consecutive loads). M0 is written here only;
// nothing else in these kernels uses it. The s_nop is the one wait state the
// GFX9 family requires between an SALU write of M0 and an LDS-DMA load.
__device__ __forceinline__ void load_lds16(const void* gptr, const void* lds_dst) {
  const uint32_t lds = (uint32_t)(uintptr_t)(lds_void_t*)lds_dst;
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(gptr), "s"(__builtin_amdgcn_readfirstlane(lds))
               : "memory");
}

// One 4-byte direct HBM -> LDS load per lane (lane i writes LDS bytes
// [lds_base + 4 i, lds_base + 4 i + 4)); same conventions as load_lds16.
__device__ __forceinline__ void load_lds4(const void* gptr, const void* lds_dst) {
  const uint32_t lds = (uint32_t)(uintptr_t)(lds_void_t*)lds_dst;
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
               :
               : "v"(gptr), "s"(__builtin_amdgcn_readfirstlane(lds))
               : "memory");
}

// The same loads addressed as a wave-uniform 64-bit base (SGPR pair) plus a
// 32-bit per-lane byte offset: one VGPR per address instead of two.
__device__ __forceinline__ void load_lds16_sb(const void* base, uint32_t off, const void* lds_dst) {
  const uint32_t lds = (uint32_t)(uintptr_t)(lds_void_t*)lds_dst;
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(off), "s"(base), "s"(__builtin_amdgcn_readfirstlane(lds))
               : "memory");
}
__device__ __forceinline__ void load_lds4_sb(const void* base, uint32_t off, const void* lds_dst) {
  const uint32_t lds = (uint32_t)(uintptr_t)(lds_void_t*)lds_dst;
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1"
               :
               : "v"(off), "s"(base), "s"(__builtin_amdgcn_readfirstlane(lds))
               : "memory");
}

typedef int v8i __attribute__((ext_vector_type(8)));

// s_waitcnt with only the vector-memory counter constrained to <= N.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// s_waitcnt with only the LDS/scalar-memory counter constrained to 0.
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xF | (0x7 << 4) | (0x3 << 14)); }

// Barrier without a memory fence: the fence of __syncthreads() would drain
// the next slab's in-flight loads. Each wavefront first waits for its own
// loads of the slab (vmcnt), so after the barrier the whole slab is in LDS.
// The empty asm keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void bar() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// s_waitcnt allowing `ahead` slabs of R loads each to stay in flight.
template <int R>
__device__ __forceinline__ void wait_slabs(int ahead) {
  if (ahead >= 3)
    wait_vmcnt<3 * R>();
  else if (ahead == 2)
    wait_vmcnt<2 * R>();
  else if (ahead == 1)
    wait_vmcnt<R>();
  else
    wait_vmcnt<0>();
}

// Wavefronts per workgroup: 8 for 256x256 tiles (two per SIMD in a 2x4 grid
// of 128x64 blocks, so one wavefront's LDS and barrier waits are covered by
// the other's MFMAs), else 4 (one per SIMD, a 2x2 grid).
template <int BM, int BN>
struct BigCfg {
  // 256 x 256 and 256 x 128 tiles: 8 wavefronts (two per SIMD), in a 2 x 4
  // grid of 128 x 64 blocks and a 4 x 2 grid of 64 x 64 blocks; the others 4
  // wavefronts in a 2 x 2 grid
  static constexpr int NW = (BM == 256 && (BN == 256 || BN == 128)) ? 8 : 4;
  static constexpr int WGN = (BM == 256 && BN == 256) ? 4 : 2;  // wavefronts along N
  static constexpr int WGM = NW / WGN;                          // wavefronts along M
  static constexpr int NTHR = NW * 64;
  static constexpr int WPE = NW / 4;  // wavefronts per SIMD
};

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

// One 32x32x16 MFMA on 16-bit operands: bf16, or fp16 (the same bits
// reinterpreted) for the fp16 anchor down projection.
template <bool F16>
__device__ __forceinline__ f32x16 mfma16(bf16x8 a, bf16x8 b, f32x16 c) {
  if constexpr (F16)
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                  0, 0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// F16: A and W are fp16, both scaled by powers of two (A row r by
// 2^a_row_exp[r], weight matrix i by 2^b_exp[i]); the epilogue multiplies
// each output row by 2^-(a_row_exp[row] + b_exp[widx]), an exact rescale.
// OUT2 >= 0: a second, independent product p2 in the same launch (same tile
// shape and operand precision; its own operands, tile table, columns and
// output format OUT2). Its work items follow p's in one persistent schedule,
// so the two products share one tail instead of ending in two.
template <int OUT>
struct OutC {
  static constexpr int value = OUT;
};

template <int BM, int BN, int OUT, bool LO8, bool F16, int OUT2>
__device__ __forceinline__ void gemm_big_body(const GemmArgs& p, int ntn, const GemmArgs& p2, int ntn2) {
  static_assert(!LO8 || (BM == 256 && BN == 256), "fp8 lo: 256 x 256 tiles");
  static_assert(!(LO8 && F16), "one precision mode at a time");
  constexpr int NTHR = BigCfg<BM, BN>::NTHR, WGN = BigCfg<BM, BN>::WGN;
  constexpr int WM = BM / BigCfg<BM, BN>::WGM, WN = BN / WGN;  // a wavefront's block
  constexpr int MI = WM / 32;              // 32-row MFMA blocks per wavefront
  constexpr int NI = WN / 32;              // 32-column MFMA blocks per wavefront
  constexpr int A_ROUNDS = BM * 8 / NTHR;  // 16-byte chunks per thread per slab
  constexpr int B_ROUNDS = BN * 8 / NTHR;
  constexpr int ROUNDS = A_ROUNDS + B_ROUNDS;
  // LDS: NST stages of [A | B] within 128 KB (2 for 256x256 tiles, up to 4
  // for the smaller ones, which stream more bytes per MFMA and need more
  // slabs in flight); the epilogue reuses it.
  constexpr int SA = BM * BK2, SB = BN * BK2;
  constexpr int NST_FIT = 65536 / (SA + SB);
  constexpr int NST = NST_FIT > 4 ? 4 : NST_FIT;
  static_assert(NST >= 2, "two stages must fit");
  __shared__ __attribute__((aligned(1024))) u16 smem[NST * (SA + SB)];
  // fp16 operands: the scale exponents of the tile's A rows (read by the
  // epilogue; loaded when the item starts)
  __shared__ int s_rexp[F16 ? BM : 1];
  // OUT_F16T: every wavefront's largest magnitude in the tile
  __shared__ float s_tmax[BigCfg<BM, BN>::NW];
  u16* const sA0 = smem;
  u16* const sB0 = smem + SA;
  u16* const sA1 = smem + SA + SB;
  u16* const sB1 = smem + 2 * SA + SB;

  // Work items (tile, n-tile) of each product: XCD x owns a contiguous range
  // of p's items and one of p2's (each product split evenly over the XCDs, the
  // remainders from opposite ends so that no XCD gets two extra items); its mx
  // workgroups take every mx-th item of [its p items, then its p2 items]. The
  // host launches either one workgroup per item or a multiple of 8
  // workgroups, so every XCD with items has at least one workgroup.
  const int n1 = *p.n_tiles * ntn;
  const int n2 = OUT2 >= 0 ? *p2.n_tiles * ntn2 : 0;
  const int x = blockIdx.x % NXCD;
  const int q1 = n1 / NXCD, r1 = n1 % NXCD;
  const int b1 = x * q1 + (x < r1 ? x : r1), c1 = q1 + (x < r1 ? 1 : 0);
  const int q2 = n2 / NXCD, r2 = n2 % NXCD, xr = NXCD - 1 - x;
  const int b2 = xr * q2 + (xr < r2 ? xr : r2), c2 = q2 + (xr < r2 ? 1 : 0);
  const int mx = ((int)gridDim.x - x + NXCD - 1) / NXCD;

  // One work item of product g (item Li of its own list, ntn_i column tiles
  // per row tile, output format decltype(oc)::value), inlined once per product
  // so that each copy reads its own arguments directly.
  auto item = [&](const GemmArgs& g, const int Li, const int ntn_i, auto oc) __attribute__((always_inline)) {
    constexpr int O = decltype(oc)::value;
    // The empty asm makes the lane index opaque per item, so the per-lane
    // address arithmetic below is recomputed each item instead of being
    // hoisted out of the item loop (where it would not fit in registers).
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int wave = tid >> 6, lane = tid & 63;
    const int wm = wave / WGN, wn = wave % WGN;
    // item -> (row tile, column tile): with more than 8 column tiles, in bands
    // of 8 (band-major), so the 32 workgroups of an XCD that run together
    // cover 4 row tiles x 8 column tiles and each weight slab is shared by 4
    int ti, nt;
    if (ntn_i > 8 && ntn_i % 8 == 0) {
      const int per_band = *g.n_tiles * 8;
      const int band = Li / per_band, rem = Li - band * per_band;
      ti = rem >> 3;
      nt = band * 8 + (rem & 7);
    } else {
      ti = Li / ntn_i;
      nt = Li % ntn_i;
    }
    const int ncol = g.ncols[0] + g.ncols[1];
    const int K = g.K;
    const int Kb = g.Kb > 0 ? g.Kb : K;
    const int nk = K / BK2;
    const u16* __restrict__ Ab = (const u16*)g.A;

    // The two weight parts form one column range [0, ncol): column n < ncols[0]
    // is row n of part 0, otherwise row n - ncols[0] of part 1.
    const TileEntry te = g.tiles[ti];
    // weight index: the tile's, or that of the tile node's ancestor at
    // another level (a leaf-row product with an upper level's weights)
    // (widx_own1: that lookup is part 0's only, part 1 takes the tile's own)
    int widx = te.widx;
    if (g.widx_anc) {
      const int an = g.widx_anc[te.node];
      widx = an >= 0 ? g.widx_fac[an] : -1;
    }
    int widx1 = g.widx_own1 ? te.widx : widx;
    // a leaf-level tile whose node (or ancestor) has no factor (it is listed
    // for the products that merge the levels above it): nothing to do here;
    // with two weight sources a missing one reads matrix 0 (its outputs are
    // never used)
    if (widx < 0 && widx1 < 0) return;
    if (widx < 0) widx = 0;
    if (widx1 < 0) widx1 = 0;
    const int n0 = nt * BN;
    const int tpart = n0 < g.ncols[0] ? 0 : 1;
    const int akoff = g.a_koff[tpart];
    if constexpr (F16) {
      for (int row = tid; row < BM; row += NTHR) s_rexp[row] = g.a_row_exp[te.row0 + (row < te.nrows ? row : te.nrows - 1)];
      asm volatile("" ::: "memory");
      wait_lgkm0();
    }
    const u16* __restrict__ Bw0 = (const u16*)g.B[0] + (int64_t)widx * g.b_stride[0];
    const u16* __restrict__ Bw1 = (const u16*)g.B[1] + (int64_t)widx1 * g.b_stride[1];

    // Per-thread source offsets (elements, chunk offset folded in) for each
    // 16-byte chunk it loads. LDS slot P = round*256 + tid holds row P>>3,
    // physical chunk P&7, i.e. logical chunk (P&7) ^ swz(row). 32-bit A
    // offsets: the host routes A operands with 2^31 or more elements elsewhere.
    uint32_t aoff[A_ROUNDS];
#pragma unroll
    for (int j = 0; j < A_ROUNDS; ++j) {
      const int Ps = j * NTHR + tid;
      const int row = Ps >> 3;
      const int c = (Ps & 7) ^ swzb(row);
      const int r = row < te.nrows ? row : te.nrows - 1;
      const int src = g.a_rows ? g.a_rows[te.row0 + r] : te.row0 + r;
      aoff[j] = (uint32_t)src * (uint32_t)g.lda + (uint32_t)(akoff + c * 8);
    }
    const u16* bptr[B_ROUNDS];
#pragma unroll
    for (int j = 0; j < B_ROUNDS; ++j) {
      const int Ps = j * NTHR + tid;
      const int row = Ps >> 3;
      const int c = (Ps & 7) ^ swzb(row);
      const int n = n0 + row < ncol ? n0 + row : ncol - 1;
      bptr[j] = (n < g.ncols[0] ? Bw0 + (int64_t)n * Kb : Bw1 + (int64_t)(n - g.ncols[0]) * Kb) + c * 8;
    }

    // Slab kt covers A columns [ka, ka + 64) and weight columns [kb, kb + 64)
    // with the K periods interleaved: slab kt = q * nper + per reads period
    // per of weight slab q, so the periods that reuse one weight slab (hi and
    // lo halves) run back to back and the second read hits in cache.
    const int nper = K / Kb;
    // A period Kb that is a multiple of 8 but not of 64 (ranks 32 and 96 on
    // their (hi | lo) operands): slabs in plain K order (A columns
    // [64 kt, 64 kt + 64)), each 8-column chunk of a slab taking its weight
    // columns modulo Kb, so a slab that crosses from the hi to the lo half
    // reads the end and then the start of the weight row.
    const bool wrap = (Kb % BK2) != 0;
#define LX_ISSUE(SA_, SB_, KT)                                                      \
  do {                                                                              \
    if (!wrap) {                                                                    \
      const int q_ = (KT) / nper, per_ = (KT) - q_ * nper;                          \
      const int kb_ = q_ * BK2, ka_ = per_ * Kb + kb_;                              \
      _Pragma("unroll") for (int j = 0; j < A_ROUNDS; ++j)                          \
          load_lds16(Ab + (aoff[j] + (uint32_t)ka_), &(SA_)[(j * NTHR + wave * 64) * 8]);  \
      _Pragma("unroll") for (int j = 0; j < B_ROUNDS; ++j)                          \
          load_lds16(bptr[j] + kb_, &(SB_)[(j * NTHR + wave * 64) * 8]);            \
    } else {                                                                        \
      const int ka_ = (KT) * BK2, k0_ = ka_ % Kb;                                   \
      _Pragma("unroll") for (int j = 0; j < A_ROUNDS; ++j)                          \
          load_lds16(Ab + (aoff[j] + (uint32_t)ka_), &(SA_)[(j * NTHR + wave * 64) * 8]);  \
      _Pragma("unroll") for (int j = 0; j < B_ROUNDS; ++j) {                        \
        const int ps_ = j * NTHR + tid, row_ = ps_ >> 3;                            \
        const int c8_ = (((ps_ & 7) ^ swzb(row_)) << 3);                            \
        const int w_ = k0_ + c8_ >= Kb ? k0_ - Kb : k0_;                            \
        load_lds16(bptr[j] + w_, &(SB_)[(j * NTHR + wave * 64) * 8]);               \
      }                                                                             \
    }                                                                               \
  } while (0)

    f32x16 acc[MI][NI];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int ni = 0; ni < NI; ++ni)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[mi][ni][i] = 0.f;

    // One K-slab of MFMAs from stage (SA_, SB_), fragments double-buffered in
    // registers: the LDS reads of k-step s+1 are issued before the MFMAs of
    // step s (pinned by scheduling fences).
    bf16x8 fa0[MI], fb0[NI], fa1[MI], fb1[NI];
#define LX_FRAG(SA_, SB_, KS, FA, FB)                                               \
  do {                                                                              \
    const int kc_ = (KS) * 2 + (lane >> 5);                                         \
    _Pragma("unroll") for (int mi = 0; mi < MI; ++mi)                               \
      FA[mi] = *(const bf16x8*)&(SA_)[lds_offb(wm * WM + mi * 32 + (lane & 31), kc_)]; \
    _Pragma("unroll") for (int ni = 0; ni < NI; ++ni)                               \
      FB[ni] = *(const bf16x8*)&(SB_)[lds_offb(wn * WN + ni * 32 + (lane & 31), kc_)]; \
  } while (0)
#define LX_MFMAS(FA, FB)                                                            \
  do {                                                                              \
    _Pragma("unroll") for (int mi = 0; mi < MI; ++mi)                               \
      _Pragma("unroll") for (int ni = 0; ni < NI; ++ni)                             \
        acc[mi][ni] = mfma16<F16>(FA[mi], FB[ni], acc[mi][ni]);                   \
  } while (0)
#define LX_COMPUTE(SA_, SB_)                                                        \
  do {                                                                              \
    LX_FRAG(SA_, SB_, 0, fa0, fb0);                                                 \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_FRAG(SA_, SB_, 1, fa1, fb1);                                                 \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_MFMAS(fa0, fb0);                                                             \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_FRAG(SA_, SB_, 2, fa0, fb0);                                                 \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_MFMAS(fa1, fb1);                                                             \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_FRAG(SA_, SB_, 3, fa1, fb1);                                                 \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_MFMAS(fa0, fb0);                                                             \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_MFMAS(fa1, fb1);                                                             \
  } while (0)

    if constexpr (NST > 2) {
      // Ring of NST stages, one barrier per slab: slab kt lives in stage
      // kt % NST; after the barrier that follows slab kt's compute every
      // wavefront is done with that stage and slab kt + NST goes there.
      const int npre = nk < NST ? nk : NST;
      for (int i = 0; i < npre; ++i) LX_ISSUE(smem + i * (SA + SB), smem + i * (SA + SB) + SA, i);
      wait_slabs<ROUNDS>(npre - 1);
      bar();
      for (int kt = 0; kt < nk; ++kt) {
        const int st = kt % NST;
        u16* const cA = smem + st * (SA + SB);
        u16* const cB = cA + SA;
        LX_COMPUTE(cA, cB);
        if (kt + 1 < nk) {
          const int last = kt + NST - 1 < nk - 1 ? kt + NST - 1 : nk - 1;
          wait_slabs<ROUNDS>(last - (kt + 1));
          bar();
          if (kt + NST < nk) LX_ISSUE(cA, cB, kt + NST);
        }
      }
      bar();
    } else if constexpr (LO8) {
      // K = 2 Kb: slab kt = 2 q + per is the hi (per 0) or lo (per 1) half of
      // weight slab q. Hi slabs always sit in stage 0 ([A | B] bf16, 64 KB),
      // lo slabs in stage 1: [A lo8 16 KB | B lo8 16 KB | A scale words 1 KB |
      // B scale words 1 KB]. A lo slab is 5 direct loads per lane (2 + 2
      // 16-byte rounds, one 4-byte scale load), a hi slab ROUNDS.
      constexpr int RLO = 5;
      uint8_t* const L1 = (uint8_t*)sA1;
      const uint8_t* const Abytes = (const uint8_t*)g.A;
      const uint32_t apitch = 2 * (uint32_t)g.lda;
      const uint8_t* const B8 = g.b8 + (int64_t)widx * g.b_stride[0];
      const uint32_t* const BS = g.bsc + (int64_t)widx * (g.b_stride[0] / 64);
      const u16* const Bhi = Bw0;
      // byte offsets (32 bit: the host routes operands of 2^31 or more
      // elements elsewhere) of this thread's hi-slab chunks of B and of its lo
      // and scale loads, slab 0
      uint32_t bhoff[B_ROUNDS];
#pragma unroll
      for (int j = 0; j < B_ROUNDS; ++j) bhoff[j] = (uint32_t)((bptr[j] - Bhi) * 2);
      uint32_t aloff[2], bloff[2];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int Ps = j * NTHR + tid;
        const int row = Ps >> 2;
        const int c = (Ps & 3) ^ ((row >> 2) & 3);
        const int r = row < te.nrows ? row : te.nrows - 1;
        aloff[j] = (uint32_t)(te.row0 + r) * apitch + (uint32_t)g.a_lo8_off + c * 16;
        const int n = n0 + row < ncol ? n0 + row : ncol - 1;
        bloff[j] = (uint32_t)n * (uint32_t)Kb + c * 16;
      }
      uint32_t scoff;
      {
        const int row = (wave & 3) * 64 + lane;
        if (wave < 4) {
          const int r = row < te.nrows ? row : te.nrows - 1;
          scoff = (uint32_t)(te.row0 + r) * apitch + (uint32_t)g.a_sc_off;
        } else {
          const int n = n0 + row < ncol ? n0 + row : ncol - 1;
          scoff = (uint32_t)n * (uint32_t)(Kb / BK2) * 4;
        }
      }
      auto issue_hi = [&](int kt) {
        const int kb = (kt >> 1) * BK2;
#pragma unroll
        for (int j = 0; j < A_ROUNDS; ++j)
          load_lds16(Ab + (aoff[j] + (uint32_t)kb), &sA0[(j * NTHR + wave * 64) * 8]);
#pragma unroll
        for (int j = 0; j < B_ROUNDS; ++j)
          load_lds16_sb(Bhi, bhoff[j] + (uint32_t)kb * 2, &sB0[(j * NTHR + wave * 64) * 8]);
      };
      auto issue_lo = [&](int kt) {
        const int q = kt >> 1, kb = q * BK2;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          load_lds16_sb(Abytes, aloff[j] + kb, L1 + (j * NTHR + wave * 64) * 16);
          load_lds16_sb(B8, bloff[j] + kb, L1 + 16384 + (j * NTHR + wave * 64) * 16);
        }
        if (wave < 4)
          load_lds4_sb(Abytes, scoff + q * 4, L1 + 32768 + wave * 256);
        else
          load_lds4_sb(BS, scoff + q * 4, L1 + 33792 + (wave - 4) * 256);
      };
      // lo fragments: lane (row, half h) holds K [16h, 16h + 16) of the slab in
      // bytes 0-15 and K [32 + 16h, 48 + 16h) in bytes 16-31 (scale block h);
      // rows are 64 bytes, 16-byte chunks XOR-swizzled by (row / 4) % 4
      auto compute_lo = [&]() {
        const int h = lane >> 5;
        v8i fb8[NI], fa8[2];
        int sb[NI], sa[2];
        auto lda8 = [&](int mi, int slot) {
          const int row = wm * WM + mi * 32 + (lane & 31);
          const int sw = (row >> 2) & 3;
          const uint4 x0 = *(const uint4*)(L1 + row * 64 + ((h ^ sw) << 4));
          const uint4 x1 = *(const uint4*)(L1 + row * 64 + (((2 + h) ^ sw) << 4));
          fa8[slot] = v8i{(int)x0.x, (int)x0.y, (int)x0.z, (int)x0.w, (int)x1.x, (int)x1.y, (int)x1.z, (int)x1.w};
          sa[slot] = (int)((*(const uint32_t*)(L1 + 32768 + row * 4) >> (8 * h)) & 0xFFu);
        };
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) {
          const int col = wn * WN + ni * 32 + (lane & 31);
          const int sw = (col >> 2) & 3;
          const uint4 x0 = *(const uint4*)(L1 + 16384 + col * 64 + ((h ^ sw) << 4));
          const uint4 x1 = *(const uint4*)(L1 + 16384 + col * 64 + (((2 + h) ^ sw) << 4));
          fb8[ni] = v8i{(int)x0.x, (int)x0.y, (int)x0.z, (int)x0.w, (int)x1.x, (int)x1.y, (int)x1.z, (int)x1.w};
          sb[ni] = (int)((*(const uint32_t*)(L1 + 33792 + col * 4) >> (8 * h)) & 0xFFu);
        }
        lda8(0, 0);
        // A fragments double-buffered: block mi + 1 is read while mi multiplies
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
          __builtin_amdgcn_sched_barrier(0);
          if (mi + 1 < MI) lda8(mi + 1, (mi + 1) & 1);
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int ni = 0; ni < NI; ++ni)
            acc[mi][ni] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fa8[mi & 1], fb8[ni], acc[mi][ni], 0, 0,
                                                                          0, sa[mi & 1], 0, sb[ni]);
        }
        __builtin_amdgcn_sched_barrier(0);
      };
      issue_hi(0);
      issue_lo(1);
      for (int kt = 0; kt < nk; kt += 2) {
        wait_vmcnt<RLO>();
        bar();
        LX_COMPUTE(sA0, sB0);
        bar();
        const bool more = kt + 2 < nk;
        if (more) issue_hi(kt + 2);
        if (more)
          wait_vmcnt<ROUNDS>();
        else
          wait_vmcnt<0>();
        bar();
        compute_lo();
        bar();
        if (more) issue_lo(kt + 3);
      }
    } else {
    LX_ISSUE(sA0, sB0, 0);
    if (nk > 1) LX_ISSUE(sA1, sB1, 1);
    int kt = 0;
    // Slabs kt (stage 0) and kt + 1 (stage 1) are in flight at the top of
    // every iteration; one loop exit keeps the accumulators in place.
    for (; kt + 1 < nk; kt += 2) {
      wait_vmcnt<ROUNDS>();
      bar();
      LX_COMPUTE(sA0, sB0);
      bar();
      const bool more0 = kt + 2 < nk;
      if (more0) LX_ISSUE(sA0, sB0, kt + 2);
      if (more0)
        wait_vmcnt<ROUNDS>();
      else
        wait_vmcnt<0>();
      bar();
      LX_COMPUTE(sA1, sB1);
      bar();
      if (kt + 3 < nk) LX_ISSUE(sA1, sB1, kt + 3);
    }
    if (kt < nk) {  // odd slab count: the last slab is in stage 0
      wait_vmcnt<0>();
      bar();
      LX_COMPUTE(sA0, sB0);
      bar();
    }
    }
#undef LX_ISSUE
#undef LX_COMPUTE
#undef LX_FRAG
#undef LX_MFMAS

    // Epilogue (output format O). 32x32 accumulator layout: lane holds column (lane & 31) and
    // rows 8*(i/4) + 4*(lane/32) + (i%4) for i = 0..15. Each wavefront writes
    // its 32 x WN block of one mi into its own LDS region (row pitch WN + 4
    // floats), then reads it back as 4 (x16: 8) consecutive columns per lane. All
    // stages are free here (every wavefront passed the barrier above).
    {
      constexpr int PITCH = WN + 4;
      constexpr int LPR = WN / 4;    // lanes per row
      constexpr int RPP = 64 / LPR;  // rows per pass
      static_assert(BigCfg<BM, BN>::NW * 32 * PITCH * 4 <= (int)sizeof(smem), "epilogue LDS");
      float* const ep = (float*)smem + wave * (32 * PITCH);
      const int c4 = (lane % LPR) * 4;
      const int col = n0 + wn * WN + c4;
      const int bexp = F16 ? (tpart ? (g.b_exp1 ? g.b_exp1 : g.b_exp)[widx1] : g.b_exp[widx]) : 0;
      // OUT_F16T: one power-of-two scale 2^tsh for the whole tile (its rows
      // are whole rows), from the largest magnitude over every wavefront's
      // block; with fp16 operands the accumulators already carry 2^(a_row_exp
      // + bexp), which the row exponents add
      int tsh = 0;
      if constexpr (O == OUT_F16T) {
        // fp16 operands, a tile over both parts: part 1's columns carry its
        // own weight scale; bring them to part 0's (exact) so that one row
        // exponent holds for the whole row
        if constexpr (F16) {
          if (tpart == 0 && n0 + BN > g.ncols[0] && g.ncols[1] > 0) {
            const int d1 = bexp - (g.b_exp1 ? g.b_exp1 : g.b_exp)[widx1];
#pragma unroll
            for (int ni = 0; ni < NI; ++ni) {
              const bool in1 = n0 + wn * WN + ni * 32 + (lane & 31) >= g.ncols[0];
#pragma unroll
              for (int mi = 0; mi < MI; ++mi)
#pragma unroll
                for (int i = 0; i < 16; ++i)
                  if (in1) acc[mi][ni][i] = ldexpf(acc[mi][ni][i], d1);
            }
          }
        }
        float m = 0.f;
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
#pragma unroll
          for (int ni = 0; ni < NI; ++ni)
#pragma unroll
            for (int i = 0; i < 16; ++i) m = fmaxf(m, fabsf(acc[mi][ni][i]));
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, 64));
        if (lane == 0) s_tmax[wave] = m;
        __syncthreads();
        float tm = 0.f;
#pragma unroll
        for (int w = 0; w < BigCfg<BM, BN>::NW; ++w) tm = fmaxf(tm, s_tmax[w]);
        if (tm > 0.f) {
          tsh = 14 - ((int)((__float_as_uint(tm) >> 23) & 0xFF) - 127);
          tsh = tsh < -100 ? -100 : tsh > 100 ? 100 : tsh;
        }
      }
      // x16 output: 8 consecutive columns per lane (one x16 group, one
      // 16-byte store per row)
      constexpr int LPR8 = WN / 8, RPP8 = 64 / LPR8;
      static_assert(WN % 8 == 0 && 32 % RPP8 == 0, "x16 epilogue layout");
      const int c8 = (lane % LPR8) * 8;
      const int col8 = n0 + wn * WN + c8;
      X16Rows8 xr8(g.C, g.ldc, te.row0 + wm * WM + lane / LPR8, RPP8, col8);
      // full tiles store without per-row checks (a separate, branch-free copy)
      auto emit = [&](auto check) {
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
          for (int ni = 0; ni < NI; ++ni)
#pragma unroll
            for (int i = 0; i < 16; ++i)
              ep[(8 * (i >> 2) + 4 * (lane >> 5) + (i & 3)) * PITCH + ni * 32 + (lane & 31)] = acc[mi][ni][i];
          if constexpr (O == OUT_X16) {
#pragma unroll
            for (int ps = 0; ps < 32 / RPP8; ++ps) {
              const int rr = ps * RPP8 + lane / LPR8;
              float4 va = *(const float4*)&ep[rr * PITCH + c8];
              float4 vb = *(const float4*)&ep[rr * PITCH + c8 + 4];
              const int r = wm * WM + mi * 32 + rr;
              const bool ok = !decltype(check)::value || (r < te.nrows && col8 < ncol);
              if constexpr (F16) {
                if (ok) {
                  const int e = -(s_rexp[r] + bexp);
                  va = make_float4(ldexpf(va.x, e), ldexpf(va.y, e), ldexpf(va.z, e), ldexpf(va.w, e));
                  vb = make_float4(ldexpf(vb.x, e), ldexpf(vb.y, e), ldexpf(vb.z, e), ldexpf(vb.w, e));
                }
              }
              if (ok) xr8.store(va, vb);
              xr8.next();
            }
            continue;
          }
#pragma unroll
          for (int ps = 0; ps < 32 / RPP; ++ps) {
            const int rr = ps * RPP + lane / LPR;
            float4 v = *(const float4*)&ep[rr * PITCH + c4];
            const int r = wm * WM + mi * 32 + rr;
            const bool ok = !decltype(check)::value || (r < te.nrows && col < ncol);
            if constexpr (F16 && O != OUT_F16T) {
              if (ok) {
                const int e = -(s_rexp[r] + bexp);
                v = make_float4(ldexpf(v.x, e), ldexpf(v.y, e), ldexpf(v.z, e), ldexpf(v.w, e));
              }
            }
            if constexpr (O == OUT_F16T) {
              if (!ok) continue;
              typedef _Float16 h4 __attribute__((ext_vector_type(4)));
              h4 q;
              q[0] = (_Float16)ldexpf(v.x, tsh);
              q[1] = (_Float16)ldexpf(v.y, tsh);
              q[2] = (_Float16)ldexpf(v.z, tsh);
              q[3] = (_Float16)ldexpf(v.w, tsh);
              *(h4*)((_Float16*)g.C + (int64_t)(te.row0 + r) * g.ldc + col) = q;
              if (wn == 0 && lane % LPR == 0)
                g.c_row_exp[te.row0 + r] = tsh + (F16 ? s_rexp[r] + bexp : 0);
            } else if constexpr (O == OUT_HILO) {
              if (!ok) continue;
              // part p, local column c -> hi at base_p + c, lo at base_p + ncols[p] + c
              const int pp = col < g.ncols[0] ? 0 : 1;
              const int c = pp ? col - g.ncols[0] : col;
              const int hi_col = (pp ? 2 * g.ncols[0] : 0) + c;
              const int lo_col = hi_col + g.ncols[pp];
              bf16x4 h, l;
              h[0] = (__bf16)v.x;
              h[1] = (__bf16)v.y;
              h[2] = (__bf16)v.z;
              h[3] = (__bf16)v.w;
              l[0] = (__bf16)(v.x - (float)h[0]);
              l[1] = (__bf16)(v.y - (float)h[1]);
              l[2] = (__bf16)(v.z - (float)h[2]);
              l[3] = (__bf16)(v.w - (float)h[3]);
              __bf16* const rowp = (__bf16*)g.C + (int64_t)(te.row0 + r) * g.ldc;
              *(bf16x4*)(rowp + hi_col) = h;
              *(bf16x4*)(rowp + lo_col) = l;
            } else {
              if (!ok) continue;
              *(float4*)(g.C + (int64_t)(te.row0 + r) * g.ldc + col) = v;
            }
          }
        }
      };
      if (te.nrows >= BM && n0 + BN <= ncol)
        emit(std::false_type{});
      else
        emit(std::true_type{});
    }
    bar();  // the next item's loads overwrite the epilogue's LDS
  };
  for (int j = (int)blockIdx.x / NXCD; j < c1 + c2; j += mx) {
    if constexpr (OUT2 >= 0) {
      if (j >= c1)
        item(p2, b2 + j - c1, ntn2, OutC<OUT2>{});
      else
        item(p, b1 + j, ntn, OutC<OUT>{});
    } else {
      item(p, b1 + j, ntn, OutC<OUT>{});
    }
  }
}

template <int BM, int BN, int OUT, bool LO8 = false, bool F16 = false>
__global__ __launch_bounds__((BigCfg<BM, BN>::NTHR), 1)
__attribute__((amdgpu_waves_per_eu(BigCfg<BM, BN>::WPE, BigCfg<BM, BN>::WPE)))
void k_gemm_big(GemmArgs p, int ntn) {
  gemm_big_body<BM, BN, OUT, LO8, F16, -1>(p, ntn, p, 0);
}

// Two products in one persistent launch (see gemm_big_body).
template <int BM, int BN, int OUT, int OUT2, bool F16>
__global__ __launch_bounds__((BigCfg<BM, BN>::NTHR), 1)
__attribute__((amdgpu_waves_per_eu(BigCfg<BM, BN>::WPE, BigCfg<BM, BN>::WPE)))
void k_gemm_big2(GemmArgs p, int ntn, GemmArgs p2, int ntn2) {
  gemm_big_body<BM, BN, OUT, false, F16, OUT2>(p, ntn, p2, ntn2);
}

// ---------------------------------------------------------------- segmented
// The correction products of several tree levels that land on the same rows
// (the leaf rows), as one 256 x 256-tile GEMM whose K runs over the levels'
// operands in turn (segments). Everything else is the 256 x 256 x16
// configuration of k_gemm_big: 8 wavefronts in a 2 x 4 grid of 128 x 64
// blocks, both operands HBM -> LDS by direct loads into a 2-stage ring of
// 64-wide K-slabs, persistent XCD-ordered work items, epilogue through LDS.
// bf16 (F16 false): within a segment of rank r the slabs alternate hi and
// lo halves of A against each 64-column weight slab (K = 2 r, the weight slab
// read twice back to back). fp16 (F16 true): one slab per 64 columns of the
// rank; A row a and weight matrix i of part p carry the scales 2^a_exp[a] and
// 2^b_exp[p][i], so segment s adds its products at scale 2^E_s(row) with
// E_s(row) = a_exp[map_s(row)] + b_exp[p][widx_s]; the accumulators are
// multiplied row by row by 2^(E_next - E_prev) when the segment changes and by
// 2^-E_last at the end (exact power-of-two steps). A segment's A rows come
// through its own row map (entries below 0 read the segment's zero row), its
// weights from its own level.
constexpr int kSegMax = LX_MAX_LEVELS;

template <bool F16>
__global__ __launch_bounds__(512, 1) __attribute__((amdgpu_waves_per_eu(2, 2)))
void k_gemm_seg(GemmArgs p, SegArgs sg, int ntn) {
  constexpr int BM = 256, BN = 256, NTHR = 512, WGN = 4;
  constexpr int MI = BM / 64, NI = BN / (32 * WGN), WM = BM / 2, WN = BN / WGN;
  constexpr int A_ROUNDS = BM * 8 / NTHR, B_ROUNDS = BN * 8 / NTHR, ROUNDS = A_ROUNDS + B_ROUNDS;
  constexpr int SA = BM * BK2, SB = BN * BK2;
  // epilogue: 8 consecutive columns per lane (LPR lanes per row, RPP rows per pass)
  constexpr int PITCH = WN + 4, LPR = WN / 8, RPP = 64 / LPR;
  static_assert(8 % RPP == 0, "epilogue rows");
  __shared__ __attribute__((aligned(1024))) u16 smem[2 * (SA + SB)];
  u16* const sA0 = smem;
  u16* const sB0 = smem + SA;
  u16* const sA1 = smem + SA + SB;
  u16* const sB1 = smem + 2 * SA + SB;
  // epilogue transposes, 8 rows at a time per wavefront, apart from the
  // stages: the next item's first two slabs load while this item's outputs
  // are stored
  __shared__ __attribute__((aligned(16))) float s_ep[8][8 * PITCH];
  // fp16 segments: scale exponent E_s of each tile row per segment, one
  // buffer per item parity (the next item's table is written while this
  // item's may still be read)
  __shared__ __attribute__((aligned(16))) int s_e[F16 ? 2 : 1][F16 ? kSegMax : 1][BM];

  // work item = (row tile, group of ngrp consecutive column tiles of one
  // part): the tile's setup (weight indices, row exponents) is done once per
  // group, then each column tile of the group runs its K loop and epilogue
  const int ngrp = sg.ngrp, nsg = ntn / ngrp;
  const int real = *p.n_tiles * nsg;
  const int q = real / NXCD, rmd = real % NXCD;
  const int x = blockIdx.x % NXCD;
  const int xbeg = x * q + (x < rmd ? x : rmd);
  const int xend = xbeg + q + (x < rmd ? 1 : 0);
  const int mx = ((int)gridDim.x - x + NXCD - 1) / NXCD;
  const int ncol = p.ncols[0] + p.ncols[1];
  const int nseg = sg.nseg;
  int Lg = xbeg + (int)blockIdx.x / NXCD;
  if (Lg >= xend) return;

  // the lane index is made opaque once per item (below), so per-lane address
  // arithmetic is recomputed per item instead of being kept live throughout
  int tid = threadIdx.x;

  // the item being loaded: its tile, n-tile, part, factor index and slab
  // count of every segment (0 for segments that do not apply)
  TileEntry te;
  int n0 = 0, tpart = 0, nk = 0, eb = 0;
  int widx[kSegMax], nsl[kSegMax];
  // operand addresses of the segment being issued (set at its first slab):
  // wave-uniform bases and 32-bit per-lane byte offsets
  int cur = -1, crank = 0;
  const u16* Ab = nullptr;
  const u16* Bb = nullptr;
  uint32_t aoff[A_ROUNDS], boff[B_ROUNDS];

  auto setup = [&](int L_) {
    const int ti = L_ / nsg, grp = L_ % nsg;
    te = p.tiles[ti];
    n0 = grp * ngrp * BN;
    tpart = n0 < p.ncols[0] ? 0 : 1;
    nk = 0;
    cur = -1;
#pragma unroll
    for (int sI = 0; sI < kSegMax; ++sI) {
      int w = -1;
      if (sI < nseg) {
        const SegDesc& dsc = sg.s[sI];
        if (dsc.anc_off < 0) {
          w = te.widx;
        } else {
          const int node = sg.anc[dsc.anc_off + te.node];
          w = node >= 0 ? dsc.fac[node] : -1;
        }
      }
      widx[sI] = w;
      nsl[sI] = w >= 0 ? (F16 ? 1 : 2) * sg.s[sI].rank / BK2 : 0;
      nk += nsl[sI];
    }
    if constexpr (F16) {
      // every row's exponent per active segment (visible to all wavefronts
      // after the K loop's first barrier, before any use)
#pragma unroll
      for (int sI = 0; sI < kSegMax; ++sI) {
        if (sI >= nseg || widx[sI] < 0) continue;
        const SegDesc& dsc = sg.s[sI];
        for (int row = tid; row < BM; row += NTHR) {
          const int r = row < te.nrows ? row : te.nrows - 1;
          const int src = dsc.map ? dsc.map[te.row0 + r] : te.row0 + r;
          s_e[eb][sI][row] = (src >= 0 ? dsc.a_exp[src] : 0) + dsc.b_exp[tpart][widx[sI]];
        }
      }
      asm volatile("" ::: "memory");
      wait_lgkm0();
    }
  };
  auto set_seg = [&](int sI) {
    const SegDesc& dsc = sg.s[sI];
    int w = 0;
#pragma unroll
    for (int u = 0; u < kSegMax; ++u)
      if (u == sI) w = widx[u];
    Ab = (const u16*)dsc.A;
    crank = dsc.rank;
    const int akoff = tpart ? dsc.akoff1 : 0;
#pragma unroll
    for (int j = 0; j < A_ROUNDS; ++j) {
      const int Ps = j * NTHR + tid;
      const int row = Ps >> 3;
      const int c = (Ps & 7) ^ swzb(row);
      const int r = row < te.nrows ? row : te.nrows - 1;
      int src = dsc.map ? dsc.map[te.row0 + r] : te.row0 + r;
      if (src < 0) src = dsc.zero_row;
      aoff[j] = ((uint32_t)src * (uint32_t)dsc.lda + (uint32_t)(dsc.a_col0 + akoff + c * 8)) * 2u;
    }
    // the tile lies inside one part: one weight matrix for all its rows
    Bb = (const u16*)dsc.B[tpart] + (int64_t)w * dsc.b_stride[tpart];
    const int nbase = tpart ? p.ncols[0] : 0;
    const int nlast = tpart ? ncol - 1 : p.ncols[0] - 1;
#pragma unroll
    for (int j = 0; j < B_ROUNDS; ++j) {
      const int Ps = j * NTHR + tid;
      const int row = Ps >> 3;
      const int c = (Ps & 7) ^ swzb(row);
      const int n = n0 + row < nlast ? n0 + row : nlast;
      boff[j] = ((uint32_t)(n - nbase) * (uint32_t)crank + (uint32_t)(c * 8)) * 2u;
    }
  };
  // segment of slab kt and the slab's index within it
  auto seg_of = [&](int kt, int& loc) {
    int sel = 0;
    loc = kt;
    bool found = false;
#pragma unroll
    for (int u = 0; u < kSegMax; ++u) {
      if (!found) {
        if (loc < nsl[u]) {
          sel = u;
          found = true;
        } else {
          loc -= nsl[u];
        }
      }
    }
    return sel;
  };
  // slab kt of the loaded item (slabs of a bf16 segment: weight slab qq, hi
  // then lo)
  auto issue = [&](u16* sA_, u16* sB_, int kt) {
    int loc;
    const int sel = seg_of(kt, loc);
    if (sel != cur) {
      set_seg(sel);
      cur = sel;
    }
    const int qq = F16 ? loc : loc >> 1, per = F16 ? 0 : loc & 1;
    const int kb = qq * BK2, ka = per * crank + kb;
#pragma unroll
    for (int j = 0; j < A_ROUNDS; ++j)
      load_lds16_sb(Ab, aoff[j] + (uint32_t)ka * 2u, &sA_[(j * NTHR + (tid >> 6) * 64) * 8]);
#pragma unroll
    for (int j = 0; j < B_ROUNDS; ++j)
      load_lds16_sb(Bb, boff[j] + (uint32_t)kb * 2u, &sB_[(j * NTHR + (tid >> 6) * 64) * 8]);
  };

  f32x16 acc[MI][NI];
  bf16x8 fa0[MI], fb0[NI], fa1[MI], fb1[NI];
#define LX_SFRAG(SA_, SB_, KS, FA, FB)                                              \
  do {                                                                              \
    const int kc_ = (KS) * 2 + (lane >> 5);                                         \
    _Pragma("unroll") for (int mi = 0; mi < MI; ++mi)                               \
      FA[mi] = *(const bf16x8*)&(SA_)[lds_offb(wm * WM + mi * 32 + (lane & 31), kc_)]; \
    _Pragma("unroll") for (int ni = 0; ni < NI; ++ni)                               \
      FB[ni] = *(const bf16x8*)&(SB_)[lds_offb(wn * WN + ni * 32 + (lane & 31), kc_)]; \
  } while (0)
#define LX_SMFMAS(FA, FB)                                                           \
  do {                                                                              \
    _Pragma("unroll") for (int mi = 0; mi < MI; ++mi)                               \
      _Pragma("unroll") for (int ni = 0; ni < NI; ++ni)                             \
        acc[mi][ni] = mfma16<F16>(FA[mi], FB[ni], acc[mi][ni]);                   \
  } while (0)
#define LX_SCOMPUTE(SA_, SB_)                                                       \
  do {                                                                              \
    LX_SFRAG(SA_, SB_, 0, fa0, fb0);                                                \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_SFRAG(SA_, SB_, 1, fa1, fb1);                                                \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_SMFMAS(fa0, fb0);                                                            \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_SFRAG(SA_, SB_, 2, fa0, fb0);                                                \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_SMFMAS(fa1, fb1);                                                            \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_SFRAG(SA_, SB_, 3, fa1, fb1);                                                \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_SMFMAS(fa0, fb0);                                                            \
    __builtin_amdgcn_sched_barrier(0);                                              \
    LX_SMFMAS(fa1, fb1);                                                            \
  } while (0)

  // fp16: accumulators from scale 2^E_from to 2^E_to row by row (to < 0:
  // the true scale), table buffer tb. Lane rows of block mi: 8 q + 4 (lane /
  // 32) + j for accumulator element 4 q + j.
  auto rescale = [&](int tb, int from, int to) {
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        const int rb = ((tid >> 6) / WGN) * WM + mi * 32 + 8 * qd + 4 * ((tid & 63) >> 5);
        const int4 ef = *(const int4*)&s_e[tb][from][rb];
        int4 et = make_int4(0, 0, 0, 0);
        if (to >= 0) et = *(const int4*)&s_e[tb][to][rb];
        const int dd[4] = {et.x - ef.x, et.y - ef.y, et.z - ef.z, et.w - ef.w};
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[mi][ni][4 * qd + j] = ldexpf(acc[mi][ni][4 * qd + j], dd[j]);
      }
  };

  // 2-stage ring: slab kt lives in stage kt & 1; one issue site and one
  // compute site per item (the segment switch inside issue() is then inlined
  // once). Slabs 0 and 1 of an item are issued before the previous item's
  // epilogue.
  setup(Lg);
  int gi = 0;  // column tile within the item's group
  for (int i = 0; i < 2 && i < nk; ++i) issue(i ? sA1 : sA0, i ? sB1 : sB0, i);
  while (true) {
    asm volatile("" : "+v"(tid));
    const int wave = tid >> 6, lane = tid & 63;
    const int wm = wave / WGN, wn = wave % WGN;
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int ni = 0; ni < NI; ++ni)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[mi][ni][i] = 0.f;
    int aseg = -1;  // segment whose scale the accumulators carry
    for (int kt = 0; kt < nk; ++kt) {
      u16* const cA = (kt & 1) ? sA1 : sA0;
      u16* const cB = (kt & 1) ? sB1 : sB0;
      if (kt + 1 < nk)
        wait_vmcnt<ROUNDS>();
      else
        wait_vmcnt<0>();
      bar();
      if constexpr (F16) {
        int loc;
        const int sel = seg_of(kt, loc);
        if (sel != aseg) {
          if (aseg >= 0) rescale(eb, aseg, sel);
          aseg = sel;
        }
      }
      LX_SCOMPUTE(cA, cB);
      bar();
      if (kt + 2 < nk) issue(cA, cB, kt + 2);
    }
    if constexpr (F16) {
      if (aseg >= 0) rescale(eb, aseg, -1);
    }

    // every wavefront is done with both stages: load the next column tile's
    // first slabs (the group's next one, or the next item's first), then
    // store this one's outputs
    const int row0 = te.row0, nrows = te.nrows, en0 = n0;
    int nLg = Lg, ngi = gi + 1;
    if (ngi == ngrp) {
      ngi = 0;
      nLg = Lg + mx;
    }
    const bool more = nLg < xend;
    if (more) {
      if (ngi == 0) {
        if constexpr (F16) eb ^= 1;
        setup(nLg);
      } else {
        n0 += BN;  // same rows, weights and exponents
        cur = -1;
      }
      for (int i = 0; i < 2 && i < nk; ++i) issue(i ? sA1 : sA0, i ? sB1 : sB0, i);
    }

    // Epilogue (as k_gemm_big's x16 output): per-wavefront LDS transpose of
    // 8 rows at a time, then 8 consecutive columns per lane.
    {
      float* const ep = s_ep[wave];
      const int c8 = (lane % LPR) * 8;
      const int col = en0 + wn * WN + c8;
      X16Rows8 xr(p.C, p.ldc, row0 + wm * WM + lane / LPR, RPP, col);
      // full tiles store without per-row checks (a separate, branch-free copy)
      auto emit = [&](auto check) {
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
#pragma unroll
          for (int qd = 0; qd < 4; ++qd) {
            // rows 8 qd .. 8 qd + 7 of block mi: elements 4 qd + j (row 4 (lane / 32) + j)
#pragma unroll
            for (int ni = 0; ni < NI; ++ni)
#pragma unroll
              for (int j = 0; j < 4; ++j)
                ep[(4 * (lane >> 5) + j) * PITCH + ni * 32 + (lane & 31)] = acc[mi][ni][4 * qd + j];
#pragma unroll
            for (int ps = 0; ps < 8 / RPP; ++ps) {
              const int rr = ps * RPP + lane / LPR;
              const float4 va = *(const float4*)&ep[rr * PITCH + c8];
              const float4 vb = *(const float4*)&ep[rr * PITCH + c8 + 4];
              if (!decltype(check)::value || (wm * WM + mi * 32 + 8 * qd + rr < nrows && col < ncol)) xr.store(va, vb);
              xr.next();
            }
          }
      };
      if (nrows >= BM && en0 + BN <= ncol)
        emit(std::false_type{});
      else
        emit(std::true_type{});
    }
    if (!more) break;
    Lg = nLg;
    gi = ngi;
    cur = -1;  // the next issue recomputes the operand offsets (not kept live across the epilogue)
  }
#undef LX_SCOMPUTE
#undef LX_SMFMAS
#undef LX_SFRAG
}

// ---------------------------------------------------------------- skinny
// Tiles of a product: the bucketing's tile table, or implicit dense tiles.
__device__ __forceinline__ int skinny_tiles(const GemmArgs& g) {
  return g.tiles ? *g.n_tiles : (g.dense_rows + kSkinnyBM - 1) / kSkinnyBM;
}

// Device-scope coherent 32-bit store and load (relaxed agent-scope atomics):
// another XCD's workgroup that reads the location after this access has
// completed sees its value.
__device__ __forceinline__ void store_dev(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_dev(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// 32 x 64 output tile per 128-thread workgroup (two wavefronts, one 32x32
// MFMA block each). The K loop runs over steps through an LDS ring of SK_NST
// stages; a step is one 64-wide slab of A's K with its weight slab, or, for
// a bf16 (hi, lo) input against one weight row (K = 2 Kb) longer than two
// weight slabs, one weight slab with both halves of A, so every weight slab
// is fetched once. Rings: 4
// stages of 12 KB or 3 of 16 KB (three workgroups per compute unit, two or
// three steps in flight while one is consumed), 2 stages for products of at
// most two steps. With few rows per tile the kernel streams weights and is
// bound by HBM, not by the MFMAs. A product with few output tiles and a long
// K (e.g. a down projection at batch 1) is split along K so that enough
// workgroups stream weight slabs at once; the partial tiles meet in the
// workspace and the last workgroup of a tile adds them.
constexpr int SK_THR = 128;


// Several independent GEMMs in one launch (e.g. the anchor and correction
// products that read the same input rows): problem i owns workgroups
// [base[i], base[i+1]); every base is a multiple of 8, so the XCD of a
// workgroup is its index within the problem modulo 8.
// One work unit of a skinny launch: problem, (item, split), tile, K range.
struct SkUnit {
  const GemmArgs* p;
  int ntn, ofmt, S, Lg, item, kt0, nkl, Kb, nper, n0, ncol, akoff;
  TileEntry te;
};

// Decode this workgroup's unit; false if it has none. spw = K-loop steps per
// weight slab (nper for the slab-per-step LDS kernel in PER == 1 mode, 1
// when a step covers every period of a weight slab).
__device__ __forceinline__ bool sk_unit(const SkinnyBatch& b, bool step_per_weight_slab, SkUnit& u) {
  int pi = 0;
  while (pi + 1 < b.n && (int)blockIdx.x >= b.base[pi + 1]) ++pi;
  const GemmArgs& p = b.g[pi];
  u.p = &p;
  u.ntn = b.ntn[pi];
  u.ofmt = b.ofmt[pi];
  const int wg = (int)blockIdx.x - b.base[pi];
  const int K = p.K;
  u.Kb = p.Kb > 0 ? p.Kb : K;
  const int nk = K / BK2;
  // slab kt: period kt % nper of weight slab kt / nper (as in k_gemm_big)
  u.nper = K / u.Kb;
  const int nkw = nk / u.nper;
  const int spw = step_per_weight_slab ? 1 : u.nper;

  // Split-K when the launch's work items are few: each product's items get
  // S splits of cw weight slabs (the last possibly shorter, none empty),
  // with S * (items of the whole launch) <= split_cap.
  const int items = skinny_tiles(p) * u.ntn;
  int S = 1, cw = nkw;
  if (p.split_force > 1) {
    S = skinny_splits(nkw, p.split_force);
    cw = (nkw + p.split_force - 1) / p.split_force;
  } else if (p.part && items > 0) {
    int all = 0;
    for (int i = 0; i < b.n; ++i) all += skinny_tiles(b.g[i]) * b.ntn[i];
    int s = p.split_cap / all;
    s = s < nkw / kSplitMinSlabs ? s : nkw / kSplitMinSlabs;
    if (s > 1) {
      cw = (nkw + s - 1) / s;
      S = skinny_splits(nkw, s);
    }
  }
  u.S = S;
  // one work unit (item, split) per workgroup, XCD-contiguous order
  // (workgroups >= units)
  const int real = items * S;
  const int q = real / NXCD, rmd = real % NXCD;
  const int x = wg % NXCD;
  const int Lg = x * q + (x < rmd ? x : rmd) + wg / NXCD;
  if (Lg >= x * q + (x < rmd ? x : rmd) + q + (x < rmd ? 1 : 0)) return false;
  u.Lg = Lg;
  u.item = Lg / S;
  const int sp = Lg - u.item * S;
  const int ti = u.item / u.ntn, nt = u.item % u.ntn;
  u.kt0 = sp * cw * spw;
  u.nkl = ((sp + 1) * cw < nkw ? (sp + 1) * cw : nkw) * spw - u.kt0;
  if (p.tiles) {
    u.te = p.tiles[ti];
  } else {
    u.te.widx = 0;
    u.te.row0 = ti * kSkinnyBM;
    u.te.nrows = p.dense_rows - u.te.row0 < kSkinnyBM ? p.dense_rows - u.te.row0 : kSkinnyBM;
    u.te.node = 0;
  }
  u.n0 = nt * kSkinnyBN;
  u.ncol = p.ncols[0] + p.ncols[1];
  u.akoff = p.a_koff[u.n0 < p.ncols[0] ? 0 : 1];
  return true;
}

// Epilogue of a unit: 32 x 32 block per wavefront through its LDS region ep
// (pitch 36 floats), then 4 consecutive columns per lane; with a split, the
// partial-tile hand-off first. Every wavefront of the workgroup calls it.
__device__ __forceinline__ void sk_epilogue(const SkUnit& u, const f32x16& acc, float* ep) {
  constexpr int BM = kSkinnyBM, BN = kSkinnyBN, PITCH = 36, LPR = 8, RPP = 8;
  const GemmArgs& p = *u.p;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const TileEntry& te = u.te;
#pragma unroll
  for (int i = 0; i < 16; ++i) ep[(8 * (i >> 2) + 4 * (lane >> 5) + (i & 3)) * PITCH + (lane & 31)] = acc[i];
  const int c4 = (lane % LPR) * 4;
  const int col = u.n0 + wave * 32 + c4;
  if (u.S > 1) {
    // Partial tile -> slot Lg; the last workgroup of the item to arrive adds
    // the item's S slots in split order (same sum whatever the arrival
    // order). The slots and the counter are only accessed with device-scope
    // coherent operations (they bypass the per-XCD L2 copies), so completing
    // the slot stores before the counter increment is all the ordering the
    // hand-off needs; no cache-wide write-back or invalidation is involved.
    // Slot layout [wavefront][row][32 columns]: each 4-byte access
    // instruction covers two rows, 256 contiguous bytes.
    __shared__ int s_last;
    const int nr = te.nrows;
    const int rr = lane >> 5, cc = lane & 31;
    float* const slot = p.part + (int64_t)u.Lg * (BM * BN) + wave * (32 * 32);
    for (int r = rr; r < nr; r += 2) store_dev(slot + r * 32 + cc, ep[r * PITCH + cc]);
    if (p.defer) return;  // the consumer adds the slots
    wait_vmcnt<0>();
    __syncthreads();
    if (tid == 0)
      s_last = __hip_atomic_fetch_add(p.cnt + u.item, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
               (unsigned)(u.S - 1);
    __syncthreads();
    if (!s_last) return;
    if (tid == 0)  // ready for the next product of this level
      __hip_atomic_store(p.cnt + u.item, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const float* const first = p.part + (int64_t)u.item * u.S * (BM * BN) + wave * (32 * 32);
    for (int r = rr; r < nr; r += 2) {
      float v = load_dev(first + r * 32 + cc);
      for (int t = 1; t < u.S; ++t) v += load_dev(first + (int64_t)t * (BM * BN) + r * 32 + cc);
      ep[r * PITCH + cc] = v;
    }
  }
  if (u.ofmt == OUT_X16) {
    // 8 consecutive columns per lane (one x16 group), 16 rows per pass
    constexpr int LPR8 = 4, RPP8 = 16;
    const int c8 = (lane % LPR8) * 8;
    const int col8 = u.n0 + wave * 32 + c8;
#pragma unroll
    for (int ps = 0; ps < 32 / RPP8; ++ps) {
      const int r = ps * RPP8 + lane / LPR8;
      const float4 va = *(const float4*)&ep[r * PITCH + c8];
      const float4 vb = *(const float4*)&ep[r * PITCH + c8 + 4];
      if (r < te.nrows && col8 < u.ncol)
        *(uint4*)((uint8_t*)p.C + ((int64_t)(te.row0 + r) * p.ldc + col8) * 2) = x16_pack8(va, vb);
    }
    return;
  }
#pragma unroll
  for (int ps = 0; ps < 32 / RPP; ++ps) {
    const int r = ps * RPP + lane / LPR;
    const float4 v = *(const float4*)&ep[r * PITCH + c4];
    if (r >= te.nrows || col >= u.ncol) continue;
    if (u.ofmt == OUT_HILO) {
      const int pp = col < p.ncols[0] ? 0 : 1;
      const int c = pp ? col - p.ncols[0] : col;
      const int hi_col = (pp ? 2 * p.ncols[0] : 0) + c;
      const int lo_col = hi_col + p.ncols[pp];
      bf16x4 h, l;
      h[0] = (__bf16)v.x;
      h[1] = (__bf16)v.y;
      h[2] = (__bf16)v.z;
      h[3] = (__bf16)v.w;
      l[0] = (__bf16)(v.x - (float)h[0]);
      l[1] = (__bf16)(v.y - (float)h[1]);
      l[2] = (__bf16)(v.z - (float)h[2]);
      l[3] = (__bf16)(v.w - (float)h[3]);
      __bf16* const rowp = (__bf16*)p.C + (int64_t)(te.row0 + r) * p.ldc;
      *(bf16x4*)(rowp + hi_col) = h;
      *(bf16x4*)(rowp + lo_col) = l;
    } else {
      *(float4*)(p.C + (int64_t)(te.row0 + r) * p.ldc + col) = v;
    }
  }
}

template <int SK_NST, int PER>
__global__ __launch_bounds__(SK_THR) void k_gemm_skinny(SkinnyBatch b) {
  constexpr int BM = kSkinnyBM, BN = kSkinnyBN;
  constexpr int A_ROUNDS = BM * 8 / SK_THR, B_ROUNDS = BN * 8 / SK_THR;
  constexpr int R = PER * A_ROUNDS + B_ROUNDS;
  constexpr int SA = BM * BK2, STAGE = (PER * BM + BN) * BK2;
  __shared__ __attribute__((aligned(1024))) u16 smem[SK_NST * STAGE];

  // A step of the K loop: PER == 1, one 64-wide slab of A's K (any nper);
  // PER == 2 (nper == 2), one weight slab, multiplied by both periods of A
  // (the weight slab is loaded once for the hi and the lo half)
  SkUnit u;
  if (!sk_unit(b, PER == 2, u)) return;
  const GemmArgs& p = *u.p;
  const int Kb = u.Kb, nper = u.nper, kt0 = u.kt0, nkl = u.nkl;
  const TileEntry& te = u.te;

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int ncol = u.ncol;
  const u16* __restrict__ Ab = (const u16*)p.A;
  const u16* __restrict__ Bw0 = (const u16*)p.B[0] + (int64_t)te.widx * p.b_stride[0];
  const u16* __restrict__ Bw1 = (const u16*)p.B[1] + (int64_t)te.widx * p.b_stride[1];

  // LDS slot P = round * 128 + tid holds row P >> 3, physical chunk P & 7
  // (logical chunk (P & 7) ^ swz(row)); rows past the tile are clamped.
  uint32_t aoff[A_ROUNDS];
#pragma unroll
  for (int j = 0; j < A_ROUNDS; ++j) {
    const int Ps = j * SK_THR + tid;
    const int row = Ps >> 3;
    const int c = (Ps & 7) ^ swz2(row);
    const int r = row < te.nrows ? row : te.nrows - 1;
    const int src = p.a_rows ? p.a_rows[te.row0 + r] : te.row0 + r;
    aoff[j] = (uint32_t)src * (uint32_t)p.lda + (uint32_t)(u.akoff + c * 8);
  }
  const u16* bptr[B_ROUNDS];
#pragma unroll
  for (int j = 0; j < B_ROUNDS; ++j) {
    const int Ps = j * SK_THR + tid;
    const int row = Ps >> 3;
    const int c = (Ps & 7) ^ swz2(row);
    const int n = u.n0 + row < ncol ? u.n0 + row : ncol - 1;
    bptr[j] = (n < p.ncols[0] ? Bw0 + (int64_t)n * Kb : Bw1 + (int64_t)(n - p.ncols[0]) * Kb) + c * 8;
  }
  // stage = [A period 0 | (A period 1) | B], one 64-wide K slab each
  auto issue = [&](int st, int kt) {
    u16* const sA = smem + st * STAGE;
    int kb;
    if (PER == 1) {
      const int qq = kt / nper, per = kt - qq * nper;
      kb = qq * BK2;
      const int ka = per * Kb + kb;
#pragma unroll
      for (int j = 0; j < A_ROUNDS; ++j)
        load_lds16(Ab + (aoff[j] + (uint32_t)ka), sA + (j * SK_THR + wave * 64) * 8);
    } else {
      kb = kt * BK2;
#pragma unroll
      for (int per = 0; per < PER; ++per)
#pragma unroll
        for (int j = 0; j < A_ROUNDS; ++j)
          load_lds16(Ab + (aoff[j] + (uint32_t)(per * Kb + kb)), sA + per * SA + (j * SK_THR + wave * 64) * 8);
    }
#pragma unroll
    for (int j = 0; j < B_ROUNDS; ++j) load_lds16(bptr[j] + kb, sA + PER * SA + (j * SK_THR + wave * 64) * 8);
  };

  f32x16 acc;
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.f;
  auto compute = [&](int st) {
    const u16* const sA = smem + st * STAGE;
    const u16* const sB = sA + PER * SA;
    const int ra = lane & 31, rb = wave * 32 + (lane & 31);
    bf16x8 fa[PER][4], fb[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int kc = ks * 2 + (lane >> 5);
#pragma unroll
      for (int per = 0; per < PER; ++per) fa[per][ks] = *(const bf16x8*)&sA[per * SA + lds_off2(ra, kc)];
      fb[ks] = *(const bf16x8*)&sB[lds_off2(rb, kc)];
    }
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int per = 0; per < PER; ++per)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[per][ks], fb[ks], acc, 0, 0, 0);
  };

  // Local step i (global kt0 + i) lives in stage i % SK_NST. Steps
  // 0 .. SK_NST-1 are issued up front; after the barrier that follows step
  // i's compute, stage i % SK_NST is free and step i + SK_NST goes there.
  static_assert(SK_NST >= 2 && SK_NST <= 4, "ring depth");
  const int npre = nkl < SK_NST ? nkl : SK_NST;
  for (int i = 0; i < npre; ++i) issue(i, kt0 + i);
  wait_slabs<R>(npre - 1);
  bar();
  for (int i = 0; i < nkl; ++i) {
    compute(i % SK_NST);
    if (i + 1 < nkl) {
      // steps issued so far: 0 .. min(i + SK_NST - 1, nkl - 1); wait for i + 1
      const int last = i + SK_NST - 1 < nkl - 1 ? i + SK_NST - 1 : nkl - 1;
      wait_slabs<R>(last - (i + 1));
      wait_lgkm0();
      bar();
      if (i + SK_NST < nkl) issue(i % SK_NST, kt0 + i + SK_NST);
    }
  }
  wait_lgkm0();
  bar();  // every wavefront is done with the stages: the epilogue reuses them
  sk_epilogue(u, acc, (float*)smem + wave * (32 * 36));
}


// Wide variant for products whose K is one weight slab (K = 64, or a bf16
// (hi, lo) pair against a 64-column weight row): a workgroup takes NB
// consecutive 64-column tiles of one row tile, loads the A slab(s) once and
// every weight slab at once (no K loop, nothing to pipeline), so the fixed
// per-workgroup latency (tile entry, row map, one load round trip, epilogue)
// is paid once per NB tiles. Wavefront w computes columns w * 32 .. w * 32 + 31
// of each of its tiles.
template <int NB, int PER>
__global__ __launch_bounds__(SK_THR) void k_gemm_skinny_wide(SkinnyBatch b) {
  constexpr int BM = kSkinnyBM, BN = kSkinnyBN;
  constexpr int A_ROUNDS = BM * 8 / SK_THR, B_ROUNDS = BN * 8 / SK_THR;
  constexpr int SA = BM * BK2, SBt = BN * BK2;
  __shared__ __attribute__((aligned(1024))) u16 smem[PER * SA + NB * SBt];

  int pi = 0;
  while (pi + 1 < b.n && (int)blockIdx.x >= b.base[pi + 1]) ++pi;
  const GemmArgs& p = b.g[pi];
  const int ntn = b.ntn[pi], ofmt = b.ofmt[pi];
  const int ngr = (ntn + NB - 1) / NB;  // column groups
  const int wg = (int)blockIdx.x - b.base[pi];
  const int real = skinny_tiles(p) * ngr;
  const int q = real / NXCD, rmd = real % NXCD;
  const int x = wg % NXCD;
  const int Lg = x * q + (x < rmd ? x : rmd) + wg / NXCD;
  if (Lg >= x * q + (x < rmd ? x : rmd) + q + (x < rmd ? 1 : 0)) return;
  const int ti = Lg / ngr, gr = Lg % ngr;
  SkUnit u;
  u.p = &p;
  u.ntn = ntn;
  u.ofmt = ofmt;
  u.S = 1;
  u.Lg = Lg;
  u.item = 0;
  u.kt0 = 0;
  u.nkl = 1;
  u.Kb = p.Kb > 0 ? p.Kb : p.K;
  u.nper = p.K / u.Kb;
  if (p.tiles) {
    u.te = p.tiles[ti];
  } else {
    u.te.widx = 0;
    u.te.row0 = ti * BM;
    u.te.nrows = p.dense_rows - u.te.row0 < BM ? p.dense_rows - u.te.row0 : BM;
    u.te.node = 0;
  }
  u.ncol = p.ncols[0] + p.ncols[1];
  const TileEntry& te = u.te;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int Kb = u.Kb;
  const u16* __restrict__ Ab = (const u16*)p.A;
  const u16* __restrict__ Bw0 = (const u16*)p.B[0] + (int64_t)te.widx * p.b_stride[0];
  const u16* __restrict__ Bw1 = (const u16*)p.B[1] + (int64_t)te.widx * p.b_stride[1];
  const int n0g = gr * NB * BN;
  // the group's A column offset: its tiles lie in one part (the host checks
  // that the part boundary is a multiple of NB * 64 when the parts differ)
  const int akoff = p.a_koff[n0g < p.ncols[0] ? 0 : 1];

#pragma unroll
  for (int per = 0; per < PER; ++per)
#pragma unroll
    for (int j = 0; j < A_ROUNDS; ++j) {
      const int Ps = j * SK_THR + tid;
      const int row = Ps >> 3;
      const int c = (Ps & 7) ^ swz2(row);
      const int r = row < te.nrows ? row : te.nrows - 1;
      const int src = p.a_rows ? p.a_rows[te.row0 + r] : te.row0 + r;
      load_lds16(Ab + ((uint32_t)src * (uint32_t)p.lda + (uint32_t)(akoff + per * Kb + c * 8)),
                 smem + per * SA + (j * SK_THR + wave * 64) * 8);
    }
#pragma unroll
  for (int t = 0; t < NB; ++t)
#pragma unroll
    for (int j = 0; j < B_ROUNDS; ++j) {
      const int Ps = j * SK_THR + tid;
      const int row = Ps >> 3;
      const int c = (Ps & 7) ^ swz2(row);
      int n = n0g + t * BN + row;
      n = n < u.ncol ? n : u.ncol - 1;
      const u16* bp = (n < p.ncols[0] ? Bw0 + (int64_t)n * Kb : Bw1 + (int64_t)(n - p.ncols[0]) * Kb) + c * 8;
      load_lds16(bp, smem + PER * SA + t * SBt + (j * SK_THR + wave * 64) * 8);
    }
  wait_vmcnt<0>();
  bar();
  f32x16 acc[NB];
#pragma unroll
  for (int t = 0; t < NB; ++t)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[t][i] = 0.f;
  const int ra = lane & 31, rb = wave * 32 + (lane & 31);
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    const int kc = ks * 2 + (lane >> 5);
    bf16x8 fa[PER];
#pragma unroll
    for (int per = 0; per < PER; ++per) fa[per] = *(const bf16x8*)&smem[per * SA + lds_off2(ra, kc)];
#pragma unroll
    for (int t = 0; t < NB; ++t) {
      const bf16x8 fb = *(const bf16x8*)&smem[PER * SA + t * SBt + lds_off2(rb, kc)];
#pragma unroll
      for (int per = 0; per < PER; ++per)
        acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[per], fb, acc[t], 0, 0, 0);
    }
  }
  wait_lgkm0();
  bar();  // the epilogue reuses the LDS
  float* const ep = (float*)smem + wave * (32 * 36);
#pragma unroll
  for (int t = 0; t < NB; ++t) {
    u.n0 = n0g + t * BN;
    if (u.n0 >= u.ncol) break;  // uniform
    u.akoff = akoff;
    sk_epilogue(u, acc[t], ep);
    bar();  // ep is rewritten by the next tile
  }
}

template <int BM, int BN>
hipError_t launch_bn(const GemmArgs& g, int ofmt, int grid, int ntn, hipStream_t s) {
  if constexpr (BM == 256 && BN >= 128) {
    if (ofmt == OUT_F16T) {
      hipLaunchKernelGGL((k_gemm_big<BM, BN, OUT_F16T>), dim3(grid), dim3(BigCfg<BM, BN>::NTHR), 0, s, g, ntn);
      return hipGetLastError();
    }
  }
  if (ofmt == OUT_F16T) return hipErrorInvalidValue;
  if (ofmt == OUT_HILO)
    hipLaunchKernelGGL((k_gemm_big<BM, BN, OUT_HILO>), dim3(grid), dim3(BigCfg<BM, BN>::NTHR), 0, s, g, ntn);
  else if (ofmt == OUT_X16)
    hipLaunchKernelGGL((k_gemm_big<BM, BN, OUT_X16>), dim3(grid), dim3(BigCfg<BM, BN>::NTHR), 0, s, g, ntn);
  else
    hipLaunchKernelGGL((k_gemm_big<BM, BN, OUT_F32>), dim3(grid), dim3(BigCfg<BM, BN>::NTHR), 0, s, g, ntn);
  return hipGetLastError();
}

// fp8 copy of bf16 weights: one thread per (row, 64-column slab); each
// 32-column block gets its own E8M0 scale (block max in [128, 256)).
__global__ __launch_bounds__(256) void k_quantize_f8(const u16* __restrict__ w, int64_t n_rows, int cols,
                                                     uint8_t* __restrict__ w8, uint32_t* __restrict__ sc) {
  const int nsl = cols / BK2;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_rows * nsl) return;
  const int64_t row = i / nsl;
  const int sl = (int)(i - row * nsl);
  const u16* src = w + row * cols + sl * BK2;
  uint8_t* dst = w8 + row * cols + sl * BK2;
  uint32_t word = 0;
  for (int b = 0; b < 2; ++b) {
    float v[32];
    float amax = 0.f;
    for (int e = 0; e < 32; ++e) {
      v[e] = __uint_as_float((uint32_t)src[b * 32 + e] << 16);
      amax = fmaxf(amax, fabsf(v[e]));
    }
    const uint32_t be = e8m0_for(amax);
    word |= be << (8 * b);
    for (int e = 0; e < 32; e += 4) {
      const uint32_t q = f32_to_e4m3(e8m0_unscale(v[e], be)) | (f32_to_e4m3(e8m0_unscale(v[e + 1], be)) << 8) |
                         (f32_to_e4m3(e8m0_unscale(v[e + 2], be)) << 16) |
                         (f32_to_e4m3(e8m0_unscale(v[e + 3], be)) << 24);
      *(uint32_t*)(dst + b * 32 + e) = q;
    }
  }
  sc[row * nsl + sl] = word;
}

// fp16 copy of bf16 weights, scaled per matrix by a power of two so that its
// largest magnitude lands in [2^14, 2^15): max |w| per matrix (float bits
// compare as integers for non-negative values), then the exponents, then the
// conversion (round to nearest even; exact for every bf16 value down to
// 2^-28 of the matrix maximum).
__global__ __launch_bounds__(256) void k_absmax_bits(const u16* __restrict__ w, int64_t per, int n,
                                                     uint32_t* __restrict__ mx) {
  const int i = blockIdx.y;
  uint32_t m = 0;
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < per; j += (int64_t)gridDim.x * blockDim.x)
    m = max(m, (uint32_t)(w[(int64_t)i * per + j] & 0x7FFFu) << 16);
  for (int off = 32; off >= 1; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off, 64));
  if ((threadIdx.x & 63) == 0) atomicMax(mx + i, m);
}

__device__ __forceinline__ int f16_exp_for(uint32_t maxbits) {
  if (maxbits == 0) return 0;
  const int e = (int)(maxbits >> 23) - 127;  // floor(log2(max)); subnormal maxima count as 2^-127
  const int s = 14 - e;
  return s < -100 ? -100 : s > 100 ? 100 : s;
}

__global__ __launch_bounds__(256) void k_to_f16(const u16* __restrict__ w, int64_t per, int n,
                                                const uint32_t* __restrict__ mx, _Float16* __restrict__ w16) {
  const int i = blockIdx.y;
  const int s = f16_exp_for(mx[i]);
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < per; j += (int64_t)gridDim.x * blockDim.x) {
    const float v = __uint_as_float((uint32_t)w[(int64_t)i * per + j] << 16);
    w16[(int64_t)i * per + j] = (_Float16)ldexpf(v, s);
  }
}

// Zero-padded copy [n][rows][cols] -> [n][rows_out][cols_out]: fp16 scaled
// as k_to_f16 (F16), or the bf16 values unchanged.
template <bool F16>
__global__ __launch_bounds__(256) void k_copy_pad(const u16* __restrict__ w, int rows, int cols, int rows_out,
                                                  int cols_out, const uint32_t* __restrict__ mx,
                                                  u16* __restrict__ out) {
  const int i = blockIdx.y;
  const int s = F16 ? f16_exp_for(mx[i]) : 0;
  const int64_t per_out = (int64_t)rows_out * cols_out;
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < per_out; j += (int64_t)gridDim.x * blockDim.x) {
    const int r = (int)(j / cols_out), c = (int)(j - (int64_t)r * cols_out);
    u16 v = 0;
    if (r < rows && c < cols) {
      const u16 b = w[((int64_t)i * rows + r) * cols + c];
      if constexpr (F16)
        v = __builtin_bit_cast(u16, (_Float16)ldexpf(__uint_as_float((uint32_t)b << 16), s));
      else
        v = b;
    }
    out[(int64_t)i * per_out + j] = v;
  }
}

__global__ void k_f16_exps(uint32_t* __restrict__ mx, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) mx[i] = (uint32_t)f16_exp_for(mx[i]);
}

__global__ void k_zero_u32(uint32_t* __restrict__ p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

}  // namespace

hipError_t launch_convert_f16(const void* w, int n, int64_t per, void* w16, int32_t* exps, hipStream_t s) {
  if (n <= 0 || per <= 0) return hipSuccess;
  uint32_t* const mx = (uint32_t*)exps;
  const int g1 = (n + 255) / 256;
  hipLaunchKernelGGL(k_zero_u32, dim3(g1), dim3(256), 0, s, mx, n);
  const int gx = (int)std::min<int64_t>((per + 255) / 256, 1024);
  hipLaunchKernelGGL(k_absmax_bits, dim3(gx, n), dim3(256), 0, s, (const u16*)w, per, n, mx);
  hipLaunchKernelGGL(k_to_f16, dim3(gx, n), dim3(256), 0, s, (const u16*)w, per, n, mx, (_Float16*)w16);
  hipLaunchKernelGGL(k_f16_exps, dim3(g1), dim3(256), 0, s, mx, n);
  return hipGetLastError();
}

hipError_t launch_copy_pad(const void* w, int n, int rows, int cols, int rows_out, int cols_out, void* out,
                           int32_t* exps, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int gx = (int)std::min<int64_t>(((int64_t)rows_out * cols_out + 255) / 256, 1024);
  if (!exps) {
    hipLaunchKernelGGL(k_copy_pad<false>, dim3(gx, n), dim3(256), 0, s, (const u16*)w, rows, cols, rows_out, cols_out,
                       (const uint32_t*)nullptr, (u16*)out);
    return hipGetLastError();
  }
  uint32_t* const mx = (uint32_t*)exps;
  const int g1 = (n + 255) / 256;
  const int64_t per = (int64_t)rows * cols;
  hipLaunchKernelGGL(k_zero_u32, dim3(g1), dim3(256), 0, s, mx, n);
  const int ga = (int)std::min<int64_t>((per + 255) / 256, 1024);
  hipLaunchKernelGGL(k_absmax_bits, dim3(ga, n), dim3(256), 0, s, (const u16*)w, per, n, mx);
  hipLaunchKernelGGL(k_copy_pad<true>, dim3(gx, n), dim3(256), 0, s, (const u16*)w, rows, cols, rows_out, cols_out,
                     (const uint32_t*)mx, (u16*)out);
  hipLaunchKernelGGL(k_f16_exps, dim3(g1), dim3(256), 0, s, mx, n);
  return hipGetLastError();
}

bool gemm_f16_ok(const GemmArgs& g, int bn, int ofmt, int64_t a_rows_total) {
  if (!g.a_row_exp || !g.b_exp || g.a_rows || g.K <= 0 || g.K % BK2 || (g.Kb > 0 && g.Kb != g.K)) return false;
  if (ofmt == OUT_F16T) {
    if (bn != 64 && bn != 128 && bn != 256) return false;
    if (!g.c_row_exp || g.ncols[0] + g.ncols[1] > bn || ((uintptr_t)g.c_row_exp & 3)) return false;
  } else if (bn != 256 || (ofmt != OUT_X16 && ofmt != OUT_F32)) {
    return false;
  }
  return gemm_big_ok(g, bn, a_rows_total);
}

// x16 rows need a row length that keeps every 8-byte mantissa word aligned.
// x16 outputs: whole 8-value groups per part, 16-byte aligned rows
static bool x16_shape_ok(const GemmArgs& g, int ofmt) {
  return ofmt != OUT_X16 || (g.ldc % 8 == 0 && g.ncols[0] % 8 == 0 && g.ncols[1] % 8 == 0 && ((uintptr_t)g.C & 15) == 0);
}

hipError_t launch_gemm_f16(const GemmArgs& g, int bn, int ofmt, int grid_tiles, hipStream_t s) {
  if (!x16_shape_ok(g, ofmt)) return hipErrorInvalidValue;
  const int ntn = (g.ncols[0] + g.ncols[1] + bn - 1) / bn;
  int grid = grid_tiles * ntn;
  if (grid <= 0) return hipSuccess;
  const int cap = grid_cap();
  if (grid > cap) grid = cap;
  if (ofmt == OUT_F16T && bn == 64)
    hipLaunchKernelGGL((k_gemm_big<256, 64, OUT_F16T, false, true>), dim3(grid), dim3(BigCfg<256, 64>::NTHR), 0, s,
                       g, ntn);
  else if (ofmt == OUT_F16T && bn == 128)
    hipLaunchKernelGGL((k_gemm_big<256, 128, OUT_F16T, false, true>), dim3(grid), dim3(BigCfg<256, 128>::NTHR), 0,
                       s, g, ntn);
  else if (ofmt == OUT_F16T && bn == 256)
    hipLaunchKernelGGL((k_gemm_big<256, 256, OUT_F16T, false, true>), dim3(grid), dim3(512), 0, s, g, ntn);
  else if (ofmt == OUT_X16 && bn == 256)
    hipLaunchKernelGGL((k_gemm_big<256, 256, OUT_X16, false, true>), dim3(grid), dim3(512), 0, s, g, ntn);
  else if (ofmt == OUT_F32 && bn == 256)
    hipLaunchKernelGGL((k_gemm_big<256, 256, OUT_F32, false, true>), dim3(grid), dim3(512), 0, s, g, ntn);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_gemm_f16_pair(const GemmArgs& g0, int grid_tiles0, const GemmArgs& g1, int ofmt1,
                                int grid_tiles1, hipStream_t s) {
  if (!x16_shape_ok(g0, OUT_X16) || !x16_shape_ok(g1, ofmt1)) return hipErrorInvalidValue;
  const int ntn0 = (g0.ncols[0] + g0.ncols[1] + 255) / 256;
  const int ntn1 = (g1.ncols[0] + g1.ncols[1] + 255) / 256;
  int grid = grid_tiles0 * ntn0 + grid_tiles1 * ntn1;
  if (grid <= 0) return hipSuccess;
  // a multiple of 8: the second product's remainder items go to the XCDs
  // from the last one down, so every XCD needs a workgroup
  grid = (grid + NXCD - 1) / NXCD * NXCD;
  const int cap = grid_cap();
  if (grid > cap) grid = cap;
  if (ofmt1 == OUT_F16T)
    hipLaunchKernelGGL((k_gemm_big2<256, 256, OUT_X16, OUT_F16T, true>), dim3(grid), dim3(512), 0, s, g0, ntn0, g1,
                       ntn1);
  else if (ofmt1 == OUT_X16)
    hipLaunchKernelGGL((k_gemm_big2<256, 256, OUT_X16, OUT_X16, true>), dim3(grid), dim3(512), 0, s, g0, ntn0, g1,
                       ntn1);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

bool gemm_lo8_ok(const GemmArgs& g, int64_t a_rows_total) {
  if (!g.b8 || !g.bsc || g.a_rows || g.ncols[1] != 0 || g.Kb <= 0 || g.K != 2 * g.Kb || g.Kb % BK2) return false;
  if (((uintptr_t)g.b8 & 15) || ((uintptr_t)g.bsc & 3) || (g.a_lo8_off & 15) || (g.a_sc_off & 3)) return false;
  if (g.a_lo8_off < 2 * g.Kb || g.a_sc_off < g.a_lo8_off + g.Kb || g.a_sc_off + g.Kb / 16 > 2 * g.lda) return false;
  if ((2 * g.lda) % 16) return false;
  return gemm_big_ok(g, 256, a_rows_total);
}

hipError_t launch_quantize_f8(const void* w, int64_t n_rows, int cols, uint8_t* w8, uint32_t* sc, hipStream_t s) {
  const int64_t n = n_rows * (cols / BK2);
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_quantize_f8, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, (const u16*)w, n_rows,
                     cols, w8, sc);
  return hipGetLastError();
}

bool gemm_big_ok(const GemmArgs& g, int bn, int64_t a_rows_total) {
  const int Kb = g.Kb > 0 ? g.Kb : g.K;
  // 64-wide K-slabs; a period Kb < K that is not a multiple of 64 is taken
  // chunk by chunk (large-tile kernel only, 8-column chunks)
  if (g.K <= 0 || g.K % BK2 || Kb % 8 || g.K % Kb || (Kb % BK2 && Kb == g.K)) return false;
  if (g.a_koff[0] + g.K > g.lda || (g.ncols[1] > 0 && g.a_koff[1] + g.K > g.lda)) return false;
  if (g.ncols[1] > 0 && g.a_koff[0] != g.a_koff[1] && g.ncols[0] % bn) return false;
  // the epilogue stores 4 consecutive columns per lane
  if (g.ncols[0] % 4 || g.ncols[1] % 4 || g.ldc % 4 || ((uintptr_t)g.C & 15)) return false;
  return a_rows_total * g.lda < ((int64_t)1 << 31);
}

namespace {
// Persistent grid cap: the largest multiple of 8 not above the device's
// compute-unit count (one 128 KB-LDS workgroup fits per compute unit).
int grid_cap() {
  static std::mutex mu;
  static int cap[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  std::lock_guard<std::mutex> lk(mu);
  if (!cap[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 8) n = 256;
    cap[dev] = n / NXCD * NXCD;
  }
  return cap[dev];
}
}  // namespace

hipError_t launch_gemm_big(const GemmArgs& g, int bm, int bn, int ofmt, int grid_tiles, hipStream_t s) {
  if (!x16_shape_ok(g, ofmt)) return hipErrorInvalidValue;
  // fp16 output with one scale per tile: the tile spans whole rows
  if (ofmt == OUT_F16T && (!g.c_row_exp || g.ncols[0] + g.ncols[1] > bn || bm != 256 || bn < 128))
    return hipErrorInvalidValue;
  const int ntn = (g.ncols[0] + g.ncols[1] + bn - 1) / bn;
  int grid = grid_tiles * ntn;  // upper bound on work items
  if (grid <= 0) return hipSuccess;
  const int cap = grid_cap();
  if (grid > cap) grid = cap;
  if (bm == 256) {
    if (bn == 256) return launch_bn<256, 256>(g, ofmt, grid, ntn, s);
    if (bn == 128) return launch_bn<256, 128>(g, ofmt, grid, ntn, s);
    return launch_bn<256, 64>(g, ofmt, grid, ntn, s);
  }
  if (bn == 256) return launch_bn<128, 256>(g, ofmt, grid, ntn, s);
  if (bn == 128) return launch_bn<128, 128>(g, ofmt, grid, ntn, s);
  return launch_bn<128, 64>(g, ofmt, grid, ntn, s);
}

bool gemm_seg_ok(const GemmArgs& g, const SegArgs& sa, int64_t out_rows) {
  if (sa.nseg < 1 || sa.nseg > kSegMax || !sa.anc || !g.tiles || !g.n_tiles) return false;
  const int ncol = g.ncols[0] + g.ncols[1];
  // tiles never straddle the two parts (their A columns differ)
  if (g.ncols[1] > 0 && g.ncols[0] % 256) return false;
  // (x16 output, 8 columns per lane: 16-byte aligned rows)
  if (g.ncols[0] % 8 || g.ncols[1] % 8 || g.ldc % 8 || g.ldc < ncol || ((uintptr_t)g.C & 15)) return false;
  if (out_rows * g.ldc * 3 >= ((int64_t)1 << 40)) return false;
  for (int i = 0; i < sa.nseg; ++i) {
    const SegDesc& d = sa.s[i];
    if (!d.A || !d.B[0] || (g.ncols[1] > 0 && !d.B[1]) || d.rank <= 0 || d.rank % BK2) return false;
    if (d.anc_off >= 0 && !d.fac) return false;
    const int kw = sa.f16 ? d.rank : 2 * d.rank;  // A columns per part
    if (d.a_col0 < 0 || d.a_col0 % 8 || d.a_col0 + d.akoff1 + kw > d.lda || (g.ncols[1] == 0 && d.a_col0 + kw > d.lda))
      return false;
    if (sa.f16 && (!d.a_exp || !d.b_exp[0] || (g.ncols[1] > 0 && !d.b_exp[1]))) return false;
    if (((uintptr_t)d.A & 15) || ((uintptr_t)d.B[0] & 15) || ((uintptr_t)d.B[1] & 15)) return false;
    // 32-bit byte offsets: the weight rows of one factor
    if ((int64_t)ncol * d.rank * 2 >= ((int64_t)1 << 31)) return false;
  }
  return true;
}

hipError_t launch_gemm_seg(const GemmArgs& g, const SegArgs& sa_in, int grid_tiles, hipStream_t s) {
  const int ntn = (g.ncols[0] + g.ncols[1] + 255) / 256;
  // column tiles per work item: 4 (or 2) when every part is a whole number of
  // such groups, so a group never straddles the parts
  SegArgs sa = sa_in;
  sa.ngrp = 1;
  for (const int gsz : {4, 2})
    if (g.ncols[0] % (gsz * 256) == 0 && g.ncols[1] % (gsz * 256) == 0) {
      sa.ngrp = gsz;
      break;
    }
  int grid = grid_tiles * (ntn / sa.ngrp);
  if (grid <= 0) return hipSuccess;
  const int cap = grid_cap();
  if (grid > cap) grid = cap;
  if (sa.f16)
    hipLaunchKernelGGL(k_gemm_seg<true>, dim3(grid), dim3(512), 0, s, g, sa, ntn);
  else
    hipLaunchKernelGGL(k_gemm_seg<false>, dim3(grid), dim3(512), 0, s, g, sa, ntn);
  return hipGetLastError();
}

hipError_t launch_gemm_lo8(const GemmArgs& g, int ofmt, int grid_tiles, hipStream_t s) {
  if (!x16_shape_ok(g, ofmt)) return hipErrorInvalidValue;
  const int ntn = (g.ncols[0] + 255) / 256;
  int grid = grid_tiles * ntn;
  if (grid <= 0) return hipSuccess;
  const int cap = grid_cap();
  if (grid > cap) grid = cap;
  if (ofmt == OUT_X16)
    hipLaunchKernelGGL((k_gemm_big<256, 256, OUT_X16, true>), dim3(grid), dim3(512), 0, s, g, ntn);
  else
    hipLaunchKernelGGL((k_gemm_big<256, 256, OUT_F32, true>), dim3(grid), dim3(512), 0, s, g, ntn);
  return hipGetLastError();
}

hipError_t launch_gemm_skinny_batch(const GemmArgs* g, const int* ofmt, const int* grid_tiles, int n,
                                    hipStream_t s) {
  if (n < 1 || n > kSkinnyMaxProblems) return hipErrorInvalidValue;
  for (int i = 0; i < n; ++i)
    if (!x16_shape_ok(g[i], ofmt[i])) return hipErrorInvalidValue;
  SkinnyBatch b{};
  int wg = 0;
  for (int i = 0; i < n; ++i) {
    b.g[i] = g[i];
    b.ntn[i] = (g[i].ncols[0] + g[i].ncols[1] + kSkinnyBN - 1) / kSkinnyBN;
    b.ofmt[i] = ofmt[i];
    b.base[i] = wg;
    wg += skinny_grid(g[i], (int64_t)grid_tiles[i] * b.ntn[i]);  // a multiple of 8
  }
  b.base[n] = wg;
  b.n = n;
  if (wg <= 0) return hipSuccess;
  // every product a bf16 (hi, lo) pair against one weight row, some longer
  // than two weight slabs: one weight slab per step for both halves
  // (3-stage ring of 16 KB stages)
  bool pair = true;
  int max_steps = 0;
  for (int i = 0; i < n; ++i) {
    const int Kb = g[i].Kb > 0 ? g[i].Kb : g[i].K;
    pair = pair && g[i].K == 2 * Kb;
    max_steps = std::max(max_steps, g[i].K / BK2);
  }
  // every product one weight slab of 64 (K = 64, or a hi/lo pair of them),
  // no split, part boundaries that no 4-tile group straddles, and enough row
  // tiles that 4-tile groups still give at least 512 workgroups: wide
  // (with few row tiles, e.g. one token, the narrow kernel keeps more
  // workgroups, hence more loads, in flight)
  bool wide = true;
  int64_t groups = 0;
  for (int i = 0; i < n; ++i) groups += (int64_t)grid_tiles[i] * ((b.ntn[i] + 3) / 4);
  wide = groups >= 512;
  for (int i = 0; i < n; ++i) {
    const int Kb = g[i].Kb > 0 ? g[i].Kb : g[i].K;
    wide = wide && Kb == BK2 && (g[i].K == BK2 || g[i].K == 2 * BK2) && g[i].K == g[0].K && g[i].split_force <= 1 &&
           (g[i].ncols[1] == 0 || g[i].a_koff[0] == g[i].a_koff[1] || g[i].ncols[0] % (4 * kSkinnyBN) == 0);
  }
  if (wide) {
    SkinnyBatch bw = b;
    int wgw = 0;
    for (int i = 0; i < n; ++i) {
      bw.base[i] = wgw;
      const int ngr = (b.ntn[i] + 3) / 4;
      wgw += (grid_tiles[i] * ngr + NXCD - 1) / NXCD * NXCD;
    }
    bw.base[n] = wgw;
    if (wgw <= 0) return hipSuccess;
    if (g[0].K == 2 * BK2)
      hipLaunchKernelGGL((k_gemm_skinny_wide<4, 2>), dim3(wgw), dim3(SK_THR), 0, s, bw);
    else
      hipLaunchKernelGGL((k_gemm_skinny_wide<4, 1>), dim3(wgw), dim3(SK_THR), 0, s, bw);
    return hipGetLastError();
  }
  if (pair && max_steps > 4) {
    hipLaunchKernelGGL((k_gemm_skinny<3, 2>), dim3(wg), dim3(SK_THR), 0, s, b);
  } else if (max_steps <= 2) {
    hipLaunchKernelGGL((k_gemm_skinny<2, 1>), dim3(wg), dim3(SK_THR), 0, s, b);
  } else {
    hipLaunchKernelGGL((k_gemm_skinny<4, 1>), dim3(wg), dim3(SK_THR), 0, s, b);
  }
  return hipGetLastError();
}

int skinny_grid(const GemmArgs& g, int64_t items_max) {
  const int Kb = g.Kb > 0 ? g.Kb : g.K;
  int64_t n = items_max;
  if (g.split_force > 1)
    n = items_max * skinny_splits(Kb / BK2, g.split_force);  // Kb / 64 weight slabs
  else if (g.part && Kb / BK2 >= 2 * kSplitMinSlabs)
    n = std::max<int64_t>(n, g.split_cap);
  return (int)((n + NXCD - 1) / NXCD * NXCD);
}

hipError_t launch_gemm_skinny(const GemmArgs& g, int ofmt, int grid_tiles, hipStream_t s) {
  if (!x16_shape_ok(g, ofmt)) return hipErrorInvalidValue;
  return launch_gemm_skinny_batch(&g, &ofmt, &grid_tiles, 1, s);
}

}  // namespace lx

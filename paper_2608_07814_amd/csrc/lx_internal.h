// Internal declarations shared by the host orchestration and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "lorex.h"

namespace lx {

// ---------------------------------------------------------------- x16 rows
// Intermediates that only the elementwise kernels read back (gate|up
// outputs, down outputs) are stored as groups of 8 consecutive values (a
// group starts at a column that is a multiple of 8) in 16 bytes: eight
// 16-bit slots. They share one exponent, the biased exponent byte E of the
// group's largest magnitude (mx in [2^(E-127), 2^(E-126))). Slot i holds value
// i as the 15-bit signed integer m = round(32767 * v * 2^(125 - E)) (|v|
// 2^(125-E) < 1/2, so -16384 <= m <= 16383) in its bits 15..1, and bit i of E
// in its bit 0: v = m / 32767 * 2^(E - 125). The error of a value is at most
// half a step, 2^-15 of 2^(E-126), i.e. 2^-14 of the group's largest magnitude. One
// conversion instruction (v_cvt_pknorm_i16_f32: clamp to [-1, 1], scale by
// 32767, round to nearest) encodes two values. A row of n values (n a multiple
// of 8) is 2n bytes; the exponent travels with the mantissas, so a group is
// one 16-byte store and one 16-byte load.
typedef short x16_short2 __attribute__((ext_vector_type(2)));

// values [0, 4) = a, [4, 8) = b of a group
__device__ __forceinline__ uint4 x16_pack8(float4 a, float4 b) {
  const float mx = fmaxf(fmaxf(fmaxf(fabsf(a.x), fabsf(a.y)), fmaxf(fabsf(a.z), fabsf(a.w))),
                         fmaxf(fmaxf(fabsf(b.x), fabsf(b.y)), fmaxf(fabsf(b.z), fabsf(b.w))));
  const uint32_t e = (__float_as_uint(mx) >> 23) & 0xFFu;
  const int sh = 125 - (int)e;
  auto pk = [&](float u, float v, int k) {
    const x16_short2 q = __builtin_amdgcn_cvt_pknorm_i16(ldexpf(u, sh), ldexpf(v, sh));
    // exponent bits 2k, 2k + 1 at bit 0 of each 16-bit half
    const uint32_t t = __builtin_amdgcn_ubfe(e, 2 * k, 2);
    const uint32_t eb = (t | (t << 15)) & 0x10001u;
    // each half shifted up by one (its top bit is a copy of the sign), the
    // exponent bits into the freed low bits
    return ((__builtin_bit_cast(uint32_t, q) << 1) & 0xFFFEFFFEu) | eb;
  };
  return make_uint4(pk(a.x, a.y, 0), pk(a.z, a.w, 1), pk(b.x, b.y, 2), pk(b.z, b.w, 3));
}

// the group's exponent byte from its slots' low bits
__device__ __forceinline__ uint32_t x16_exp8(const uint4& w) {
  return (w.x & 1u) | ((w.x >> 15) & 2u) | ((w.y & 1u) << 2) | ((w.y >> 13) & 8u) | ((w.z & 1u) << 4) |
         ((w.z >> 11) & 32u) | ((w.w & 1u) << 6) | ((w.w >> 9) & 128u);
}

// values 4 h .. 4 h + 3 of a group (h = 0 or 1)
__device__ __forceinline__ float4 x16_unpack4(const uint4& w, int h) {
  const float s = ldexpf(1.0f / 32767.0f, (int)x16_exp8(w) - 125);
  const uint32_t p = h ? w.z : w.x, q = h ? w.w : w.y;
  // (int32)(slot << 16) >> 17 and (int32)slot >> 17: the signed 15-bit value
  return make_float4((float)((int32_t)(p << 16) >> 17) * s, (float)((int32_t)p >> 17) * s,
                     (float)((int32_t)(q << 16) >> 17) * s, (float)((int32_t)q >> 17) * s);
}

// all 8 values of a group
__device__ __forceinline__ void x16_unpack8(const uint4& w, float4& a, float4& b) {
  const float s = ldexpf(1.0f / 32767.0f, (int)x16_exp8(w) - 125);
  auto lo = [](uint32_t u) { return (float)((int32_t)(u << 16) >> 17); };
  auto hi = [](uint32_t u) { return (float)((int32_t)u >> 17); };
  a = make_float4(lo(w.x) * s, hi(w.x) * s, lo(w.y) * s, hi(w.y) * s);
  b = make_float4(lo(w.z) * s, hi(w.z) * s, lo(w.w) * s, hi(w.w) * s);
}

// The group holding column c of row `row` (n values per row) at base.
__device__ __forceinline__ uint4 x16_load8(const void* base, int64_t row, int64_t n, int64_t c) {
  return *(const uint4*)((const uint8_t*)base + (row * n + (c & ~(int64_t)7)) * 2);
}

// A lane's x16 stores down a group of 8 columns [c, c + 8) (c a multiple of
// 8): rows row, row + step, row + 2 step, ... of a row-major x16 matrix with
// n values per row, one 16-byte store per row; the row address advances by a
// constant stride instead of being multiplied out per row.
struct X16Rows8 {
  uint8_t* m;
  int64_t stride;
  __device__ __forceinline__ X16Rows8(void* base, int64_t n, int64_t row, int step, int64_t c) {
    m = (uint8_t*)base + (row * n + c) * 2;
    stride = n * step * 2;
  }
  __device__ __forceinline__ void store(float4 a, float4 b) const { *(uint4*)m = x16_pack8(a, b); }
  __device__ __forceinline__ void next() { m += stride; }
};

// Output format of a GEMM: fp32, a bf16 (hi, lo) pair, x16, or OUT_F16T:
// fp16 [rows][ldc] with one power-of-two scale per tile (the tile spans whole
// rows), the scale's exponent s written per row to GemmArgs::c_row_exp
// (stored value = true value * 2^s).
enum OutFmt { OUT_F32 = 0, OUT_HILO = 1, OUT_X16 = 2, OUT_F16T = 3 };
// Format of the weighted activation sums (the down GEMMs' input); HBAR_F16:
// fp16 rows of f values scaled by 2^exp (exp per row, in a separate array;
// one value for all of a token's fp16 rows, chosen so that their largest
// magnitude lands in [2^14, 2^15)).
enum HbarMode { HBAR_F32 = 0, HBAR_HILO = 1, HBAR_LO8 = 2, HBAR_F16 = 3 };

// ---------------------------------------------------------------- fp8 lo
// The low half of a bf16 (hi, lo) split only needs a few bits: where the
// anchor down weights come with an fp8 copy, the anchor activation sums are
// stored as bf16 hi plus an fp8 (OCP e4m3) lo with one power-of-two scale per
// 32 consecutive values (E8M0 exponent byte, value 2^(byte - 127)), and the
// anchor down GEMM multiplies the lo half with the block-scaled fp8 MFMA.
// Scale words: one uint32 per 64 values, bytes 0 and 1 the exponents of its
// two 32-value blocks, bytes 2 and 3 zero.

// E8M0 exponent byte for a block whose largest magnitude is amax: the block
// max lands in [128, 256), inside e4m3's normal range (max 448).
__device__ __forceinline__ uint32_t e8m0_for(float amax) {
  const int e = (int)((__float_as_uint(amax) >> 23) & 0xFF) - 127;  // floor(log2) for normal amax
  int b = e - 7 + 127;
  b = b < 1 ? 1 : b > 254 ? 254 : b;
  return (uint32_t)b;
}

// x * 2^(127 - b): the inverse of the block scale, exact.
__device__ __forceinline__ float e8m0_unscale(float x, uint32_t b) {
  return x * __uint_as_float((254u - b) << 23);
}

// fp32 -> OCP e4m3 byte, round to nearest even, for |x| <= 448 (the callers'
// block scaling guarantees it); values below 2^-6 become e4m3 subnormals.
__device__ __forceinline__ uint32_t f32_to_e4m3(float x) {
  const uint32_t u = __float_as_uint(x);
  const uint32_t sign = (u >> 24) & 0x80u;
  const float a = fabsf(x);
  uint32_t code;
  if (a < 0.015625f) {  // subnormal: multiples of 2^-9 (rounding up to 8 gives 2^-6, code 0x08)
    code = (uint32_t)__float2int_rn(a * 512.f);
  } else {
    const uint32_t v = __float_as_uint(a);
    const uint32_t r = v + 0x7FFFFu + ((v >> 20) & 1u);  // keep 3 mantissa bits, ties to even
    code = ((((r >> 23) & 0xFF) - 120u) << 3) | ((r >> 20) & 7u);
    code = code > 0x7Eu ? 0x7Eu : code;
  }
  return sign | code;
}

constexpr int kTokTile = 64;          // tokens per bucketing tile (one wavefront)
constexpr int kMaxLvl = LX_MAX_LEVELS + 1;  // anchor level + correction levels

// One GEMM tile: rows [row0, row0 + nrows) of the level's row list, all
// belonging to `node`, whose weights are at index `widx` of the weight arrays.
struct TileEntry {
  int32_t widx;
  int32_t row0;
  int32_t nrows;
  int32_t node;
};

// ---------------------------------------------------------------- bucketing
// GEMM tile tables built by the bucketing, one per tile height: the
// register-staged kernel, the large-tile kernel and the skinny kernel.
constexpr int kTabSmall = 0, kTabBig = 1, kTabSkinny = 2, kNumTab = 3;

struct BucketLevel {
  int32_t n_nodes;
  int32_t tile_bm[kNumTab];  // tile height of each table
  uint32_t tab_mask;         // bit b: table b is needed (built) at this level
  int32_t work_all;        // 1: every node does GEMM work (anchor level)
  const uint8_t* work_node;  // if set: node n does work iff work_node[n] != 0
                             // (the leaf level of a tree whose correction
                             // outputs are merged: a factor anywhere on the path)
  const int32_t* fac;      // validated factor index per node (-1 none)
  int32_t* hist;           // [n_nodes][n_tok_tiles], scanned in place
  int32_t* offsets;        // [n_nodes + 1]
  int32_t* row_token;      // [rows_max]
  int32_t* slot_row;       // [T * k]
  uint8_t* slot_flags;     // [T * k] bit0: first slot of its row, bit1: the row's
                           // node does work at this level (always at level 0)
  TileEntry* tiles[kNumTab];  // [tiles_max of the table]
  int32_t* n_tiles[kNumTab];  // [1] each
  uint32_t* split_cnt;        // [n_split_cnt] split-K arrival counters, zeroed
  int32_t n_split_cnt;        // here for the level's skinny GEMMs
};

// Router top-k fused into the first bucketing kernel: the logits of the
// router GEMM (final [T][E], or S split-K partial tiles, as for launch_topk)
// are turned into the ids and weights that the rest of the bucketing and
// the forward read (written to BucketArgs::ids / w, which are then outputs).
struct RouteIn {
  const float* logits;     // null: no fused router (ids and w are inputs)
  const float* part;
  int32_t S;
};

struct BucketArgs {
  int32_t T, k, E, L;      // L = number of correction levels
  int32_t n_tok_tiles;
  const int32_t* ids;      // [T * k]
  const float* w;          // [T * k] routing weights, or null (bucketing only)
  float* slot_wsum;        // [T * k] at the expert level: a distinct expert's first
                           // slot holds the sum of its slots' weights, others 0
  const int32_t* anc;      // [(L + 1) * E] ancestor per level, -1 = invalid expert
  uint32_t* flags;
  RouteIn route;
  BucketLevel lv[kMaxLvl];
};

struct PrepareArgs {
  int32_t E, L;
  int32_t n_nodes[kMaxLvl];            // n_nodes[0] = anchors
  int32_t n_factors[kMaxLvl];          // per correction level (index 0 unused)
  const int32_t* parent[kMaxLvl];      // parent[l] for l >= 1
  const int32_t* factor_of[kMaxLvl];   // factor_of[l] for l >= 1
  int32_t* anc;                        // out [(L + 1) * E]
  int32_t* fac[kMaxLvl];               // out, validated factor index (l >= 1)
  uint8_t* path_work;                  // out [E] (optional): 1 if a node on the
                                       // expert's path carries a factor
  uint32_t* flags;
};

hipError_t launch_prepare(const PrepareArgs& a, hipStream_t s);
hipError_t launch_bucket_hist(const BucketArgs& a, hipStream_t s);
// With a.route set: top-k of every token (ids and weights written to a.ids
// and a.w) and the histogram of every level, one workgroup per token tile.
hipError_t launch_bucket_hist_route(const BucketArgs& a, hipStream_t s);
hipError_t launch_bucket_scan(const BucketArgs& a, hipStream_t s);
hipError_t launch_bucket_place(const BucketArgs& a, hipStream_t s);
// Merged correction outputs of a tree (after placement): for every leaf
// row r of level L and every intermediate level l (1 <= l < L),
// leaf_row_map[l][r] = the level-l row of r's token and node.
struct LeafMapArgs {
  int32_t T, k, L;
  const int32_t* slot_row[kMaxLvl];
  const uint8_t* slot_flags[kMaxLvl];
  int32_t* leaf_row_map[kMaxLvl];
};
hipError_t launch_leaf_maps(const LeafMapArgs& a, hipStream_t s);
// Batches of 1..64 tokens: prepare + hist + scan + place in one workgroup.
bool bucket_small_ok(const BucketArgs& a);
hipError_t launch_bucket_small(const PrepareArgs& pa, const BucketArgs& a, hipStream_t s);

// ---------------------------------------------------------------- GEMM
// C[row, coloff[p] + n] = sum_k A[arow(row), akoff[p] + k] * B_p[widx][n][k]
// for the tiles of a row list; two weight "parts" share the A rows (e.g. the
// gate and up projections of one anchor).
struct GemmArgs {
  const TileEntry* tiles;
  const int32_t* n_tiles;
  const void* A;
  int64_t lda;
  const int32_t* a_rows;     // gather map row -> A row, or null (identity)
  int32_t a_koff[2];
  const void* B[2];
  int64_t b_stride[2];       // elements between consecutive weight indices
  int32_t ncols[2];          // output columns of each part
  int32_t K;                 // reduction length of A
  int32_t Kb;                // row length of W (0: K). When Kb < K the weight
                             // columns repeat with period Kb: A = [A_hi | A_lo]
                             // against the same W, i.e. C = (A_hi + A_lo) W^T
  float* C;
  int64_t ldc;
  int32_t c_coloff[2];
  // fp8 lo half (anchor down projection, K = 2 Kb, A rows without a gather
  // map): A row = [bf16 hi (Kb) | fp8 lo (Kb bytes) at byte a_lo8_off |
  // scale words (Kb / 64) at byte a_sc_off], row pitch 2 lda bytes; the
  // weights' fp8 copy and scale words:
  const uint8_t* b8;         // [widx][n][Kb]
  const uint32_t* bsc;       // [widx][n][Kb / 64]
  int32_t a_lo8_off, a_sc_off;
  // split-K (skinny kernel only): when the routed tiles give fewer work
  // items than split_cap, each item's weight slabs are divided over up to
  // split_cap / items workgroups. Each writes its fp32 partial tile to its
  // slot of part ([split_cap][kSkinnyBM][kSkinnyBN]); the last of an item's
  // workgroups to arrive (per-item counters cnt, zero on entry and left zero)
  // adds the partials in split order and writes C. Null part: no split.
  float* part;
  uint32_t* cnt;
  int32_t split_cap;
  // split_force > 1: split into that many pieces before normalisation (the
  // caller's count, at most the weight slabs / kSplitMinSlabs; the splits
  // actually made are skinny_splits(weight slabs, split_force)); with defer
  // set, every split only writes its partial tile to its slot of part and
  // the consumer of C adds the slots (no counters).
  int32_t split_force;
  int32_t defer;
  // tiles == null: implicit tiles of kSkinnyBM consecutive rows over
  // dense_rows rows of A (identity row map, weight index 0)
  int32_t dense_rows;
  // large-tile kernel: when widx_anc is set, a tile's weight index is
  // widx_fac[widx_anc[tile node]] (the factor of the tile node's ancestor at
  // another level; below 0: the tile is skipped) instead of its own
  const int32_t* widx_anc;
  const int32_t* widx_fac;
  int32_t widx_own1;         // with widx_anc: part 1 uses the tile's own widx
  // fp16 operands (launch_gemm_f16): A row r is scaled by 2^a_row_exp[r],
  // weight matrix i of part 0 by 2^b_exp[i], of part 1 by 2^b_exp1[i] (null:
  // b_exp)
  const int32_t* a_row_exp;
  const int32_t* b_exp;
  const int32_t* b_exp1;
  // OUT_F16T: per-row scale exponents of the output
  int32_t* c_row_exp;
};

enum AMode { A_BF16 = 0, A_F32_HILO = 1 };

// Grid: x = upper bound on tiles, y = BN-tiles of part 0 then of part 1.
int gemm_bm(lx_dtype dt);
int gemm_bn(lx_dtype dt);
hipError_t launch_gemm(const GemmArgs& g, lx_dtype dt, AMode am, int grid_x, hipStream_t s);

// Large-tile kernel (BM x BN tiles, direct HBM->LDS loads). Applicable when A
// is bf16, K and Kb are multiples of 64, the parts either share A columns or
// the part boundary is a multiple of BN, and A's element count fits in 31
// bits. fp32 and x16 output is written at columns [0, ncols[0] + ncols[1]) of
// C (the parts adjacent; ldc in values, an x16 row is 2 ldc bytes); bf16
// (hi, lo) output writes part p's hi values at columns base_p + c and lo
// values at base_p + ncols[p] + c, base_0 = 0, base_1 = 2 ncols[0] (ldc in
// bf16 elements).
constexpr int kBigBM = 256;
static_assert((kBigBM & (kBigBM - 1)) == 0, "tile heights are powers of two (bucketing shifts)");
bool gemm_big_ok(const GemmArgs& g, int bn, int64_t a_rows_total);
// The fp8-lo variant (256 x 256 tiles) of the large-tile kernel: hi slabs as
// above, lo slabs from the fp8 copies with the block-scaled fp8 MFMA.
bool gemm_lo8_ok(const GemmArgs& g, int64_t a_rows_total);
hipError_t launch_gemm_lo8(const GemmArgs& g, int ofmt, int grid_tiles, hipStream_t s);
// The fp16 variant (256 x bn tiles, K = Kb): A and W fp16 with their
// power-of-two scales (GemmArgs::a_row_exp, b_exp, b_exp1), undone exactly in
// the epilogue (x16 or fp32 output) or carried into the output's row
// exponents (OUT_F16T).
bool gemm_f16_ok(const GemmArgs& g, int bn, int ofmt, int64_t a_rows_total);
hipError_t launch_gemm_f16(const GemmArgs& g, int bn, int ofmt, int grid_tiles, hipStream_t s);
// Two independent fp16 products with 256 x 256 tiles in one persistent launch
// (g0's work items, then g1's: one schedule and one tail for both); output
// formats x16 for g0 and x16 or OUT_F16T for g1, each product as accepted by
// gemm_f16_ok.
hipError_t launch_gemm_f16_pair(const GemmArgs& g0, int grid_tiles0, const GemmArgs& g1, int ofmt1,
                                int grid_tiles1, hipStream_t s);
// Weights [n][per] bf16 -> fp16 [n][per] scaled per matrix i by 2^exps[i]
// (exps[i] puts the matrix's largest magnitude in [2^14, 2^15); 0 for an
// all-zero matrix).
hipError_t launch_convert_f16(const void* w, int n, int64_t per, void* w16, int32_t* exps, hipStream_t s);
// Zero-padded copy [n][rows][cols] bf16 -> [n][rows_out][cols_out]: fp16 as
// launch_convert_f16 (exps non-null; the exponents of the unpadded matrices)
// or bf16 (exps null).
hipError_t launch_copy_pad(const void* w, int n, int rows, int cols, int rows_out, int cols_out, void* out,
                           int32_t* exps, hipStream_t s);
// Weights [n][rows][cols] bf16 -> fp8 copy [n][rows][cols] and scale words
// [n][rows][cols / 64] (cols a multiple of 64).
hipError_t launch_quantize_f8(const void* w, int64_t n_rows, int cols, uint8_t* w8, uint32_t* sc, hipStream_t s);
hipError_t launch_gemm_big(const GemmArgs& g, int bm, int bn, int ofmt, int grid_tiles,
                           hipStream_t s);

// Segmented large-tile GEMM (256 x 256 tiles, x16 output): the correction
// products of several tree levels that land on the same output rows, as one
// GEMM whose K is the concatenation of the levels' operands:
//   C[row] = sum over segments s of A_s[map_s(row)] * W_s[widx_s]^T
// over the tiles of the leaf level (p.tiles, p.n_tiles, p.ncols, p.C,
// p.ldc; the other GemmArgs fields are unused). Segment s is active for a
// tile when its factor index widx_s (the tile's own widx for the leaf
// segment, else the validated factor of the leaf's ancestor at the
// segment's level) is >= 0; rank a multiple of 64. bf16 segments: K is 2
// rank (hi then lo against the same weight columns). fp16 segments (f16 set):
// K is rank, A row a carries 2^a_exp[a] and weight matrix i of part p
// 2^b_exp[p][i]; the accumulators are rescaled row by row when the segment
// changes, so each level's products are added at the true scale. An A row
// index below 0 in a segment's map selects that segment's zero row.
struct SegDesc {
  const void* A;           // bf16 or fp16 [rows][lda]; part 1 starts at column akoff1
  int64_t lda;             // elements
  const int32_t* map;      // output row -> A row (null: identity)
  int32_t zero_row;        // A row of zeros used for map entries < 0
  int32_t rank;            // weight row length
  int32_t akoff1;
  int32_t anc_off;         // level * E into SegArgs::anc; -1: the tile's widx
  const int32_t* fac;      // validated factor index per node of the level
  const void* B[2];        // weights of the two parts [widx][n][rank]
  int64_t b_stride[2];
  const int32_t* a_exp;    // fp16 segments: row exponents of A
  const int32_t* b_exp[2]; // fp16 segments: exponents of the weight matrices
  int32_t a_col0;          // first A column of this segment's operand
};
struct SegArgs {
  int32_t nseg;
  int32_t f16;             // fp16 segments
  int32_t ngrp;            // consecutive column tiles per work item (set by launch_gemm_seg)
  const int32_t* anc;      // [(L + 1) * E] ancestor of each expert per level
  SegDesc s[LX_MAX_LEVELS];
};
bool gemm_seg_ok(const GemmArgs& g, const SegArgs& sa, int64_t out_rows);
hipError_t launch_gemm_seg(const GemmArgs& g, const SegArgs& sa, int grid_tiles, hipStream_t s);

// Skinny kernel for levels with few rows per node (decode-sized batches):
// 32-row tiles, 64 output columns per workgroup, a 4-stage LDS ring and
// several workgroups per compute unit, so weight streaming is limited by
// HBM rather than by MFMA work on padding rows. Same operand conventions and
// applicability as the large-tile kernel (with bn = kSkinnyBN).
constexpr int kSkinnyBM = 32, kSkinnyBN = 64;
static_assert((kSkinnyBM & (kSkinnyBM - 1)) == 0, "tile heights are powers of two (bucketing shifts)");
// Split-K: partial-tile slots per level (three 48 KB-LDS workgroups per
// compute unit on 256 compute units) and the fewest weight slabs (64 K
// values) a split covers.
constexpr int kSplitCap = 768, kSplitMinSlabs = 4;
// Splits made of nkw weight slabs asked to split s ways: pieces of
// ceil(nkw / s) slabs, none empty.
__host__ __device__ inline int skinny_splits(int nkw, int s) {
  if (s <= 1) return 1;
  const int cw = (nkw + s - 1) / s;
  return (nkw + cw - 1) / cw;
}
// Workgroups the skinny kernel launches for a product with at most
// items_max work items (all splits of all items fit when splitting).
int skinny_grid(const GemmArgs& g, int64_t items_max);
hipError_t launch_gemm_skinny(const GemmArgs& g, int ofmt, int grid_tiles, hipStream_t s);
// Up to kSkinnyMaxProblems independent skinny GEMMs in one launch.
constexpr int kSkinnyMaxProblems = 1 + LX_MAX_LEVELS;
struct SkinnyBatch {
  GemmArgs g[kSkinnyMaxProblems];
  int32_t ntn[kSkinnyMaxProblems];
  int32_t ofmt[kSkinnyMaxProblems];  // OutFmt
  int32_t base[kSkinnyMaxProblems + 1];  // first workgroup of each problem
  int32_t n;
};
hipError_t launch_gemm_skinny_batch(const GemmArgs* g, const int* ofmt, const int* grid_tiles, int n,
                                    hipStream_t s);

// ---------------------------------------------------------------- elementwise
struct TokenArgs {
  int32_t T, k, E, L, d, f;
  const int32_t* slot_row[kMaxLvl];
  const uint8_t* slot_flags[kMaxLvl];
  const float* slot_wsum;
  const float* gu0;                    // [rows0][2f] anchor gate|up
  const float* dgu[kMaxLvl];           // [rows_l][2f] correction gate|up (l >= 1)
  int32_t x16[kMaxLvl];                // level l's gate|up and down rows are x16
                                       // (else fp32)
  float* hbar[kMaxLvl];                // weighted activation sums, rows of 4f bytes:
                                       // HBAR_F32 fp32 [f]; HBAR_HILO bf16 hi [f] then
                                       // lo [f]; HBAR_LO8 bf16 hi [f], fp8 lo [f bytes],
                                       // scale words [f / 64]
  int32_t hbar_mode[kMaxLvl];
  int32_t* hbar_exp[kMaxLvl];          // HBAR_F16: per-row scale exponents
  const float* y[kMaxLvl];             // [rows_l][d] down outputs per level
  int32_t merged;                      // 1: the gate|up and down corrections of
                                       // levels 1 .. L-1 are folded into level
                                       // L's rows (their dgu / y are not read)
  void* out;
  lx_dtype out_dtype;
};

// ---------------------------------------------------------------- router
// Top-k over router logits: logits [T][E] fp32 (S == 1), or the S partial
// tiles per (32-row tile, 64-column tile) item that a deferred split-K
// skinny GEMM left in part (slot (item * S + split), layout [wavefront][row]
// [32 columns]). 1 <= k <= min(E, LX_MAX_K), E <= kRouteMaxE.
constexpr int kRouteMaxE = 512;
hipError_t launch_topk(const float* logits, const float* part, int S, int T, int E, int k, int32_t* ids,
                       float* weights, hipStream_t s);

// ---------------------------------------------------------------- clustering
// Router profiling counts and the NPMI distance (fire [E], pair [E][E]
// symmetric, dist [E][E] fp64), and frequency-seeded k-medoids (E <=
// kClusterMaxE, protected experts as a bit mask).
constexpr int kClusterMaxE = 1024;
struct ProtMask {
  uint32_t bits[kClusterMaxE / 32];
};
hipError_t launch_coact(const int32_t* ids, int N, int k, int E, uint32_t* fire, uint32_t* pair, double* dist,
                        hipStream_t s);
hipError_t launch_kmedoids(const double* dist, const uint32_t* fire, int E, int C, const ProtMask& pm, int P,
                           int max_iter, int32_t* cluster_of, int32_t* factor_of, int32_t* dominant,
                           int32_t* iterations, hipStream_t s);

// ---------------------------------------------------------------- stage 3
// Alignment cost [f][f] fp64 of two experts (workspace 2 f (3d + 1)
// doubles); rank-r factors of the aligned residual by a randomized SVD with
// sketch width l = r + p <= 128 (workspace lowrank_ws_doubles).
hipError_t launch_align_cost(const void* dg, const void* du, const void* dd, const void* mg, const void* mu,
                             const void* md, int bf16, int f, int d, double* cost, double* ws, hipStream_t s);
size_t lowrank_ws_doubles(int rows, int cols, int l);
// activation-weighted fit: the same randomized solver on M = R Xp^T, Xp =
// [X; sqrt(damp) I] with np = n (+ cols when damp > 0) rows
size_t weighted_ws_doubles(int rows, int cols, int np, int l);
hipError_t launch_weighted(const void* wd, const void* wm, int bf16, int rows, int cols, const int32_t* perm, int axis,
                           const void* x, int x_bf16, int n, double damp, int r, int l, int q, const double* omega,
                           float* A, float* B, double* sigma, double* ws, hipStream_t s);
hipError_t launch_lowrank(const void* wd, const void* wm, int bf16, int rows, int cols, const int32_t* perm, int axis,
                          int r, int l, int q, const double* omega, float* A, float* B, double* sigma, double* ws,
                          hipStream_t s);

hipError_t launch_swiglu_reduce(const TokenArgs& a, hipStream_t s);
hipError_t launch_combine(const TokenArgs& a, hipStream_t s);

}  // namespace lx

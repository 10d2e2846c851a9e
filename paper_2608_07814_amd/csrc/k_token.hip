// Per-token kernels: SwiGLU with the amortized weighted reduction, and the
// deterministic combine. SwiGLU runs one workgroup per (token, 256-neuron
// chunk), combine one per token; every thread owns 4 consecutive neurons
// (SwiGLU) or output columns (combine), so every access is one vector: 16
// bytes of fp32, or an 8-byte word and an exponent byte of x16 (the format
// of the gate|up and down rows written by the bf16 GEMM kernels).
//
// For a token t with selected experts e_j (j ascending), every tree level l
// has one row per distinct level-l node among the e_j (from the bucketing,
// which also marks each slot's first-of-row and has-work bits and stores each
// distinct expert's summed routing weight on its first slot).
//   swiglu_reduce: for each distinct expert of t
//       g = anchor gate row + sum over levels of the node's gate correction,
//       u likewise, h = w * silu(g) * u;
//     every level-l row of t then gets hbar_l[row] = sum of the h of the
//     experts under it, in slot order (the anchor level always, correction
//     levels where the node carries a factor). By linearity the down
//     projections then run once per row (Sec. 5.1 amortized forward).
//   combine: out[t] = sum over levels, over t's rows of the level, of that
//     level's down-projection output row, in a fixed order (level, then slot)
//     with no atomics, so the result is bit-reproducible.
#include "lx_internal.h"

#include <type_traits>

namespace lx {
namespace {

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

struct TokenMeta {
  int row[kMaxLvl][LX_MAX_K];
  unsigned char fl[kMaxLvl][LX_MAX_K];
  float w[LX_MAX_K];
};

// Threads 0..k-1 load the slot metadata of token t; caller synchronizes.
__device__ inline void token_meta(const TokenArgs& a, int t, TokenMeta& m) {
  const int j = threadIdx.x;
  if (j >= a.k) return;
  const int64_t s = (int64_t)t * a.k + j;
  for (int l = 0; l <= a.L; ++l) {
    m.row[l][j] = a.slot_row[l][s];
    m.fl[l][j] = a.slot_flags[l][s];
  }
  m.w[j] = a.slot_wsum[s];
}

__device__ __forceinline__ float4 ld4(const float* p) { return *(const float4*)p; }
// 4 consecutive values at column c of row `row` (row length ld values) of an
// fp32 or x16 matrix.
__device__ __forceinline__ float4 ldrow4(const float* base, bool x16, int64_t row, int64_t ld, int c) {
  if (x16) return x16_unpack4(x16_load8(base, row, ld, c), (c >> 2) & 1);
  return *(const float4*)(base + row * ld + c);
}
__device__ __forceinline__ void add4(float4& a, const float4& b) {
  a.x += b.x;
  a.y += b.y;
  a.z += b.z;
  a.w += b.w;
}
__device__ __forceinline__ float silu_mul(float g, float u) { return g / (1.f + expf(-g)) * u; }

// hbar row segment (4 neurons at column c), rows of 4f bytes: fp32; or a
// bf16 (hi, lo) pair (hi half, lo half); or bf16 hi, fp8 lo and one E8M0
// scale per 32 neurons (HBAR_LO8). HBAR_LO8 reduces the block maximum over
// the 8 lanes that hold a 32-neuron block, so those lanes must execute the
// call together (columns 4 per lane, blocks aligned to 32 columns).
__device__ __forceinline__ void hbar_store(void* base, int mode, int row, int c, int f, float4 v) {
  if (mode == HBAR_F32) {
    *(float4*)((float*)base + (int64_t)row * f + c) = v;
    return;
  }
  __bf16* hb = (__bf16*)base + (int64_t)row * 2 * f;
  bf16x4 hi;
  hi[0] = (__bf16)v.x;
  hi[1] = (__bf16)v.y;
  hi[2] = (__bf16)v.z;
  hi[3] = (__bf16)v.w;
  *(bf16x4*)(hb + c) = hi;
  const float l0 = v.x - (float)hi[0], l1 = v.y - (float)hi[1], l2 = v.z - (float)hi[2], l3 = v.w - (float)hi[3];
  if (mode == HBAR_HILO) {
    bf16x4 lo;
    lo[0] = (__bf16)l0;
    lo[1] = (__bf16)l1;
    lo[2] = (__bf16)l2;
    lo[3] = (__bf16)l3;
    *(bf16x4*)(hb + f + c) = lo;
    return;
  }
  float amax = fmaxf(fmaxf(fabsf(l0), fabsf(l1)), fmaxf(fabsf(l2), fabsf(l3)));
  amax = fmaxf(amax, __shfl_xor(amax, 1, 64));
  amax = fmaxf(amax, __shfl_xor(amax, 2, 64));
  amax = fmaxf(amax, __shfl_xor(amax, 4, 64));
  const uint32_t be = e8m0_for(amax);
  uint8_t* const rb = (uint8_t*)base + (int64_t)row * 4 * f;
  *(uint32_t*)(rb + 2 * f + c) = f32_to_e4m3(e8m0_unscale(l0, be)) | (f32_to_e4m3(e8m0_unscale(l1, be)) << 8) |
                                 (f32_to_e4m3(e8m0_unscale(l2, be)) << 16) |
                                 (f32_to_e4m3(e8m0_unscale(l3, be)) << 24);
  // the first lane of each 64-neuron slab writes the slab's scale word
  const uint32_t be_next = __shfl_down(be, 8, 64);
  if ((c & 63) == 0) *(uint32_t*)(rb + 3 * f + (c >> 6) * 4) = be | (be_next << 8);
}
// HBAR_F16: a token's fp16 rows share one power-of-two scale 2^sh, chosen
// from the largest magnitude over all of the token's fp16 rows (the rows are
// partial sums of the same activations, within a few binades of each other,
// and fp16 keeps 11 bits of every value within 29 binades of the maximum).
// Every thread of the workgroup holds 4 values of every row and calls this
// with its own maximum; returns sh (largest magnitude in [2^14, 2^15)).
constexpr int kMaxWaves = 16;
__device__ __forceinline__ int f16_token_shift(float m) {
  __shared__ float s_red[kMaxWaves];
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, 64));
  if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6] = m;
  __syncthreads();
  float rm = 0.f;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) rm = fmaxf(rm, s_red[i]);
  __syncthreads();  // s_red is reused by the next token
  int sh = 0;
  if (rm > 0.f) {
    sh = 14 - ((int)((__float_as_uint(rm) >> 23) & 0xFF) - 127);
    sh = sh < -100 ? -100 : sh > 100 ? 100 : sh;
  }
  return sh;
}
// The row's 4 values at column c as fp16 scaled by 2^sh; thread 0 records sh.
__device__ __forceinline__ void hbar_store_f16(void* base, int32_t* exps, int row, int c, int f, float4 v, int sh) {
  typedef _Float16 h4 __attribute__((ext_vector_type(4)));
  h4 q;
  q[0] = (_Float16)ldexpf(v.x, sh);
  q[1] = (_Float16)ldexpf(v.y, sh);
  q[2] = (_Float16)ldexpf(v.z, sh);
  q[3] = (_Float16)ldexpf(v.w, sh);
  *(h4*)((_Float16*)base + (int64_t)row * f + c) = q;
  if (threadIdx.x == 0) exps[row] = sh;
}

constexpr int kTokThr = 64, kTokCols = 4 * kTokThr;
constexpr int kSlotGroups = 16;  // SwiGLU: up to 16 slots processed side by side

// Phase 1: every distinct expert of token t (first slot of its leaf row)
// gets h = w * silu(g) * u for this thread's 4 neurons, one slot group per
// slot, all loads in flight together; h goes to LDS. Phase 2: each row of
// each level is summed in slot order by the thread group of its first slot
// and stored once (no read-modify-write of the sums in memory).
__global__ __launch_bounds__(kTokThr * kSlotGroups) void k_swiglu_reduce(TokenArgs a) {
  __shared__ TokenMeta m;
  extern __shared__ float4 s_h[];  // [k][kTokThr]
  const int t = blockIdx.x;
  token_meta(a, t, m);
  __syncthreads();
  const int k = a.k, L = a.L, f = a.f;
  const int64_t ld = 2 * (int64_t)f;
  const int lane = threadIdx.x % kTokThr, sg = threadIdx.x / kTokThr;
  const int nsg = blockDim.x / kTokThr;
  const int c = (blockIdx.y * kTokThr + lane) * 4;
  const bool colok = c < f;
  for (int j = sg; j < k && colok; j += nsg) {
    if (!(m.fl[L][j] & 1)) continue;  // not the first slot of a valid expert
    const bool f0 = a.x16[0] != 0;
    float4 g = ldrow4(a.gu0, f0, m.row[0][j], ld, c), u = ldrow4(a.gu0, f0, m.row[0][j], ld, f + c);
    for (int l = 1; l <= L; ++l) {
      if (!(m.fl[l][j] & 2) || (a.merged && l < L)) continue;
      const bool fl = a.x16[l] != 0;
      add4(g, ldrow4(a.dgu[l], fl, m.row[l][j], ld, c));
      add4(u, ldrow4(a.dgu[l], fl, m.row[l][j], ld, f + c));
    }
    const float w = m.w[j];
    s_h[j * kTokThr + lane] = make_float4(w * silu_mul(g.x, u.x), w * silu_mul(g.y, u.y),
                                          w * silu_mul(g.z, u.z), w * silu_mul(g.w, u.w));
  }
  __syncthreads();
  if (!colok) return;
  for (int j0 = sg; j0 < k; j0 += nsg) {
    for (int l = 0; l <= L; ++l) {
      const unsigned char fl0 = m.fl[l][j0];
      if ((fl0 & 3) != 3) continue;  // j0 starts a level-l row that does work
      if (a.merged && l > 0 && l < L) continue;  // folded into the leaf rows
      const int r = m.row[l][j0];
      float4 hs = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int j = j0; j < k; ++j)
        if (m.row[l][j] == r && (m.fl[L][j] & 1)) add4(hs, s_h[j * kTokThr + lane]);
      hbar_store(a.hbar[l], a.hbar_mode[l], r, c, f, hs);
    }
  }
}

// Combine, one workgroup per token (whole output rows, so every row of the
// token is read as one contiguous stretch): wavefront 0 lists the token's rows
// to sum (first slot of a row that does work) in (level, slot) order with a
// ballot compaction; then every thread sums its 4 columns over that list, 16
// row loads in flight at a time, adding in list order. Rows are fp32 or x16
// per level; s_rows holds each row's first byte and s_x16 its format.
constexpr int kCombMaxThr = 512;
__global__ __launch_bounds__(kCombMaxThr) void k_combine(TokenArgs a) {
  __shared__ const uint8_t* s_rows[kMaxLvl * LX_MAX_K];
  __shared__ uint8_t s_x16[kMaxLvl * LX_MAX_K];
  __shared__ int s_n;
  const int t = blockIdx.x;
  const int k = a.k, L = a.L, d = a.d;
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    const int nq = (L + 1) * k;
    int base = 0;
    for (int q0 = 0; q0 < nq; q0 += 64) {
      const int q = q0 + lane;
      bool take = false, x16 = false;
      const uint8_t* ptr = nullptr;
      if (q < nq) {
        const int l = q / k, j = q - l * k;
        const int64_t sl = (int64_t)t * k + j;
        const int row = a.slot_row[l][sl];  // loaded alongside the flags
        if ((a.slot_flags[l][sl] & 3) == 3 && !(a.merged && l > 0 && l < L)) {
          take = true;
          x16 = a.x16[l] != 0;
          ptr = (const uint8_t*)a.y[l] + (int64_t)row * d * (x16 ? 2 : 4);
        }
      }
      const uint64_t bal = __ballot(take);
      if (take) {
        const int at = base + __popcll(bal & ((1ull << lane) - 1));
        s_rows[at] = ptr;
        s_x16[at] = x16 ? 1 : 0;
      }
      base += __popcll(bal);
    }
    if (lane == 0) s_n = base;
  }
  __syncthreads();
  const int n = s_n;
  for (int c = threadIdx.x * 4; c < d; c += blockDim.x * 4) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int b = 0; b < n; b += 16) {
      float4 v[16];
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (b + i < n)
          v[i] = s_x16[b + i] ? x16_unpack4(*(const uint4*)(s_rows[b + i] + (c & ~7) * 2), (c >> 2) & 1)
                              : *(const float4*)(s_rows[b + i] + c * 4);
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (b + i < n) add4(acc, v[i]);
    }
    if (a.out_dtype == LX_F32) {
      *(float4*)((float*)a.out + (int64_t)t * d + c) = acc;
    } else {
      bf16x4 o;
      o[0] = (__bf16)acc.x;
      o[1] = (__bf16)acc.y;
      o[2] = (__bf16)acc.z;
      o[3] = (__bf16)acc.w;
      *(bf16x4*)((uint16_t*)a.out + (int64_t)t * d + c) = o;
    }
  }
}

// Fast paths for k <= 8 slots and NL <= 2 correction levels (the flat layer
// and the two-level tree): one workgroup per (token, column block) and no
// LDS or barriers. The token's slot metadata is read with wavefront-uniform
// (scalar) loads, every thread issues the loads of all its slots at once,
// and the sums run over registers in the same order as the general kernels.
constexpr int kFastK = 8, kFastL = 2, kFastThr = 256;

// Slot metadata of token t for slots j < kFastK (rows and flags per level,
// summed weights): lane j of every wavefront loads slot j, then each value is
// broadcast from its lane, so the results are wavefront-uniform (absent
// slots: row -1, flags 0).
template <int NL>
__device__ __forceinline__ void token_meta_fast(const TokenArgs& a, int t, int (&row)[NL + 1][kFastK],
                                                int (&fl)[NL + 1][kFastK], float (&w)[kFastK]) {
  const int lane = threadIdx.x & 63;
  const bool on = lane < a.k;
  const int64_t s = (int64_t)t * a.k + lane;
  int rv[NL + 1], fv[NL + 1];
#pragma unroll
  for (int l = 0; l <= NL; ++l) {
    rv[l] = on ? a.slot_row[l][s] : -1;
    fv[l] = on ? a.slot_flags[l][s] : 0;
  }
  const float wv = on ? a.slot_wsum[s] : 0.f;
#pragma unroll
  for (int j = 0; j < kFastK; ++j) {
#pragma unroll
    for (int l = 0; l <= NL; ++l) {
      row[l][j] = __builtin_amdgcn_readlane(rv[l], j);
      fl[l][j] = __builtin_amdgcn_readlane(fv[l], j);
    }
    w[j] = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, wv), j));
  }
}

// Raw row segment (4 values at column c; x16: the 8-value group holding
// them): loaded in one pass, converted in a later one, so every load of a
// thread is in flight before the first use.
template <bool X16>
struct Raw4 {
  using T = typename std::conditional<X16, uint4, float4>::type;
  T v;
};
template <bool X16>
__device__ __forceinline__ Raw4<X16> ldraw(const float* base, int64_t row, int64_t ld, int c) {
  Raw4<X16> r;
  if constexpr (X16)
    r.v = x16_load8(base, row, ld, c);
  else
    r.v = *(const float4*)(base + row * ld + c);
  return r;
}
// Conversion in the arithmetic pass (c: the column the segment was loaded
// at). x16 words go through an empty asm first: a row that is loaded only
// under a condition is otherwise merged with the skipped path's placeholder
// after the unpacking's first operations, which the compiler then performs in
// the load branch, right after the load (and waits for it there).
template <bool X16>
__device__ __forceinline__ float4 cvt(Raw4<X16> r, int c) {
  if constexpr (X16) {
    asm volatile("" : "+v"(r.v.x), "+v"(r.v.y), "+v"(r.v.z), "+v"(r.v.w));
    return x16_unpack4(r.v, (c >> 2) & 1);
  } else {
    return r.v;
  }
}

template <int NL, bool X16>
__global__ __launch_bounds__(kFastThr) void k_swiglu_fast(TokenArgs a) {
  const int t = blockIdx.x, k = a.k, f = a.f;
  const int c = (blockIdx.y * blockDim.x + threadIdx.x) * 4;
  if (c >= f) return;
  const int64_t ld = 2 * (int64_t)f;
  int row[NL + 1][kFastK], fl[NL + 1][kFastK];
  float w[kFastK];
  token_meta_fast<NL>(a, t, row, fl, w);
  const bool merged = a.merged != 0;
  // loads of every distinct expert's gate|up rows, then h = w silu(g) u
  Raw4<X16> gv[kFastK][NL + 1], uv[kFastK][NL + 1];
#pragma unroll
  for (int j = 0; j < kFastK; ++j) {
    if (!(fl[NL][j] & 1)) continue;
    gv[j][0] = ldraw<X16>(a.gu0, row[0][j], ld, c);
    uv[j][0] = ldraw<X16>(a.gu0, row[0][j], ld, f + c);
#pragma unroll
    for (int l = 1; l <= NL; ++l) {
      if (!(fl[l][j] & 2) || (merged && l < NL)) continue;
      gv[j][l] = ldraw<X16>(a.dgu[l], row[l][j], ld, c);
      uv[j][l] = ldraw<X16>(a.dgu[l], row[l][j], ld, f + c);
    }
  }
  float4 h[kFastK];
#pragma unroll
  for (int j = 0; j < kFastK; ++j) {
    h[j] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (!(fl[NL][j] & 1)) continue;
    float4 g = cvt<X16>(gv[j][0], c), u = cvt<X16>(uv[j][0], f + c);
#pragma unroll
    for (int l = 1; l <= NL; ++l) {
      if (!(fl[l][j] & 2) || (merged && l < NL)) continue;
      add4(g, cvt<X16>(gv[j][l], c));
      add4(u, cvt<X16>(uv[j][l], f + c));
    }
    h[j] = make_float4(w[j] * silu_mul(g.x, u.x), w[j] * silu_mul(g.y, u.y), w[j] * silu_mul(g.z, u.z),
                       w[j] * silu_mul(g.w, u.w));
  }
  // each level-l row that does work: the sum of its experts' h in slot order
  // (merged trees: the intermediate levels' down products run on the leaf
  // rows' sums, so only the anchor and leaf levels are stored)
  auto row_sum = [&](int l, int j0) {
    float4 hs = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int j = j0; j < kFastK; ++j)
      if (row[l][j] == row[l][j0] && (fl[NL][j] & 1)) add4(hs, h[j]);
    return hs;
  };
  auto stored = [&](int l, int j0) { return (fl[l][j0] & 3) == 3 && !(merged && l > 0 && l < NL); };
  // fp16 rows: one scale for the token (whole rows per workgroup: see the
  // launch), from the largest magnitude over its fp16 rows
  bool any16 = false;
#pragma unroll
  for (int l = 0; l <= NL; ++l) any16 |= a.hbar_mode[l] == HBAR_F16;
  int sh = 0;
  if (any16) {
    float m = 0.f;
#pragma unroll
    for (int l = 0; l <= NL; ++l)
#pragma unroll
      for (int j0 = 0; j0 < kFastK; ++j0) {
        if (!stored(l, j0) || a.hbar_mode[l] != HBAR_F16) continue;
        const float4 hs = row_sum(l, j0);
        m = fmaxf(m, fmaxf(fmaxf(fabsf(hs.x), fabsf(hs.y)), fmaxf(fabsf(hs.z), fabsf(hs.w))));
      }
    sh = f16_token_shift(m);
  }
#pragma unroll
  for (int l = 0; l <= NL; ++l)
#pragma unroll
    for (int j0 = 0; j0 < kFastK; ++j0) {
      if (!stored(l, j0)) continue;
      const float4 hs = row_sum(l, j0);
      if (a.hbar_mode[l] == HBAR_F16)
        hbar_store_f16(a.hbar[l], a.hbar_exp[l], row[l][j0], c, f, hs, sh);
      else
        hbar_store(a.hbar[l], a.hbar_mode[l], row[l][j0], c, f, hs);
    }
}

// x16 gate|up rows and fp16 activation sums on every stored level, 8
// columns per thread: one 16-byte load (an x16 group) per row half; whole rows per
// workgroup (threads past f / 8 only join the token's scale reduction).
// Same sums, in the same order, as k_swiglu_fast.
template <int NL, bool MERGED>
__global__ __launch_bounds__(kFastThr) void k_swiglu_x16w(TokenArgs a) {
  const int t = blockIdx.x, f = a.f;
  const int c = threadIdx.x * 8;
  const bool act = c < f;
  const int64_t ld = 2 * (int64_t)f;  // values per gate|up row
  int row[NL + 1][kFastK], fl[NL + 1][kFastK];
  float w[kFastK];
  token_meta_fast<NL>(a, t, row, fl, w);
  constexpr bool merged = MERGED;  // (a.merged, as a template argument)
  typedef uint4 Raw8;  // one x16 group
  auto ld8 = [&](const float* base, int r, int col) {
    return *(const uint4*)((const uint8_t*)base + ((int64_t)r * ld + col) * 2);
  };
  auto add8 = [&](float4 (&acc)[2], const Raw8& v) {
    float4 va, vb;
    x16_unpack8(v, va, vb);
    add4(acc[0], va);
    add4(acc[1], vb);
  };
  auto live = [&](int l, int j) { return (fl[l][j] & 2) && !(merged && l < NL); };
  Raw8 gv[kFastK][NL + 1], uv[kFastK][NL + 1];
#pragma unroll
  for (int j = 0; j < kFastK; ++j) {
    if (!act || !(fl[NL][j] & 1)) continue;
    gv[j][0] = ld8(a.gu0, row[0][j], c);
    uv[j][0] = ld8(a.gu0, row[0][j], f + c);
#pragma unroll
    for (int l = 1; l <= NL; ++l) {
      if (!live(l, j)) continue;
      gv[j][l] = ld8(a.dgu[l], row[l][j], c);
      uv[j][l] = ld8(a.dgu[l], row[l][j], f + c);
    }
  }
  float4 h[kFastK][2];
#pragma unroll
  for (int j = 0; j < kFastK; ++j) {
    h[j][0] = h[j][1] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (!act || !(fl[NL][j] & 1)) continue;
    float4 g[2] = {make_float4(0.f, 0.f, 0.f, 0.f), make_float4(0.f, 0.f, 0.f, 0.f)};
    float4 u[2] = {g[0], g[0]};
    add8(g, gv[j][0]);
    add8(u, uv[j][0]);
#pragma unroll
    for (int l = 1; l <= NL; ++l) {
      if (!live(l, j)) continue;
      add8(g, gv[j][l]);
      add8(u, uv[j][l]);
    }
#pragma unroll
    for (int q = 0; q < 2; ++q)
      h[j][q] = make_float4(w[j] * silu_mul(g[q].x, u[q].x), w[j] * silu_mul(g[q].y, u[q].y),
                            w[j] * silu_mul(g[q].z, u[q].z), w[j] * silu_mul(g[q].w, u[q].w));
  }
  auto stored = [&](int l, int j0) { return (fl[l][j0] & 3) == 3 && !(merged && l > 0 && l < NL); };
  auto row_sum = [&](int l, int j0, int q) {
    float4 hs = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int j = j0; j < kFastK; ++j)
      if (row[l][j] == row[l][j0] && (fl[NL][j] & 1)) add4(hs, h[j][q]);
    return hs;
  };
  float m = 0.f;
#pragma unroll
  for (int l = 0; l <= NL; ++l)
#pragma unroll
    for (int j0 = 0; j0 < kFastK; ++j0) {
      if (!stored(l, j0)) continue;
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const float4 hs = row_sum(l, j0, q);
        m = fmaxf(m, fmaxf(fmaxf(fabsf(hs.x), fabsf(hs.y)), fmaxf(fabsf(hs.z), fabsf(hs.w))));
      }
    }
  const int sh = f16_token_shift(m);
  typedef _Float16 h8 __attribute__((ext_vector_type(8)));
#pragma unroll
  for (int l = 0; l <= NL; ++l)
#pragma unroll
    for (int j0 = 0; j0 < kFastK; ++j0) {
      if (!stored(l, j0)) continue;
      if (act) {
        const float4 s0 = row_sum(l, j0, 0), s1 = row_sum(l, j0, 1);
        h8 o;
        o[0] = (_Float16)ldexpf(s0.x, sh);
        o[1] = (_Float16)ldexpf(s0.y, sh);
        o[2] = (_Float16)ldexpf(s0.z, sh);
        o[3] = (_Float16)ldexpf(s0.w, sh);
        o[4] = (_Float16)ldexpf(s1.x, sh);
        o[5] = (_Float16)ldexpf(s1.y, sh);
        o[6] = (_Float16)ldexpf(s1.z, sh);
        o[7] = (_Float16)ldexpf(s1.w, sh);
        *(h8*)((_Float16*)a.hbar[l] + (int64_t)row[l][j0] * f + c) = o;
      }
      if (threadIdx.x == 0) a.hbar_exp[l][row[l][j0]] = sh;
    }
}

template <int NL, bool X16>
__global__ __launch_bounds__(kFastThr) void k_combine_fast(TokenArgs a) {
  const int t = blockIdx.x, k = a.k, d = a.d;
  const int c = (blockIdx.y * blockDim.x + threadIdx.x) * 4;
  if (c >= d) return;
  int row[NL + 1][kFastK], fl[NL + 1][kFastK];
  float w[kFastK];
  token_meta_fast<NL>(a, t, row, fl, w);
  // merged trees: the intermediate levels' terms are in the leaf rows
  const bool merged = a.merged != 0;
  Raw4<X16> v[NL + 1][kFastK];
#pragma unroll
  for (int l = 0; l <= NL; ++l)
#pragma unroll
    for (int j = 0; j < kFastK; ++j)
      if ((fl[l][j] & 3) == 3 && !(merged && l > 0 && l < NL)) v[l][j] = ldraw<X16>(a.y[l], row[l][j], d, c);
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int l = 0; l <= NL; ++l)
#pragma unroll
    for (int j = 0; j < kFastK; ++j)
      if ((fl[l][j] & 3) == 3 && !(merged && l > 0 && l < NL)) add4(acc, cvt<X16>(v[l][j], c));
  if (a.out_dtype == LX_F32) {
    *(float4*)((float*)a.out + (int64_t)t * d + c) = acc;
  } else {
    bf16x4 o;
    o[0] = (__bf16)acc.x;
    o[1] = (__bf16)acc.y;
    o[2] = (__bf16)acc.z;
    o[3] = (__bf16)acc.w;
    *(bf16x4*)((uint16_t*)a.out + (int64_t)t * d + c) = o;
  }
}

// x16 rows, CPT (8 or 16) columns per thread: one 16-byte load per x16 group
// and row (a fraction of the load instructions of 4 columns per thread);
// otherwise as k_combine_fast.
template <int NL, int CPT, bool MERGED>
__global__ __launch_bounds__(kFastThr) void k_combine_x16w(TokenArgs a) {
  constexpr int NG = CPT / 4;  // 4-value groups per thread
  const int t = blockIdx.x, k = a.k, d = a.d;
  const int c = (blockIdx.y * blockDim.x + threadIdx.x) * CPT;
  if (c >= d) return;
  int row[NL + 1][kFastK], fl[NL + 1][kFastK];
  float w[kFastK];
  token_meta_fast<NL>(a, t, row, fl, w);
  // (a.merged, as a template argument: the intermediate levels' rows are
  // never loaded and take no registers)
  constexpr bool merged = MERGED;
  uint4 mv[NL + 1][kFastK][NG / 2];
#pragma unroll
  for (int l = 0; l <= NL; ++l)
#pragma unroll
    for (int j = 0; j < kFastK; ++j)
      if ((fl[l][j] & 3) == 3 && !(merged && l > 0 && l < NL)) {
        const uint8_t* rp = (const uint8_t*)a.y[l] + ((int64_t)row[l][j] * d + c) * 2;
#pragma unroll
        for (int h = 0; h < NG / 2; ++h) mv[l][j][h] = *(const uint4*)(rp + 16 * h);
      }
  float4 acc[NG];
#pragma unroll
  for (int g = 0; g < NG; ++g) acc[g] = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int l = 0; l <= NL; ++l)
#pragma unroll
    for (int j = 0; j < kFastK; ++j)
      if ((fl[l][j] & 3) == 3 && !(merged && l > 0 && l < NL)) {
#pragma unroll
        for (int h = 0; h < NG / 2; ++h) {
          float4 va, vb;
          x16_unpack8(mv[l][j][h], va, vb);
          add4(acc[2 * h], va);
          add4(acc[2 * h + 1], vb);
        }
      }
  if (a.out_dtype == LX_F32) {
    float4* o = (float4*)((float*)a.out + (int64_t)t * d + c);
#pragma unroll
    for (int g = 0; g < NG; ++g) o[g] = acc[g];
  } else {
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      bf16x4 o;
      o[0] = (__bf16)acc[g].x;
      o[1] = (__bf16)acc[g].y;
      o[2] = (__bf16)acc[g].z;
      o[3] = (__bf16)acc[g].w;
      *(bf16x4*)((uint16_t*)a.out + (int64_t)t * d + c + 4 * g) = o;
    }
  }
}

// Threads per workgroup for n 4-column groups: whole wavefronts, at most
// kFastThr; one wavefront for small batches, whose token count alone would
// give fewer workgroups than the chip has compute units.
int fast_threads(int cols, int T) {
  if (T < 512) return 64;
  const int g = (cols / 4 + 63) / 64 * 64;
  return g < 64 ? 64 : g > kFastThr ? kFastThr : g;
}

}  // namespace

// The fast paths need one row format on every level (all x16 or all fp32).
static int uniform_fmt(const TokenArgs& a) {
  for (int l = 1; l <= a.L; ++l)
    if (a.x16[l] != a.x16[0]) return -1;
  return a.x16[0] ? 1 : 0;
}

hipError_t launch_swiglu_reduce(const TokenArgs& a, hipStream_t s) {
  if (a.T == 0) return hipSuccess;
  const int fmt = uniform_fmt(a);
  bool f16 = false;
  for (int l = 0; l <= a.L; ++l) f16 |= a.hbar_mode[l] == HBAR_F16;
  // x16 rows and fp16 sums on every stored level: the wide kernel, where
  // f / 8 threads fill whole wavefronts (f = 768 measured faster on the
  // 4-column kernel)
  bool all16 = true;
  for (int l = 0; l <= a.L; ++l) all16 &= a.hbar_mode[l] == HBAR_F16 || (a.merged && l > 0 && l < a.L);
  if (a.k <= kFastK && a.L <= kFastL && fmt == 1 && all16 && a.f % 512 == 0 && a.f <= 8 * kFastThr) {
    const int thr = (a.f / 8 + 63) / 64 * 64;
    if (a.L == 0)
      hipLaunchKernelGGL((k_swiglu_x16w<0, false>), dim3(a.T), dim3(thr), 0, s, a);
    else if (a.L == 1)
      hipLaunchKernelGGL((k_swiglu_x16w<1, false>), dim3(a.T), dim3(thr), 0, s, a);
    else if (a.merged)
      hipLaunchKernelGGL((k_swiglu_x16w<2, true>), dim3(a.T), dim3(thr), 0, s, a);
    else
      hipLaunchKernelGGL((k_swiglu_x16w<2, false>), dim3(a.T), dim3(thr), 0, s, a);
    return hipGetLastError();
  }
  if (a.k <= kFastK && a.L <= kFastL && fmt >= 0) {
    const int thr = fast_threads(a.f, a.T);
    const dim3 grid(a.T, (a.f / 4 + thr - 1) / thr);
    // fp16 rows need every row's values in one workgroup, all threads live
    if (f16 && (grid.y != 1 || thr * 4 != a.f)) return hipErrorInvalidValue;
    if (a.L == 0 && fmt)
      hipLaunchKernelGGL((k_swiglu_fast<0, true>), grid, dim3(thr), 0, s, a);
    else if (a.L == 0)
      hipLaunchKernelGGL((k_swiglu_fast<0, false>), grid, dim3(thr), 0, s, a);
    else if (a.L == 1 && fmt)
      hipLaunchKernelGGL((k_swiglu_fast<1, true>), grid, dim3(thr), 0, s, a);
    else if (a.L == 1)
      hipLaunchKernelGGL((k_swiglu_fast<1, false>), grid, dim3(thr), 0, s, a);
    else if (fmt)
      hipLaunchKernelGGL((k_swiglu_fast<2, true>), grid, dim3(thr), 0, s, a);
    else
      hipLaunchKernelGGL((k_swiglu_fast<2, false>), grid, dim3(thr), 0, s, a);
    return hipGetLastError();
  }
  if (f16) return hipErrorInvalidValue;  // the general kernel splits rows
  const int groups = a.k < kSlotGroups ? a.k : kSlotGroups;
  hipLaunchKernelGGL(k_swiglu_reduce, dim3(a.T, (a.f + kTokCols - 1) / kTokCols), dim3(kTokThr * groups),
                     (size_t)a.k * kTokThr * sizeof(float4), s, a);
  return hipGetLastError();
}

hipError_t launch_combine(const TokenArgs& a, hipStream_t s) {
  if (a.T == 0) return hipSuccess;
  const int fmt = uniform_fmt(a);
  if (a.k <= kFastK && a.L <= kFastL && fmt == 1 && a.d % 64 == 0) {  // 16-byte aligned rows
    constexpr int CPT = 8;  // (16 measured no faster)
    const int thr = fast_threads(a.d * 4 / CPT, a.T);
    const dim3 grid(a.T, (a.d / CPT + thr - 1) / thr);
    if (a.L == 0)
      hipLaunchKernelGGL((k_combine_x16w<0, CPT, false>), grid, dim3(thr), 0, s, a);
    else if (a.L == 1)
      hipLaunchKernelGGL((k_combine_x16w<1, CPT, false>), grid, dim3(thr), 0, s, a);
    else if (a.merged)
      hipLaunchKernelGGL((k_combine_x16w<2, CPT, true>), grid, dim3(thr), 0, s, a);
    else
      hipLaunchKernelGGL((k_combine_x16w<2, CPT, false>), grid, dim3(thr), 0, s, a);
    return hipGetLastError();
  }
  if (a.k <= kFastK && a.L <= kFastL && fmt >= 0) {
    const int thr = fast_threads(a.d, a.T);
    const dim3 grid(a.T, (a.d / 4 + thr - 1) / thr);
    switch (a.L * 2 + fmt) {
      case 0: hipLaunchKernelGGL((k_combine_fast<0, false>), grid, dim3(thr), 0, s, a); break;
      case 1: hipLaunchKernelGGL((k_combine_fast<0, true>), grid, dim3(thr), 0, s, a); break;
      case 2: hipLaunchKernelGGL((k_combine_fast<1, false>), grid, dim3(thr), 0, s, a); break;
      case 3: hipLaunchKernelGGL((k_combine_fast<1, true>), grid, dim3(thr), 0, s, a); break;
      case 4: hipLaunchKernelGGL((k_combine_fast<2, false>), grid, dim3(thr), 0, s, a); break;
      default: hipLaunchKernelGGL((k_combine_fast<2, true>), grid, dim3(thr), 0, s, a); break;
    }
    return hipGetLastError();
  }
  int thr = (a.d / 4 + 63) / 64 * 64;
  thr = thr < 64 ? 64 : thr > kCombMaxThr ? kCombMaxThr : thr;
  hipLaunchKernelGGL(k_combine, dim3(a.T), dim3(thr), 0, s, a);
  return hipGetLastError();
}

}  // namespace lx

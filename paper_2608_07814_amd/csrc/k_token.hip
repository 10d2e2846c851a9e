// Per-token kernels: SwiGLU with the amortized weighted reduction, and the
// deterministic combine. SwiGLU runs one workgroup per (token, 256-neuron
// chunk), combine one per token; every thread owns 4 consecutive neurons
// (SwiGLU) or output columns (combine), so all accesses are 16-byte vectors.
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
__device__ __forceinline__ void add4(float4& a, const float4& b) {
  a.x += b.x;
  a.y += b.y;
  a.z += b.z;
  a.w += b.w;
}
__device__ __forceinline__ float silu_mul(float g, float u) { return g / (1.f + expf(-g)) * u; }

// hbar row segment (4 neurons at column c): fp32, or a bf16 (hi, lo) pair in
// a row of 2f (hi half, lo half).
__device__ __forceinline__ void hbar_store(void* base, bool hilo, int row, int c, int f, float4 v) {
  if (hilo) {
    __bf16* hb = (__bf16*)base + (int64_t)row * 2 * f;
    bf16x4 hi, lo;
    hi[0] = (__bf16)v.x;
    hi[1] = (__bf16)v.y;
    hi[2] = (__bf16)v.z;
    hi[3] = (__bf16)v.w;
    lo[0] = (__bf16)(v.x - (float)hi[0]);
    lo[1] = (__bf16)(v.y - (float)hi[1]);
    lo[2] = (__bf16)(v.z - (float)hi[2]);
    lo[3] = (__bf16)(v.w - (float)hi[3]);
    *(bf16x4*)(hb + c) = hi;
    *(bf16x4*)(hb + f + c) = lo;
  } else {
    *(float4*)((float*)base + (int64_t)row * f + c) = v;
  }
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
    const float* g0 = a.gu0 + m.row[0][j] * ld;
    float4 g = ld4(g0 + c), u = ld4(g0 + f + c);
    for (int l = 1; l <= L; ++l) {
      if (!(m.fl[l][j] & 2)) continue;
      const float* dg = a.dgu[l] + m.row[l][j] * ld;
      add4(g, ld4(dg + c));
      add4(u, ld4(dg + f + c));
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
      const int r = m.row[l][j0];
      float4 hs = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int j = j0; j < k; ++j)
        if (m.row[l][j] == r && (m.fl[L][j] & 1)) add4(hs, s_h[j * kTokThr + lane]);
      hbar_store(a.hbar[l], a.hbar_hilo[l], r, c, f, hs);
    }
  }
}

// Combine, one workgroup per token (whole output rows, so every row of the
// token is read as one contiguous stretch): wavefront 0 lists the token's rows
// to sum (first slot of a row that does work) in (level, slot) order with a
// ballot compaction; then every thread sums its 4 columns over that list, 16
// row loads in flight at a time, adding in list order.
constexpr int kCombMaxThr = 512;
__global__ __launch_bounds__(kCombMaxThr) void k_combine(TokenArgs a) {
  __shared__ const float* s_rows[kMaxLvl * LX_MAX_K];
  __shared__ int s_n;
  const int t = blockIdx.x;
  const int k = a.k, L = a.L, d = a.d;
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    const int nq = (L + 1) * k;
    int base = 0;
    for (int q0 = 0; q0 < nq; q0 += 64) {
      const int q = q0 + lane;
      bool take = false;
      const float* ptr = nullptr;
      if (q < nq) {
        const int l = q / k, j = q - l * k;
        const int64_t sl = (int64_t)t * k + j;
        const int row = a.slot_row[l][sl];  // loaded alongside the flags
        if ((a.slot_flags[l][sl] & 3) == 3) {
          take = true;
          ptr = a.y[l] + (int64_t)row * d;
        }
      }
      const uint64_t bal = __ballot(take);
      if (take) s_rows[base + __popcll(bal & ((1ull << lane) - 1))] = ptr;
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
        if (b + i < n) v[i] = ld4(s_rows[b + i] + c);
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

}  // namespace

hipError_t launch_swiglu_reduce(const TokenArgs& a, hipStream_t s) {
  if (a.T == 0) return hipSuccess;
  const int groups = a.k < kSlotGroups ? a.k : kSlotGroups;
  hipLaunchKernelGGL(k_swiglu_reduce, dim3(a.T, (a.f + kTokCols - 1) / kTokCols), dim3(kTokThr * groups),
                     (size_t)a.k * kTokThr * sizeof(float4), s, a);
  return hipGetLastError();
}

hipError_t launch_combine(const TokenArgs& a, hipStream_t s) {
  if (a.T == 0) return hipSuccess;
  int thr = (a.d / 4 + 63) / 64 * 64;
  thr = thr < 64 ? 64 : thr > kCombMaxThr ? kCombMaxThr : thr;
  hipLaunchKernelGGL(k_combine, dim3(a.T), dim3(thr), 0, s, a);
  return hipGetLastError();
}

}  // namespace lx

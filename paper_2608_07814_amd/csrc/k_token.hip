// Per-token kernels: SwiGLU with the amortized weighted reduction, and the
// deterministic combine. One workgroup per token; every thread owns 4
// consecutive neurons (SwiGLU) or output columns (combine), so all accesses
// are 16-byte vectors.
//
// For a token t with selected experts e_j (j ascending), every tree level l
// has one row per distinct level-l node among the e_j (from the bucketing,
// which also marks each slot's first-of-row and has-work bits and stores each
// distinct expert's summed routing weight on its first slot).
//   swiglu_reduce: for each anchor row of t, for each distinct expert under it
//       g = anchor gate row + sum over levels of the node's gate correction,
//       u likewise, h = w * silu(g) * u;
//     h is summed in registers into the anchor row's hbar0 (one write per
//     row) and accumulated into hbar_l[row_l] of every correction level whose
//     node carries a factor. By linearity the down projections then run once
//     per row (Sec. 5.1 amortized forward).
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
__device__ __forceinline__ float4 hbar_load(const void* base, bool hilo, int row, int c, int f) {
  if (hilo) {
    const __bf16* hb = (const __bf16*)base + (int64_t)row * 2 * f;
    const bf16x4 hi = *(const bf16x4*)(hb + c);
    const bf16x4 lo = *(const bf16x4*)(hb + f + c);
    return make_float4((float)hi[0] + (float)lo[0], (float)hi[1] + (float)lo[1],
                       (float)hi[2] + (float)lo[2], (float)hi[3] + (float)lo[3]);
  }
  return ld4((const float*)base + (int64_t)row * f + c);
}

__global__ __launch_bounds__(256) void k_swiglu_reduce(TokenArgs a) {
  __shared__ TokenMeta m;
  const int t = blockIdx.x;
  token_meta(a, t, m);
  __syncthreads();
  const int k = a.k, L = a.L, f = a.f;
  const int64_t ld = 2 * (int64_t)f;
  for (int c = threadIdx.x * 4; c < f; c += blockDim.x * 4) {
    for (int j0 = 0; j0 < k; ++j0) {
      if (!(m.fl[0][j0] & 1)) continue;  // start of an anchor row of t
      const int r0 = m.row[0][j0];
      const float* g0 = a.gu0 + r0 * ld;
      const float4 gb = ld4(g0 + c), ub = ld4(g0 + f + c);
      float4 hs = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int j = j0; j < k; ++j) {
        // the row's distinct experts: same anchor row, first slot of the expert
        if (m.row[0][j] != r0 || !(m.fl[L][j] & 1)) continue;
        float4 g = gb, u = ub;
        for (int l = 1; l <= L; ++l) {
          if (!(m.fl[l][j] & 2)) continue;
          const float* dg = a.dgu[l] + m.row[l][j] * ld;
          add4(g, ld4(dg + c));
          add4(u, ld4(dg + f + c));
        }
        const float w = m.w[j];
        const float4 h = make_float4(w * silu_mul(g.x, u.x), w * silu_mul(g.y, u.y),
                                     w * silu_mul(g.z, u.z), w * silu_mul(g.w, u.w));
        add4(hs, h);
        for (int l = 1; l <= L; ++l) {
          const unsigned char fl = m.fl[l][j];
          if (!(fl & 2)) continue;
          float4 v = h;
          if (!(fl & 1)) add4(v, hbar_load(a.hbar[l], a.hbar_hilo[l], m.row[l][j], c, f));
          hbar_store(a.hbar[l], a.hbar_hilo[l], m.row[l][j], c, f, v);
        }
      }
      hbar_store(a.hbar[0], a.hbar_hilo[0], r0, c, f, hs);
    }
  }
}

__global__ __launch_bounds__(256) void k_combine(TokenArgs a) {
  __shared__ TokenMeta m;
  const int t = blockIdx.x;
  token_meta(a, t, m);
  __syncthreads();
  const int k = a.k, L = a.L, d = a.d;
  for (int c = threadIdx.x * 4; c < d; c += blockDim.x * 4) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int l = 0; l <= L; ++l)
      for (int j = 0; j < k; ++j) {
        if ((m.fl[l][j] & 3) != 3) continue;  // first slot of a row that does work
        add4(acc, ld4(a.y[l] + (int64_t)m.row[l][j] * d + c));
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
  const int threads = a.f / 4 >= 256 ? 256 : ((a.f / 4 + 63) / 64) * 64;
  hipLaunchKernelGGL(k_swiglu_reduce, dim3(a.T), dim3(threads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_combine(const TokenArgs& a, hipStream_t s) {
  if (a.T == 0) return hipSuccess;
  const int threads = a.d / 4 >= 256 ? 256 : ((a.d / 4 + 63) / 64) * 64;
  hipLaunchKernelGGL(k_combine, dim3(a.T), dim3(threads), 0, s, a);
  return hipGetLastError();
}

}  // namespace lx

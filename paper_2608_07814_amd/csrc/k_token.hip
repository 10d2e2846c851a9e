// Per-token kernels: SwiGLU with the amortized weighted reduction, and the
// deterministic combine.
//
// For a token t with selected experts e_j (j ascending), every tree level l
// has one row per distinct level-l node among the e_j (from the bucketing).
//   swiglu_reduce: for each distinct expert of t (first slot j of its leaf
//     row, weight = sum of the routing weights of its slots)
//       g = anchor gate row + sum over levels of the node's gate correction,
//       u likewise, h = silu(g) * u,
//     and w*h is accumulated into hbar_l[row_l(j)] of every level that does
//     down-projection work (the anchor level always; a correction level when
//     the node carries a factor). By linearity the down projections then run
//     once per row (Sec. 5.1 amortized forward).
//   combine: out[t] = sum over levels, over t's rows of the level, of that
//     level's down-projection output row; a fixed order (level, then slot)
//     with no atomics, so the result is bit-reproducible.
#include "lx_internal.h"

namespace lx {
namespace {

struct TokenMeta {
  int row[kMaxLvl][LX_MAX_K];
  unsigned char first[kMaxLvl][LX_MAX_K];
  unsigned char work[kMaxLvl][LX_MAX_K];
  float w[LX_MAX_K];
};

// Threads 0..k-1 fill the metadata of token t; caller synchronizes.
__device__ inline void token_meta(const TokenArgs& a, int t, TokenMeta& m) {
  const int k = a.k, L = a.L, E = a.E;
  const int j = threadIdx.x;
  if (j >= k) return;
  const int64_t base = (int64_t)t * k;
  const int e = a.ids[base + j];
  const bool valid = e >= 0 && e < E && a.anc[e] >= 0;
  for (int l = 0; l <= L; ++l) {
    const int row = valid ? a.slot_row[l][base + j] : -1;
    bool first = valid;
    if (valid)
      for (int j2 = 0; j2 < j; ++j2) first &= (a.slot_row[l][base + j2] != row);
    bool work = valid;
    if (valid && l > 0) work = a.fac[l][a.anc[(int64_t)l * E + e]] >= 0;
    m.row[l][j] = row;
    m.first[l][j] = first;
    m.work[l][j] = work;
  }
  float w = 0.f;
  if (valid && m.first[L][j]) {
    const int row = m.row[L][j];
    for (int j2 = j; j2 < k; ++j2)
      if (a.slot_row[L][base + j2] == row) w += a.w[base + j2];
  }
  m.w[j] = w;
}

__global__ __launch_bounds__(256) void k_swiglu_reduce(TokenArgs a) {
  __shared__ TokenMeta m;
  const int t = blockIdx.x;
  token_meta(a, t, m);
  __syncthreads();
  const int k = a.k, L = a.L, f = a.f;
  const int64_t ld = 2 * (int64_t)f;
  for (int i = threadIdx.x; i < f; i += blockDim.x) {
    for (int j = 0; j < k; ++j) {
      if (!m.first[L][j]) continue;  // one pass per distinct expert of t
      const float* g0 = a.gu0 + m.row[0][j] * ld;
      float g = g0[i], u = g0[f + i];
      for (int l = 1; l <= L; ++l) {
        if (!m.work[l][j]) continue;
        const float* dg = a.dgu[l] + m.row[l][j] * ld;
        g += dg[i];
        u += dg[f + i];
      }
      const float h = m.w[j] * (g / (1.f + expf(-g))) * u;
      for (int l = 0; l <= L; ++l) {
        if (!m.work[l][j]) continue;
        if (a.hbar_hilo[l]) {
          // bf16 pair: hi at column i, lo = bf16(sum - hi) at column f + i.
          // The running sum is rebuilt as hi + lo, which is exact to ~2^-17.
          __bf16* hb = (__bf16*)a.hbar[l] + (int64_t)m.row[l][j] * ld;
          float sum = h;
          if (!m.first[l][j]) sum += (float)hb[i] + (float)hb[f + i];
          const __bf16 hi = (__bf16)sum;
          hb[i] = hi;
          hb[f + i] = (__bf16)(sum - (float)hi);
          continue;
        }
        float* hb = a.hbar[l] + (int64_t)m.row[l][j] * f + i;
        if (m.first[l][j])
          *hb = h;
        else
          *hb += h;
      }
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
        if (!(m.first[l][j] && m.work[l][j])) continue;
        const float4 v = *(const float4*)(a.y[l] + (int64_t)m.row[l][j] * d + c);
        acc.x += v.x;
        acc.y += v.y;
        acc.z += v.z;
        acc.w += v.w;
      }
    if (a.out_dtype == LX_F32) {
      *(float4*)((float*)a.out + (int64_t)t * d + c) = acc;
    } else {
      typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
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
  hipLaunchKernelGGL(k_swiglu_reduce, dim3(a.T), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_combine(const TokenArgs& a, hipStream_t s) {
  if (a.T == 0) return hipSuccess;
  hipLaunchKernelGGL(k_combine, dim3(a.T), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace lx

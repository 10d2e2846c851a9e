// Top-k of one token's router logits by one wavefront (device code shared by
// the router's own kernel and the bucketing kernels that fuse it).
//
// The k largest logits in descending order, equal logits ordered by the
// lower expert index, NaN below every number; the weights are the softmax of
// the chosen logits (= the full softmax restricted to them and renormalised).
// Logits come from the skinny GEMM over implicit 32-row tiles: either final
// ([T][E] fp32, S <= 1) or S partial tiles per (32-row tile, 64-column tile)
// item, added here in split order (run-to-run deterministic).
// Lane l holds experts l, l + 64, ...; k rounds of a wavefront-wide (value,
// lower index) maximum; lane j < k returns the j-th choice.
#pragma once

#include "lx_internal.h"

namespace lx {

__device__ __forceinline__ bool topk_better(float v, int i, float bv, int bi) {
  return v > bv || (v == bv && i < bi);
}

// (value, index) of lane l's partner under a DPP pattern (all lanes valid).
template <int CTRL>
__device__ __forceinline__ void dpp_pair(float v, int i, float& ov, int& oi) {
  ov = __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
  oi = __builtin_amdgcn_update_dpp(0, i, CTRL, 0xF, 0xF, false);
}

// Wavefront-wide best (value, lower index) of every lane's candidate, on
// every lane. The order is total, so the winner does not depend on the
// combining pattern: inside each row of 16 lanes by DPP (rotate by 8, by 4,
// then the quad permutations xor 2 and xor 1: VALU only), across the four
// rows by two lane exchanges.
__device__ __forceinline__ void wave_best(float& bv, int& bi) {
  float ov;
  int oi;
  dpp_pair<0x128>(bv, bi, ov, oi);  // row_ror:8
  if (topk_better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
  dpp_pair<0x124>(bv, bi, ov, oi);  // row_ror:4
  if (topk_better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
  dpp_pair<0x4E>(bv, bi, ov, oi);   // quad_perm [2, 3, 0, 1]
  if (topk_better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
  dpp_pair<0xB1>(bv, bi, ov, oi);   // quad_perm [1, 0, 3, 2]
  if (topk_better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
#pragma unroll
  for (int off = 16; off <= 32; off <<= 1) {
    ov = __shfl_xor(bv, off, 64);
    oi = __shfl_xor(bi, off, 64);
    if (topk_better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
  }
}

// NTOK tokens per wavefront at once (tok[u] < 0: no token in that place),
// their rounds interleaved so that the shuffle chains of different tokens
// overlap; every token's arithmetic is the same as with NTOK = 1. Every lane
// of the wavefront must call it (wavefront-wide shuffles).
template <int NTOK>
__device__ __forceinline__ void topk_tokens(const float* __restrict__ logits, const float* __restrict__ part, int S,
                                            int E, int k, const int (&tok)[NTOK], int (&id)[NTOK],
                                            float (&weight)[NTOK]) {
  constexpr int PER = kRouteMaxE / 64;
  const int lane = threadIdx.x & 63;
  const int ntn = (E + kSkinnyBN - 1) / kSkinnyBN;
  float v[NTOK][PER];
#pragma unroll
  for (int u = 0; u < NTOK; ++u) {
    const int t = tok[u] < 0 ? 0 : tok[u];
    const int ti = t / kSkinnyBM, row = t % kSkinnyBM;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int e = lane + 64 * j;
      float z = -INFINITY;
      if (e < E && tok[u] >= 0) {
        if (S <= 1) {
          z = logits[(int64_t)t * E + e];
        } else {
          // slot (item * S + split), item = ti * ntn + e / 64; inside a slot
          // [wavefront = (e % 64) / 32][row][e % 32]
          const float* q = part + ((int64_t)(ti * ntn + e / 64) * S) * (kSkinnyBM * kSkinnyBN) +
                           ((e & 63) >> 5) * (32 * 32) + row * 32 + (e & 31);
          z = q[0];
          for (int sp = 1; sp < S; ++sp) z += q[(int64_t)sp * (kSkinnyBM * kSkinnyBN)];
        }
      }
      v[u][j] = z == z ? z : -INFINITY;
    }
  }
  uint32_t taken0 = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j)
    if (lane + 64 * j >= E) taken0 |= 1u << j;
  uint32_t taken[NTOK];
  float my_v[NTOK];
  int my_i[NTOK];
#pragma unroll
  for (int u = 0; u < NTOK; ++u) {
    taken[u] = taken0;
    my_v[u] = -INFINITY;
    my_i[u] = 0;
  }
  for (int round = 0; round < k; ++round) {
    float bv[NTOK];
    int bi[NTOK];
#pragma unroll
    for (int u = 0; u < NTOK; ++u) {
      bv[u] = -INFINITY;
      bi[u] = 0x7FFFFFFF;
#pragma unroll
      for (int j = 0; j < PER; ++j)
        if (!((taken[u] >> j) & 1u) && topk_better(v[u][j], lane + 64 * j, bv[u], bi[u])) {
          bv[u] = v[u][j];
          bi[u] = lane + 64 * j;
        }
    }
#pragma unroll
    for (int u = 0; u < NTOK; ++u) wave_best(bv[u], bi[u]);
    // every lane holds the winner (k <= E: an untaken expert always exists)
#pragma unroll
    for (int u = 0; u < NTOK; ++u) {
      if ((bi[u] & 63) == lane) taken[u] |= 1u << (bi[u] >> 6);
      if (lane == round) {
        my_v[u] = bv[u];
        my_i[u] = bi[u];
      }
    }
  }
#pragma unroll
  for (int u = 0; u < NTOK; ++u) {
    const float m = __shfl(my_v[u], 0, 64);  // the largest chosen logit
    const float ex = lane < k ? expf(my_v[u] - m) : 0.f;
    float s = ex;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off, 64);  // same tree on every lane
    id[u] = my_i[u];
    weight[u] = ex / s;
  }
}

// One token per wavefront.
__device__ __forceinline__ void topk_token(const float* __restrict__ logits, const float* __restrict__ part, int S,
                                           int E, int k, int t, int& id, float& weight) {
  const int tok[1] = {t};
  int i1[1];
  float w1[1];
  topk_tokens<1>(logits, part, S, E, k, tok, i1, w1);
  id = i1[0];
  weight = w1[0];
}

}  // namespace lx

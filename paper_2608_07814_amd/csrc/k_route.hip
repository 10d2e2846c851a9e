// Top-k of the unchanged router, on the GPU: the k largest logits in
// descending order (equal logits: lower expert index first; NaN below every
// number), weights = the softmax of the chosen logits (= the full softmax
// restricted to them and renormalised).
//
// The logits themselves (x W_r^T, fp32 accumulation of exact bf16 products)
// come from the skinny GEMM over implicit 32-row tiles. When the tiles are
// too few to stream W_r at speed, that GEMM is split along d and leaves S
// partial tiles per (row tile, 64-column tile) item in the workspace; this
// kernel adds them in split order while it reads the logits, so the pair
// needs no counters and stays run-to-run deterministic.
//
// One wavefront per token: lane l holds experts l, l + 64, ...; k rounds of
// a wavefront-wide (value, lower index) maximum; then the softmax over the
// chosen values, lanes 0 .. k-1 holding one chosen expert each.
#include "lx_internal.h"

namespace lx {
namespace {

constexpr int TK_WAVES = 4;

__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
  return v > bv || (v == bv && i < bi);
}

__global__ __launch_bounds__(TK_WAVES * 64) void k_topk(const float* __restrict__ logits,
                                                        const float* __restrict__ part, int S, int T, int E,
                                                        int k, int32_t* __restrict__ ids,
                                                        float* __restrict__ weights) {
  constexpr int PER = kRouteMaxE / 64;
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * TK_WAVES + (threadIdx.x >> 6);
  if (t >= T) return;  // whole wavefront
  const int ntn = (E + kSkinnyBN - 1) / kSkinnyBN;
  const int ti = t / kSkinnyBM, row = t % kSkinnyBM;

  float v[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int e = lane + 64 * j;
    float z = -INFINITY;
    if (e < E) {
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
    v[j] = z == z ? z : -INFINITY;
  }
  uint32_t taken = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j)
    if (lane + 64 * j >= E) taken |= 1u << j;
  float my_v = -INFINITY;
  int my_i = 0;
  for (int round = 0; round < k; ++round) {
    float bv = -INFINITY;
    int bi = 0x7FFFFFFF;
#pragma unroll
    for (int j = 0; j < PER; ++j)
      if (!((taken >> j) & 1u) && better(v[j], lane + 64 * j, bv, bi)) {
        bv = v[j];
        bi = lane + 64 * j;
      }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const float ov = __shfl_xor(bv, off, 64);
      const int oi = __shfl_xor(bi, off, 64);
      if (better(ov, oi, bv, bi)) {
        bv = ov;
        bi = oi;
      }
    }
    // every lane holds the winner (k <= E: an untaken expert always exists)
    if ((bi & 63) == lane) taken |= 1u << (bi >> 6);
    if (lane == round) {
      my_v = bv;
      my_i = bi;
    }
  }
  const float m = __shfl(my_v, 0, 64);  // the largest chosen logit
  const float ex = lane < k ? expf(my_v - m) : 0.f;
  float s = ex;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off, 64);  // same tree on every lane
  if (lane < k) {
    ids[(int64_t)t * k + lane] = my_i;
    weights[(int64_t)t * k + lane] = ex / s;
  }
}

}  // namespace

hipError_t launch_topk(const float* logits, const float* part, int S, int T, int E, int k, int32_t* ids,
                       float* weights, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_topk, dim3((T + TK_WAVES - 1) / TK_WAVES), dim3(TK_WAVES * 64), 0, s, logits, part, S, T, E,
                     k, ids, weights);
  return hipGetLastError();
}

}  // namespace lx

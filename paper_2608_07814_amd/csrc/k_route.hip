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
#include "lx_topk.h"

namespace lx {
namespace {

constexpr int TK_WAVES = 4;

__global__ __launch_bounds__(TK_WAVES * 64) void k_topk(const float* __restrict__ logits,
                                                        const float* __restrict__ part, int S, int T, int E,
                                                        int k, int32_t* __restrict__ ids,
                                                        float* __restrict__ weights) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * TK_WAVES + (threadIdx.x >> 6);
  if (t >= T) return;  // whole wavefront
  int id;
  float wt;
  topk_token(logits, part, S, E, k, t, id, wt);
  if (lane < k) {
    ids[(int64_t)t * k + lane] = id;
    weights[(int64_t)t * k + lane] = wt;
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

// Stages 1-2 of the compression pipeline on the GPU (Sec. 3 "Compression
// pipeline"): router profiling counts, the co-activation NPMI distance of the
// Coact-NPMI variant, and frequency-seeded k-medoids with the dominant
// choice. They run once per layer on calibration routing and fix the
// cluster map and factor indices of a flat layer.
//
//   * k_coact: one thread per calibration token; an expert fires on a token
//     when it is among the token's valid ids (once per token); every
//     unordered pair of distinct firing experts co-fires once. Integer
//     atomics (order-free, so the counts are exact and reproducible); for
//     E <= 128 the counts of a workgroup's tokens are gathered in LDS first
//     and only the non-zero ones go to global memory.
//   * k_npmi: D = 1 - NPMI in fp64, one thread per (i, j).
//   * k_kmedoids: one workgroup, one thread per expert (E <= 1024). Seeds =
//     the highest-firing unprotected experts; assign (nearest medoid, ties to
//     the lower cluster, a medoid stays in its own cluster) / update (member
//     with the smallest in-cluster distance sum, summed in ascending member
//     order, ties to the lower index) until no medoid moves. Per-cluster
//     minima in LDS with 64-bit atomic min on order-preserving keys, so every
//     decision is the exact fp64 comparison a sequential loop would make.
#include "lx_internal.h"

namespace lx {
namespace {

constexpr int KM_THR = 1024;

__global__ __launch_bounds__(256) void k_fill_u32(uint32_t* __restrict__ p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

// Valid, first-occurrence ids of token t: slot j counts when 0 <= id < E and
// no earlier slot of the row holds the same id.
__device__ __forceinline__ bool first_valid(const int32_t* row, int j, int E) {
  const int e = row[j];
  if (e < 0 || e >= E) return false;
  for (int q = 0; q < j; ++q)
    if (row[q] == e) return false;
  return true;
}

template <bool LDS>
__global__ __launch_bounds__(256) void k_coact(const int32_t* __restrict__ ids, int N, int k, int E,
                                               uint32_t* __restrict__ fire, uint32_t* __restrict__ pair) {
  __shared__ uint32_t s_pair[LDS ? 128 * 128 : 1];
  __shared__ uint32_t s_fire[LDS ? 128 : 1];
  if (LDS) {
    for (int i = threadIdx.x; i < E * E; i += blockDim.x) s_pair[i] = 0u;
    for (int i = threadIdx.x; i < E; i += blockDim.x) s_fire[i] = 0u;
    __syncthreads();
  }
  for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < N; t += gridDim.x * blockDim.x) {
    const int32_t* row = ids + (int64_t)t * k;
    for (int a = 0; a < k; ++a) {
      if (!first_valid(row, a, E)) continue;
      const int ea = row[a];
      if (LDS)
        atomicAdd(&s_fire[ea], 1u);
      else
        atomicAdd(&fire[ea], 1u);
      for (int b = a + 1; b < k; ++b) {
        if (!first_valid(row, b, E)) continue;
        const int eb = row[b];
        const int lo = ea < eb ? ea : eb, hi = ea < eb ? eb : ea;
        if (LDS)
          atomicAdd(&s_pair[lo * E + hi], 1u);
        else
          atomicAdd(&pair[(int64_t)lo * E + hi], 1u);
      }
    }
  }
  if (LDS) {
    __syncthreads();
    for (int i = threadIdx.x; i < E * E; i += blockDim.x)
      if (s_pair[i]) atomicAdd(&pair[i], s_pair[i]);
    for (int i = threadIdx.x; i < E; i += blockDim.x)
      if (s_fire[i]) atomicAdd(&fire[i], s_fire[i]);
  }
}

// Counts were gathered in the upper triangle: mirror it and zero the diagonal,
// then D = 1 - NPMI.
__global__ __launch_bounds__(256) void k_npmi(const uint32_t* __restrict__ fire, uint32_t* __restrict__ pair, int N,
                                              int E, double* __restrict__ dist) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= (int64_t)E * E) return;
  const int i = (int)(q / E), j = (int)(q % E);
  if (i == j) {
    dist[q] = 0.0;
    return;
  }
  const int lo = i < j ? i : j, hi = i < j ? j : i;
  const uint32_t nij = pair[(int64_t)lo * E + hi];
  double npmi;
  if (nij == 0u) {
    npmi = -1.0;
  } else if (nij == (uint32_t)N) {
    npmi = 1.0;
  } else {
    const double n = (double)N, pij = (double)nij / n;
    npmi = log(pij / (((double)fire[i] / n) * ((double)fire[j] / n))) / (-log(pij));
  }
  dist[q] = 1.0 - npmi;
}

__global__ __launch_bounds__(256) void k_mirror(uint32_t* __restrict__ pair, int E) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= (int64_t)E * E) return;
  const int i = (int)(q / E), j = (int)(q % E);
  if (i > j) pair[q] = pair[(int64_t)j * E + i];
  if (i == j) pair[q] = 0u;
}

// Order-preserving map of doubles onto unsigned 64-bit keys.
__device__ __forceinline__ unsigned long long dkey(double v) {
  const unsigned long long b = (unsigned long long)__double_as_longlong(v);
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

__global__ __launch_bounds__(KM_THR) void k_kmedoids(const double* __restrict__ D, const uint32_t* __restrict__ fire,
                                                     int E, int C, ProtMask pm, int P, int max_iter,
                                                     int32_t* __restrict__ cluster_of,
                                                     int32_t* __restrict__ factor_of, int32_t* __restrict__ dominant,
                                                     int32_t* __restrict__ iterations) {
  __shared__ int s_cl[KM_THR];
  __shared__ int s_med[KM_THR];
  __shared__ uint32_t s_fire[KM_THR];
  __shared__ unsigned long long s_key[KM_THR];
  __shared__ int s_idx[KM_THR];
  __shared__ uint32_t s_fmax[KM_THR];
  __shared__ int s_isdom[KM_THR];
  __shared__ int s_changed;
  const int e = threadIdx.x;
  const int K = C - P;
  const bool live = e < E;
  const bool prot = live && ((pm.bits[e >> 5] >> (e & 31)) & 1u);
  const bool free_e = live && !prot;
  s_fire[e] = live ? fire[e] : 0u;
  s_cl[e] = -1;
  s_isdom[e] = 0;
  __syncthreads();
  // seeds: free experts ranked by (firing count descending, index ascending)
  if (free_e) {
    int rank = 0;
    for (int f = 0; f < E; ++f) {
      const bool pf = (pm.bits[f >> 5] >> (f & 31)) & 1u;
      if (!pf && (s_fire[f] > s_fire[e] || (s_fire[f] == s_fire[e] && f < e))) ++rank;
    }
    if (rank < K) s_med[rank] = e;
  }
  __syncthreads();
  const double* const De = D + (int64_t)(live ? e : 0) * E;
  auto assign = [&]() {
    if (free_e) {
      int own = -1;
      for (int c = 0; c < K; ++c)
        if (s_med[c] == e) own = c;
      if (own >= 0) {
        s_cl[e] = own;
      } else {
        int best = 0;
        double bd = De[s_med[0]];
        for (int c = 1; c < K; ++c) {
          const double v = De[s_med[c]];
          if (v < bd) {
            bd = v;
            best = c;
          }
        }
        s_cl[e] = best;
      }
    }
    __syncthreads();
  };
  assign();
  int it = 0;
  while (it < max_iter) {
    ++it;
    double s = 0.0;
    if (free_e) {
      const int c = s_cl[e];
      for (int j = 0; j < E; ++j)
        if (s_cl[j] == c) s += De[j];
    }
    if (e < K) {
      s_key[e] = ~0ull;
      s_idx[e] = 0x7FFFFFFF;
    }
    __syncthreads();
    if (free_e) atomicMin(&s_key[s_cl[e]], dkey(s));
    __syncthreads();
    if (free_e && dkey(s) == s_key[s_cl[e]]) atomicMin(&s_idx[s_cl[e]], e);
    if (e == 0) s_changed = 0;
    __syncthreads();
    if (e < K && s_idx[e] != s_med[e]) {
      s_med[e] = s_idx[e];
      s_changed = 1;
    }
    __syncthreads();
    if (!s_changed) break;
    assign();
  }
  // protected experts: singleton clusters after the seeded ones
  if (prot) {
    int rank = 0;
    for (int f = 0; f < e; ++f) rank += (pm.bits[f >> 5] >> (f & 31)) & 1u;
    s_cl[e] = K + rank;
  }
  if (e < C) {
    s_fmax[e] = 0u;
    s_key[e] = 0ull;
    s_idx[e] = 0x7FFFFFFF;
  }
  __syncthreads();
  // dominant: most fired, then most central (sum of 1 - D to the other
  // members, ascending member order), then lowest index
  const int c = live ? s_cl[e] : 0;
  double cent = 0.0;
  if (live)
    for (int j = 0; j < E; ++j)
      if (j != e && s_cl[j] == c) cent += 1.0 - De[j];
  if (live) atomicMax(&s_fmax[c], s_fire[e]);
  __syncthreads();
  const bool top = live && s_fire[e] == s_fmax[c];
  if (top) atomicMax(&s_key[c], dkey(cent));
  __syncthreads();
  if (top && dkey(cent) == s_key[c]) atomicMin(&s_idx[c], e);
  __syncthreads();
  if (e < C) {
    dominant[e] = s_idx[e];
    s_isdom[s_idx[e]] = 1;
  }
  __syncthreads();
  if (live) {
    int rank = 0;
    for (int f = 0; f < e; ++f) rank += s_isdom[f] ? 0 : 1;
    cluster_of[e] = c;
    factor_of[e] = s_isdom[e] ? -1 : rank;
  }
  if (e == 0) iterations[0] = it;
}

}  // namespace

hipError_t launch_coact(const int32_t* ids, int N, int k, int E, uint32_t* fire, uint32_t* pair, double* dist,
                        hipStream_t s) {
  const int64_t ee = (int64_t)E * E;
  hipLaunchKernelGGL(k_fill_u32, dim3((unsigned)((ee + 255) / 256)), dim3(256), 0, s, pair, ee);
  hipLaunchKernelGGL(k_fill_u32, dim3((unsigned)((E + 255) / 256)), dim3(256), 0, s, fire, (int64_t)E);
  if (N > 0) {
    const int blocks = (N + 255) / 256 < 512 ? (N + 255) / 256 : 512;
    if (E <= 128)
      hipLaunchKernelGGL(k_coact<true>, dim3(blocks), dim3(256), 0, s, ids, N, k, E, fire, pair);
    else
      hipLaunchKernelGGL(k_coact<false>, dim3(blocks), dim3(256), 0, s, ids, N, k, E, fire, pair);
  }
  hipLaunchKernelGGL(k_npmi, dim3((unsigned)((ee + 255) / 256)), dim3(256), 0, s, fire, pair, N, E, dist);
  hipLaunchKernelGGL(k_mirror, dim3((unsigned)((ee + 255) / 256)), dim3(256), 0, s, pair, E);
  return hipGetLastError();
}

hipError_t launch_kmedoids(const double* dist, const uint32_t* fire, int E, int C, const ProtMask& pm, int P,
                           int max_iter, int32_t* cluster_of, int32_t* factor_of, int32_t* dominant,
                           int32_t* iterations, hipStream_t s) {
  hipLaunchKernelGGL(k_kmedoids, dim3(1), dim3(KM_THR), 0, s, dist, fire, E, C, pm, P, max_iter, cluster_of,
                     factor_of, dominant, iterations);
  return hipGetLastError();
}

}  // namespace lx

// Stage 3 of the compression pipeline on the GPU (Sec. 3, "Alignment and
// low-rank decomposition"), in fp64: the neuron-alignment cost matrix
// (eq. cost), the aligned residual and its rank-r factors from a randomized
// truncated SVD with the symmetric split (eqs. svd and factors). The exact
// assignment between the two (eq. assign) runs on the host. Also the
// activation-weighted fit of the factors (Sec. 4, reconstruction fine-
// tuning; its closed form in Secs. 6-7): minimising ||(R - A B) X^T||^2 +
// damp ||R - A B||^2 over calibration activations X is the rank-r
// truncation of R L (G = X^T X + damp I = L L^T); the same randomized solver
// runs on the operator M = R Xp^T, Xp = [X; sqrt(damp) I], which has the
// left singular vectors and values of R L (M M^T = R G R^T), and B =
// sigma^(-1/2) U_r^T R, so no Cholesky factor of G or its inverse is formed.
//
//   * k_dgemm: C = alpha op(A) op(B) (+ C when accumulate), fp64, 64 x 64
//     output tiles, 16-deep K slabs through LDS, 4 x 4 outputs per thread;
//     the workhorse of every product below (all are thin: one side is the
//     sketch width l = r + p <= 128, or the cost matrix's f x f x 3d).
//   * k_chol: one workgroup, G = R^T R for an l x l Gram matrix in LDS
//     (right-looking, one column per step); k_trsm_rows: Y <- Y R^-1, one
//     thread per row. Twice in a row they make CholeskyQR2, the
//     orthonormalisation of the sketch.
//   * k_jacobi: one workgroup, the eigendecomposition of the l x l matrix
//     Q^T R R^T Q by cyclic Jacobi in the round-robin (tournament) order, so
//     each step rotates l / 2 disjoint pairs at once; matrix in LDS,
//     eigenvectors in global memory; then the eigenpairs sorted descending.
#include "lx_internal.h"

namespace lx {
namespace {

constexpr int DG_T = 64, DG_K = 16;

// Split-K: blockIdx.z takes K range [z kc, (z + 1) kc) and writes its
// partial tile to C + z * M * N (ldc = N); k_dsum adds the partials in z
// order.
__global__ __launch_bounds__(256) void k_dgemm(int M, int N, int K, double alpha, const double* __restrict__ A,
                                               int64_t lda, int ta, const double* __restrict__ B, int64_t ldb, int tb,
                                               double* __restrict__ C, int64_t ldc, int kc) {
  __shared__ double sA[DG_K][DG_T + 1];
  __shared__ double sB[DG_K][DG_T + 1];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int m0 = blockIdx.y * DG_T, n0 = blockIdx.x * DG_T;
  const int kbeg = blockIdx.z * kc, kend = kbeg + kc < K ? kbeg + kc : K;
  C += (int64_t)blockIdx.z * M * N;
  double acc[4][4] = {};
  for (int k0 = kbeg; k0 < kend; k0 += DG_K) {
    for (int q = threadIdx.x; q < DG_K * DG_T; q += 256) {
      const int kk = q / DG_T, mm = q % DG_T;
      const int gm = m0 + mm, gk = k0 + kk;
      double va = 0.0;
      if (gm < M && gk < kend) va = ta ? A[(int64_t)gk * lda + gm] : A[(int64_t)gm * lda + gk];
      sA[kk][mm] = va;
      const int gn = n0 + mm;
      double vb = 0.0;
      if (gn < N && gk < kend) vb = tb ? B[(int64_t)gn * ldb + gk] : B[(int64_t)gk * ldb + gn];
      sB[kk][mm] = vb;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < DG_K; ++kk) {
      double a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = sA[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = sB[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fma(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int gm = m0 + ty * 4 + i, gn = n0 + tx * 4 + j;
      if (gm < M && gn < N) C[(int64_t)gm * ldc + gn] = alpha * acc[i][j];
    }
}

__global__ __launch_bounds__(256) void k_dsum(const double* __restrict__ part, int S, int M, int N,
                                              double* __restrict__ C, int64_t ldc) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= (int64_t)M * N) return;
  double v = part[q];
  for (int z = 1; z < S; ++z) v += part[(int64_t)z * M * N + q];
  C[(q / N) * ldc + q % N] = v;
}

// Neuron vectors of an expert, fp64 [f][3d]: row i = (gate[i, :], up[i, :],
// down[:, i]); bf16 or fp32 storage.
__global__ __launch_bounds__(256) void k_neurons(const void* __restrict__ gate, const void* __restrict__ up,
                                                 const void* __restrict__ down, int bf16, int f, int d,
                                                 double* __restrict__ out, double* __restrict__ norms) {
  const int i = blockIdx.x;
  __shared__ double s_red[256];
  double s = 0.0;
  for (int c = threadIdx.x; c < 3 * d; c += blockDim.x) {
    int64_t src;
    const void* base;
    if (c < d) {
      base = gate;
      src = (int64_t)i * d + c;
    } else if (c < 2 * d) {
      base = up;
      src = (int64_t)i * d + (c - d);
    } else {
      base = down;
      src = (int64_t)(c - 2 * d) * f + i;
    }
    const double v = bf16 ? (double)__uint_as_float((uint32_t)((const uint16_t*)base)[src] << 16)
                          : (double)((const float*)base)[src];
    out[(int64_t)i * 3 * d + c] = v;
    s += v * v;
  }
  s_red[threadIdx.x] = s;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) s_red[threadIdx.x] += s_red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) norms[i] = s_red[0];
}

// C[i][j] = na[i] + nb[j] - 2 G[i][j], in place over G.
__global__ __launch_bounds__(256) void k_cost_finish(const double* __restrict__ na, const double* __restrict__ nb,
                                                     int f, double* __restrict__ G) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= (int64_t)f * f) return;
  G[q] = na[q / f] + nb[q % f] - 2.0 * G[q];
}

// R[i][j] = W_m^P[i][j] - W_dom[i][j]: member rows (axis 0) or columns
// (axis 1) taken in the order perm (null: identity).
__global__ __launch_bounds__(256) void k_residual(const void* __restrict__ wd, const void* __restrict__ wm, int bf16,
                                                  int rows, int cols, const int32_t* __restrict__ perm, int axis,
                                                  double* __restrict__ R) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= (int64_t)rows * cols) return;
  const int i = (int)(q / cols), j = (int)(q % cols);
  int pi = perm && axis == 0 ? perm[i] : i, pj = perm && axis == 1 ? perm[j] : j;
  // a permutation entry out of range reads a clamped (valid) element
  pi = pi < 0 ? 0 : pi >= rows ? rows - 1 : pi;
  pj = pj < 0 ? 0 : pj >= cols ? cols - 1 : pj;
  const int64_t sm = (int64_t)pi * cols + pj;
  double vd, vm;
  if (bf16) {
    vd = (double)__uint_as_float((uint32_t)((const uint16_t*)wd)[q] << 16);
    vm = (double)__uint_as_float((uint32_t)((const uint16_t*)wm)[sm] << 16);
  } else {
    vd = (double)((const float*)wd)[q];
    vm = (double)((const float*)wm)[sm];
  }
  R[q] = vm - vd;
}

// Cholesky of the l x l Gram matrix G (row-major), upper factor U with
// G = U^T U written to Rf (zero below the diagonal).
// A pivot at or below 1e-14 of the largest diagonal entry of G (a direction
// the sketch does not have: exactly low-rank residuals) gives a zero row of
// U, and k_trsm_rows then a zero column of Q; the directions kept stay
// orthonormal and the zero ones carry no weight in Q^T R.
__global__ __launch_bounds__(1024) void k_chol(const double* __restrict__ G, int l, double* __restrict__ Rf) {
  extern __shared__ double s_g[];  // [l][l]
  __shared__ double s_gmax;
  const int tid = threadIdx.x, nth = blockDim.x;
  for (int q = tid; q < l * l; q += nth) s_g[q] = G[q];
  __syncthreads();
  if (tid == 0) {
    double g = 0.0;
    for (int k = 0; k < l; ++k) g = fmax(g, s_g[k * l + k]);
    s_gmax = g;
  }
  __syncthreads();
  const double floor_ = 1e-14 * s_gmax;
  for (int k = 0; k < l; ++k) {
    // row k of U: U[k][k] = sqrt(G[k][k]), U[k][j] = G[k][j] / U[k][k]
    __syncthreads();
    const double pk = s_g[k * l + k];
    const double dkk = pk > floor_ ? sqrt(pk) : 0.0;
    __syncthreads();
    for (int j = k + tid; j < l; j += nth) s_g[k * l + j] = j == k ? dkk : (dkk > 0.0 ? s_g[k * l + j] / dkk : 0.0);
    __syncthreads();
    // trailing update: G[i][j] -= U[k][i] U[k][j] for i, j > k
    const int m = l - k - 1;
    for (int q = tid; q < m * m; q += nth) {
      const int i = k + 1 + q / m, j = k + 1 + q % m;
      s_g[i * l + j] -= s_g[k * l + i] * s_g[k * l + j];
    }
  }
  __syncthreads();
  for (int q = tid; q < l * l; q += nth) Rf[q] = (q % l) >= (q / l) ? s_g[q] : 0.0;
}

// Y[i, :] <- Y[i, :] U^-1 for the upper-triangular l x l U: x U = y, solved
// left to right, one thread per row; U and the workgroup's rw rows (pitch
// l + 1) staged in LDS.
__global__ __launch_bounds__(64) void k_trsm_rows(double* __restrict__ Y, int rows, int l, int rw,
                                                  const double* __restrict__ U) {
  extern __shared__ double s_t[];
  double* const su = s_t;
  double* const sy = s_t + l * l;
  const int r0 = blockIdx.x * rw, tid = threadIdx.x;
  const int nr = rows - r0 < rw ? rows - r0 : rw;
  for (int q = tid; q < l * l; q += 64) su[q] = U[q];
  for (int q = tid; q < nr * l; q += 64) sy[(q / l) * (l + 1) + q % l] = Y[(int64_t)(r0 + q / l) * l + q % l];
  __syncthreads();
  if (tid < nr) {
    double* const y = sy + tid * (l + 1);
    for (int j = 0; j < l; ++j) {
      double acc = y[j];
      for (int k = 0; k < j; ++k) acc -= y[k] * su[k * l + j];
      const double ujj = su[j * l + j];
      y[j] = ujj != 0.0 ? acc / ujj : 0.0;
    }
  }
  __syncthreads();
  for (int q = tid; q < nr * l; q += 64) Y[(int64_t)(r0 + q / l) * l + q % l] = sy[(q / l) * (l + 1) + q % l];
}

inline int trsm_rows_per_wg(int l) { return l <= 96 ? 64 : 16; }
inline size_t trsm_lds(int l) { return ((size_t)l * l + (size_t)trsm_rows_per_wg(l) * (l + 1)) * sizeof(double); }

// Eigendecomposition of the symmetric l x l M (l even after padding with a
// zero row/column when odd): cyclic Jacobi, round-robin pair order; V
// (lp x lp row-major, in LDS when both fit, else global) accumulates the
// rotations. Output: eigenvalues
// descending in w[0..l), eigenvectors as columns of Vs (sorted).
template <bool VLDS>
__global__ __launch_bounds__(1024) void k_jacobi(const double* __restrict__ Min, int l, int lp,
                                                 double* __restrict__ Vg, double* __restrict__ w,
                                                 double* __restrict__ Vs, int max_sweeps) {
  extern __shared__ double s_m[];  // [lp][lp], then V [lp][lp] when VLDS
  double* const V = VLDS ? s_m + lp * lp : Vg;
  __shared__ int s_p[64], s_q[64];
  __shared__ double s_c[64], s_s[64];
  __shared__ int s_order[128];
  __shared__ double s_red[1024];
  const int tid = threadIdx.x, nth = blockDim.x;
  for (int q = tid; q < lp * lp; q += nth) {
    const int i = q / lp, j = q % lp;
    s_m[q] = (i < l && j < l) ? Min[i * l + j] : 0.0;
    V[q] = i == j ? 1.0 : 0.0;
  }
  __syncthreads();
  // sum of squares of all entries (diag = 1) or of the off-diagonal ones
  auto sumsq = [&](bool diag) {
    double t = 0.0;
    for (int q = tid; q < lp * lp; q += nth)
      if (diag || q / lp != q % lp) t += s_m[q] * s_m[q];
    s_red[tid] = t;
    __syncthreads();
    for (int o = nth / 2; o > 0; o >>= 1) {
      if (tid < o) s_red[tid] += s_red[tid + o];
      __syncthreads();
    }
    const double r = s_red[0];
    __syncthreads();
    return r;
  };
  const double norm0 = sumsq(true);
  const int half = lp / 2;
  for (int sweep = 0; sweep < max_sweeps; ++sweep) {
    if (!(sumsq(false) > 1e-30 * norm0)) break;
    for (int step = 0; step < lp - 1; ++step) {
      // round-robin pairing: element 0 fixed, the others rotate
      if (tid < half) {
        auto pos = [&](int x) { return x == 0 ? 0 : 1 + (x - 1 + step) % (lp - 1); };
        int a = pos(tid), b = pos(lp - 1 - tid);
        const int p = a < b ? a : b, q = a < b ? b : a;
        const double app = s_m[p * lp + p], aqq = s_m[q * lp + q], apq = s_m[p * lp + q];
        double c = 1.0, s = 0.0;
        if (apq != 0.0) {
          const double tau = (aqq - app) / (2.0 * apq);
          const double t = (tau >= 0.0 ? 1.0 : -1.0) / (fabs(tau) + sqrt(1.0 + tau * tau));
          c = 1.0 / sqrt(1.0 + t * t);
          s = t * c;
        }
        s_p[tid] = p;
        s_q[tid] = q;
        s_c[tid] = c;
        s_s[tid] = s;
      }
      __syncthreads();
      // rows: M <- J^T M (rows p, q of every pair, all columns)
      for (int x = tid; x < half * lp; x += nth) {
        const int k = x / lp, j = x % lp;
        const int p = s_p[k], q = s_q[k];
        const double c = s_c[k], s = s_s[k];
        const double mp = s_m[p * lp + j], mq = s_m[q * lp + j];
        s_m[p * lp + j] = c * mp - s * mq;
        s_m[q * lp + j] = s * mp + c * mq;
      }
      __syncthreads();
      // columns: M <- M J, and V <- V J
      for (int x = tid; x < half * lp; x += nth) {
        const int k = x / lp, i = x % lp;
        const int p = s_p[k], q = s_q[k];
        const double c = s_c[k], s = s_s[k];
        const double mp = s_m[i * lp + p], mq = s_m[i * lp + q];
        s_m[i * lp + p] = c * mp - s * mq;
        s_m[i * lp + q] = s * mp + c * mq;
        const double vp = V[i * lp + p], vq = V[i * lp + q];
        V[i * lp + p] = c * vp - s * vq;
        V[i * lp + q] = s * vp + c * vq;
      }
      __syncthreads();
    }
  }
  // sort descending (ties: lower index first), keep the first l
  if (tid < lp) {
    const double e = s_m[tid * lp + tid];
    int rank = 0;
    for (int j = 0; j < lp; ++j) {
      const double o = s_m[j * lp + j];
      if (o > e || (o == e && j < tid)) ++rank;
    }
    s_order[rank] = tid;
  }
  __syncthreads();
  for (int x = tid; x < l * l; x += nth) {
    const int i = x / l, r = x % l;  // row i of eigenvector column r
    Vs[x] = V[i * lp + s_order[r]];
  }
  if (tid < l) w[tid] = s_m[s_order[tid] * lp + s_order[tid]];
}

// X[i][j] *= sqrt(s[k]) (or /= when invert; 0 where s[k] = 0), k = j
// (by_col) or i: the symmetric split of the singular values.
__global__ __launch_bounds__(256) void k_scale(double* __restrict__ X, int rows, int cols, const double* __restrict__ s,
                                               int by_col, int invert) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= (int64_t)rows * cols) return;
  const int k = by_col ? (int)(q % cols) : (int)(q / cols);
  const double sg = sqrt(s[k] > 0.0 ? s[k] : 0.0);
  X[q] = invert ? (sg > 0.0 ? X[q] / sg : 0.0) : X[q] * sg;
}

__global__ __launch_bounds__(256) void k_sqrt_vec(const double* __restrict__ lam, int n, double* __restrict__ sig) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) sig[i] = sqrt(lam[i] > 0.0 ? lam[i] : 0.0);
}

__global__ __launch_bounds__(256) void k_copy_f64(const double* __restrict__ x, int n, double* __restrict__ y) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) y[i] = x[i];
}

// Xp = [X; sqrt(damp) I]: rows i < n the activations X [n][cols] (bf16 or
// fp32) in fp64, rows n .. np - 1 the scaled identity (np = n or n + cols).
__global__ __launch_bounds__(256) void k_fill_act(const void* __restrict__ x, int bf16, int n, int cols, double sd,
                                                  int np, double* __restrict__ Xp) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= (int64_t)np * cols) return;
  const int i = (int)(q / cols), j = (int)(q % cols);
  if (i < n)
    Xp[q] = bf16 ? (double)__uint_as_float((uint32_t)((const uint16_t*)x)[q] << 16) : (double)((const float*)x)[q];
  else
    Xp[q] = j == i - n ? sd : 0.0;
}

__global__ __launch_bounds__(256) void k_to_f32(const double* __restrict__ x, int64_t n, float* __restrict__ y) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q < n) y[q] = (float)x[q];
}

inline unsigned blocks(int64_t n, int t = 256) { return (unsigned)((n + t - 1) / t); }

// Partial tiles for the split products: at most kDgParts doubles.
constexpr int64_t kDgParts = 384 * DG_T * DG_T;

// C = alpha op(A) op(B). With few output tiles and a long K the K range is
// split (at least 4 slabs of 16 per split, about 256 workgroups in all) over
// the partial buffer part (kDgParts doubles, may be null: no split).
hipError_t dgemm(int M, int N, int K, double alpha, const double* A, int64_t lda, int ta, const double* B, int64_t ldb,
                 int tb, double* C, int64_t ldc, hipStream_t s, double* part) {
  if (M <= 0 || N <= 0) return hipSuccess;
  const int tiles = ((M + DG_T - 1) / DG_T) * ((N + DG_T - 1) / DG_T);
  int S = 1;
  if (part && tiles < 128) {
    S = (256 + tiles - 1) / tiles;
    const int smax = K / (4 * DG_K);
    S = S < smax ? S : smax;
    while (S > 1 && (int64_t)S * M * N > kDgParts) --S;
    if (S < 1) S = 1;
  }
  const dim3 grid((N + DG_T - 1) / DG_T, (M + DG_T - 1) / DG_T, S);
  if (S == 1) {
    hipLaunchKernelGGL(k_dgemm, grid, dim3(256), 0, s, M, N, K, alpha, A, lda, ta, B, ldb, tb, C, ldc, K);
    return hipGetLastError();
  }
  const int kc = ((K + S - 1) / S + DG_K - 1) / DG_K * DG_K;
  hipLaunchKernelGGL(k_dgemm, grid, dim3(256), 0, s, M, N, K, alpha, A, lda, ta, B, ldb, tb, part, (int64_t)N, kc);
  hipLaunchKernelGGL(k_dsum, dim3(blocks((int64_t)M * N)), dim3(256), 0, s, part, S, M, N, C, ldc);
  return hipGetLastError();
}

// Y (rows x l) <- its orthonormal basis, CholeskyQR2; G, U: l x l scratch.
// Kernels with up to 128 KB of dynamic LDS: allow it once per process.
hipError_t allow_lds() {
  static hipError_t e = [] {
    const hipFuncAttribute a = hipFuncAttributeMaxDynamicSharedMemorySize;
    hipError_t r = hipFuncSetAttribute((const void*)k_chol, a, 128 * 1024);
    if (r == hipSuccess) r = hipFuncSetAttribute((const void*)k_jacobi<false>, a, 128 * 1024);
    if (r == hipSuccess) r = hipFuncSetAttribute((const void*)k_jacobi<true>, a, 2 * 96 * 96 * 8);
    if (r == hipSuccess) r = hipFuncSetAttribute((const void*)k_trsm_rows, a, 148 * 1024);
    return r;
  }();
  return e;
}

hipError_t cholqr2(double* Y, int rows, int l, double* G, double* U, hipStream_t s, double* part) {
  for (int pass = 0; pass < 2; ++pass) {
    hipError_t e = dgemm(l, l, rows, 1.0, Y, l, 1, Y, l, 0, G, l, s, part);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_chol, dim3(1), dim3(1024), (size_t)l * l * sizeof(double), s, G, l, U);
    const int rw = trsm_rows_per_wg(l);
    hipLaunchKernelGGL(k_trsm_rows, dim3((rows + rw - 1) / rw), dim3(64), trsm_lds(l), s, Y, rows, l, rw, U);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

// From an orthonormal sketch Y (rows x l) of the range of an operator M, T =
// Y^T R (l x cols) and Gm = (Y^T M)(Y^T M)^T (l x l): the eigenpairs of Gm
// (descending), sigma = the square roots of the r largest, A = Y Ut[:, :r]
// sigma^(1/2) and B = sigma^(-1/2) Ut[:, :r]^T T (rows of B with sigma = 0
// are 0); Bd (r x cols doubles) is scratch.
hipError_t factors_from_sketch(int rows, int cols, int r, int l, const double* Y, const double* T, const double* Gm,
                               double* V, double* lam, double* Ve, double* sig, double* Ad, double* Bd, float* A,
                               float* B, double* sigma, hipStream_t s, double* part) {
  const int lp = l + (l & 1);
  if (lp <= 96)
    hipLaunchKernelGGL(k_jacobi<true>, dim3(1), dim3(1024), 2 * (size_t)lp * lp * sizeof(double), s, Gm, l, lp, V, lam,
                       Ve, 40);
  else
    hipLaunchKernelGGL(k_jacobi<false>, dim3(1), dim3(1024), (size_t)lp * lp * sizeof(double), s, Gm, l, lp, V, lam,
                       Ve, 40);
  hipLaunchKernelGGL(k_sqrt_vec, dim3(1), dim3(256), 0, s, lam, r, sig);
  hipError_t e;
  if ((e = dgemm(rows, r, l, 1.0, Y, l, 0, Ve, l, 0, Ad, r, s, part)) != hipSuccess) return e;
  hipLaunchKernelGGL(k_scale, dim3(blocks((int64_t)rows * r)), dim3(256), 0, s, Ad, rows, r, sig, 1, 0);
  hipLaunchKernelGGL(k_to_f32, dim3(blocks((int64_t)rows * r)), dim3(256), 0, s, Ad, (int64_t)rows * r, A);
  if ((e = dgemm(r, cols, l, 1.0, Ve, l, 1, T, cols, 0, Bd, cols, s, part)) != hipSuccess) return e;
  hipLaunchKernelGGL(k_scale, dim3(blocks((int64_t)r * cols)), dim3(256), 0, s, Bd, r, cols, sig, 0, 1);
  hipLaunchKernelGGL(k_to_f32, dim3(blocks((int64_t)r * cols)), dim3(256), 0, s, Bd, (int64_t)r * cols, B);
  hipLaunchKernelGGL(k_copy_f64, dim3(1), dim3(256), 0, s, sig, r, sigma);
  return hipGetLastError();
}

}  // namespace

size_t lowrank_ws_doubles(int rows, int cols, int l) {
  const int lp = l + (l & 1);
  return (size_t)rows * cols + (size_t)rows * l + (size_t)cols * l + (size_t)l * cols + 4 * (size_t)lp * lp + 2 * lp +
         (size_t)rows * l + (size_t)kDgParts;
}

size_t weighted_ws_doubles(int rows, int cols, int np, int l) {
  const int lp = l + (l & 1);
  return (size_t)rows * cols + (size_t)np * cols + (size_t)cols * l + (size_t)rows * l + (size_t)np * l +
         (size_t)l * cols + (size_t)l * np + 4 * (size_t)lp * lp + 2 * lp + (size_t)rows * l + (size_t)kDgParts;
}

hipError_t launch_align_cost(const void* dg, const void* du, const void* dd, const void* mg, const void* mu,
                             const void* md, int bf16, int f, int d, double* cost, double* ws, hipStream_t s) {
  double* const a = ws;
  double* const b = a + (size_t)f * 3 * d;
  double* const na = b + (size_t)f * 3 * d;
  double* const nb = na + f;
  hipLaunchKernelGGL(k_neurons, dim3(f), dim3(256), 0, s, dg, du, dd, bf16, f, d, a, na);
  hipLaunchKernelGGL(k_neurons, dim3(f), dim3(256), 0, s, mg, mu, md, bf16, f, d, b, nb);
  hipError_t e = dgemm(f, f, 3 * d, 1.0, a, 3 * d, 0, b, 3 * d, 1, cost, f, s, nullptr);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_cost_finish, dim3(blocks((int64_t)f * f)), dim3(256), 0, s, na, nb, f, cost);
  return hipGetLastError();
}

hipError_t launch_lowrank(const void* wd, const void* wm, int bf16, int rows, int cols, const int32_t* perm, int axis,
                          int r, int l, int q, const double* omega, float* A, float* B, double* sigma, double* ws,
                          hipStream_t s) {
  const int lp = l + (l & 1);
  if (const hipError_t e0 = allow_lds(); e0 != hipSuccess) return e0;
  double* const R = ws;                              // rows x cols
  double* const Y = R + (size_t)rows * cols;         // rows x l
  double* const Z = Y + (size_t)rows * l;            // cols x l
  double* const Bs = Z + (size_t)cols * l;           // l x cols
  double* const G = Bs + (size_t)l * cols;           // lp x lp (four of them)
  double* const U = G + (size_t)lp * lp;
  double* const V = U + (size_t)lp * lp;
  double* const Ve = V + (size_t)lp * lp;
  double* const lam = Ve + (size_t)lp * lp;          // lp
  double* const sig = lam + lp;                      // lp
  double* const Ad = sig + lp;                       // rows x l (A before truncation)
  double* const part = Ad + (size_t)rows * l;        // kDgParts (split-K partial tiles)
  hipLaunchKernelGGL(k_residual, dim3(blocks((int64_t)rows * cols)), dim3(256), 0, s, wd, wm, bf16, rows, cols, perm,
                     axis, R);
  hipError_t e;
  // Y = R Omega, orthonormalised; q rounds of Z = R^T Y, Y = R Z, each
  // orthonormalised
  if ((e = dgemm(rows, l, cols, 1.0, R, cols, 0, omega, l, 0, Y, l, s, part)) != hipSuccess) return e;
  if ((e = cholqr2(Y, rows, l, G, U, s, part)) != hipSuccess) return e;
  for (int it = 0; it < q; ++it) {
    if ((e = dgemm(cols, l, rows, 1.0, R, cols, 1, Y, l, 0, Z, l, s, part)) != hipSuccess) return e;
    if ((e = cholqr2(Z, cols, l, G, U, s, part)) != hipSuccess) return e;
    if ((e = dgemm(rows, l, cols, 1.0, R, cols, 0, Z, l, 0, Y, l, s, part)) != hipSuccess) return e;
    if ((e = cholqr2(Y, rows, l, G, U, s, part)) != hipSuccess) return e;
  }
  // Bs = Y^T R (l x cols); Bs Bs^T (l x l) = Ut diag(lambda) Ut^T
  if ((e = dgemm(l, cols, rows, 1.0, Y, l, 1, R, cols, 0, Bs, cols, s, part)) != hipSuccess) return e;
  if ((e = dgemm(l, l, cols, 1.0, Bs, cols, 0, Bs, cols, 1, G, l, s, part)) != hipSuccess) return e;
  return factors_from_sketch(rows, cols, r, l, Y, Bs, G, V, lam, Ve, sig, Ad, Z, A, B, sigma, s, part);
}

hipError_t launch_weighted(const void* wd, const void* wm, int bf16, int rows, int cols, const int32_t* perm, int axis,
                           const void* x, int x_bf16, int n, double damp, int r, int l, int q, const double* omega,
                           float* A, float* B, double* sigma, double* ws, hipStream_t s) {
  const int lp = l + (l & 1);
  const int np = n + (damp > 0.0 ? cols : 0);
  if (const hipError_t e0 = allow_lds(); e0 != hipSuccess) return e0;
  double* const R = ws;                              // rows x cols
  double* const Xp = R + (size_t)rows * cols;        // np x cols: [X; sqrt(damp) I]
  double* const P = Xp + (size_t)np * cols;          // cols x l
  double* const Y = P + (size_t)cols * l;            // rows x l
  double* const Z = Y + (size_t)rows * l;            // np x l
  double* const T = Z + (size_t)np * l;              // l x cols
  double* const Wt = T + (size_t)l * cols;           // l x np
  double* const G = Wt + (size_t)l * np;             // lp x lp (four of them)
  double* const U = G + (size_t)lp * lp;
  double* const V = U + (size_t)lp * lp;
  double* const Ve = V + (size_t)lp * lp;
  double* const lam = Ve + (size_t)lp * lp;          // lp
  double* const sig = lam + lp;                      // lp
  double* const Ad = sig + lp;                       // rows x l
  double* const part = Ad + (size_t)rows * l;        // kDgParts
  hipLaunchKernelGGL(k_residual, dim3(blocks((int64_t)rows * cols)), dim3(256), 0, s, wd, wm, bf16, rows, cols, perm,
                     axis, R);
  hipLaunchKernelGGL(k_fill_act, dim3(blocks((int64_t)np * cols)), dim3(256), 0, s, x, x_bf16, n, cols, sqrt(damp),
                     np, Xp);
  hipError_t e;
  // The operator M = R Xp^T (rows x np), applied as two thin products:
  // Y = R (Xp^T Omega), orthonormalised; q rounds of Z = Xp (R^T Y) and
  // Y = R (Xp^T Z), each orthonormalised
  if ((e = dgemm(cols, l, np, 1.0, Xp, cols, 1, omega, l, 0, P, l, s, part)) != hipSuccess) return e;
  if ((e = dgemm(rows, l, cols, 1.0, R, cols, 0, P, l, 0, Y, l, s, part)) != hipSuccess) return e;
  if ((e = cholqr2(Y, rows, l, G, U, s, part)) != hipSuccess) return e;
  for (int it = 0; it < q; ++it) {
    if ((e = dgemm(cols, l, rows, 1.0, R, cols, 1, Y, l, 0, P, l, s, part)) != hipSuccess) return e;
    if ((e = dgemm(np, l, cols, 1.0, Xp, cols, 0, P, l, 0, Z, l, s, part)) != hipSuccess) return e;
    if ((e = cholqr2(Z, np, l, G, U, s, part)) != hipSuccess) return e;
    if ((e = dgemm(cols, l, np, 1.0, Xp, cols, 1, Z, l, 0, P, l, s, part)) != hipSuccess) return e;
    if ((e = dgemm(rows, l, cols, 1.0, R, cols, 0, P, l, 0, Y, l, s, part)) != hipSuccess) return e;
    if ((e = cholqr2(Y, rows, l, G, U, s, part)) != hipSuccess) return e;
  }
  // T = Y^T R (l x cols); Wt = Y^T M = T Xp^T (l x np); Wt Wt^T = Ut diag(lambda) Ut^T.
  // B = sigma^(-1/2) Ut^T T is sigma^(-1/2) U_r^T R with U_r = Y Ut[:, :r].
  if ((e = dgemm(l, cols, rows, 1.0, Y, l, 1, R, cols, 0, T, cols, s, part)) != hipSuccess) return e;
  if ((e = dgemm(l, np, cols, 1.0, T, cols, 0, Xp, cols, 1, Wt, np, s, part)) != hipSuccess) return e;
  if ((e = dgemm(l, l, np, 1.0, Wt, np, 0, Wt, np, 1, G, l, s, part)) != hipSuccess) return e;
  return factors_from_sketch(rows, cols, r, l, Y, T, G, V, lam, Ve, sig, Ad, P, A, B, sigma, s, part);
}

}  // namespace lx

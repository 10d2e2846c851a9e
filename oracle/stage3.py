"""fp64 reference of Stage 3, factor production (test infrastructure).

THIS MODULE IS TEST INFRASTRUCTURE, like the rest of the package: only the
test suite, the smoke check and the benchmark's CPU-baseline leg use it.

What it follows (Sec. 3 "Compression pipeline", Stage 3, in this library's
notation: weights [out][in], A output-side, B input-side, W ~ W_dom + A B):

* (i) neuron alignment: neuron i of an expert is the concatenation of gate
  row i, up row i and down column i (eq. cost); the cost of matching the
  dominant's neuron i with the member's neuron j is the squared distance
  ||a_i||^2 + ||b_j||^2 - 2 a_i . b_j; the permutation minimising the summed
  cost (eq. assign) is solved exactly (here: scipy's linear_sum_assignment,
  a library routine for the same problem the paper solves with
  Jonker-Volgenant). perm[i] = the member neuron matched to dominant neuron i;
  the aligned member has gate/up rows perm and down columns perm.
* (ii) the aligned residual R = W_m^P - W_dom per projection and its rank-r
  truncated SVD from a randomized solver (eq. svd), split symmetrically
  (eq. factors): A = U_r Sigma_r^(1/2), B = Sigma_r^(1/2) V_r^T.
  Randomized solver (reading; the paper names only "randomized" and r = 64):
  the subspace iteration of Halko, Martinsson and Tropp (2011), their
  Algorithm 4.4, with a Gaussian test matrix Omega [cols][r + p] passed in,
  p = 10 oversampling columns and q = 2 power iterations, each product
  re-orthonormalised (QR), then the SVD of the small matrix Q^T R.
* (iii) the activation-weighted fit (Sec. 4, reconstruction fine-tuning;
  its closed form in Sec. 6 "Calibration cost" and Sec. 7 "Hessian-weighted
  fitting"): the rank-r (A, B) that minimise the error of the emitted
  output on calibration activations X [n][cols] (rows = tokens),
  ||(R - A B) X^T||_F^2 + damp ||R - A B||_F^2 (damp >= 0: the damping the
  paper leaves unspecified, read as a ridge term). With G = X^T X + damp I =
  L L^T, the objective is ||(R - A B) L||_F^2, so the optimum is the rank-r
  truncation of R L: R L = U S V^T, A = U_r S_r^(1/2), B = S_r^(1/2) V_r^T
  L^(-1) (weighted_factors_exact). The library's route to the same optimum
  (weighted_factors): M = R X'^T with X' = [X; sqrt(damp) I] has M M^T =
  R G R^T, so M and R L share left singular vectors and values; the
  randomized solver above runs on M with a test matrix Omega [n (+ cols)]
  [r + p], and B = S_r^(-1/2) U_r^T R (equal to the formula above, since
  U_r^T R L = S_r V_r^T); rows of B (and columns of A) whose singular value
  is 0 are 0.
"""
from __future__ import annotations

import numpy as np
from scipy.optimize import linear_sum_assignment

from .moe import to_f64


def neuron_vectors(gate, up, down, dtype: str) -> np.ndarray:
    """[f, 3d] fp64: row i = (gate[i, :], up[i, :], down[:, i])."""
    return np.concatenate([to_f64(gate, dtype), to_f64(up, dtype), to_f64(down, dtype).T], axis=1)


def align_cost(dom, mem, dtype: str) -> np.ndarray:
    """C[i, j] = ||a_i||^2 + ||b_j||^2 - 2 a_i . b_j, [f, f] fp64; dom and mem
    are (gate, up, down) triples."""
    a = neuron_vectors(*dom, dtype)
    b = neuron_vectors(*mem, dtype)
    return (a * a).sum(1)[:, None] + (b * b).sum(1)[None, :] - 2.0 * (a @ b.T)


def assign(C):
    """(perm int64 [n], total cost) of the exact minimum-cost matching."""
    rows, cols = linear_sum_assignment(np.asarray(C, np.float64))
    perm = np.empty(len(rows), np.int64)
    perm[rows] = cols
    return perm, float(np.asarray(C)[rows, cols].sum())


def aligned_residual(w_dom, w_mem, perm, axis: int, dtype: str) -> np.ndarray:
    """R = W_m^P - W_dom with the member's rows (axis 0) or columns (axis 1)
    taken in the order perm."""
    m = to_f64(w_mem, dtype)
    m = m[perm, :] if axis == 0 else m[:, perm]
    return m - to_f64(w_dom, dtype)


def _orth(Y):
    q, _ = np.linalg.qr(Y)
    return q


def randomized_svd(R, omega, r: int, q: int = 2):
    """(U_r [rows, r], sigma [r], Vt_r [r, cols]) by subspace iteration."""
    Q = _orth(R @ omega)
    for _ in range(q):
        Qt = _orth(R.T @ Q)
        Q = _orth(R @ Qt)
    Bs = Q.T @ R
    Ut, s, Vt = np.linalg.svd(Bs, full_matrices=False)
    return Q @ Ut[:, :r], s[:r], Vt[:r]


def factors(R, omega, r: int, q: int = 2):
    """(A [rows, r], B [r, cols], sigma [r]) with A B the rank-r approximation."""
    U, s, Vt = randomized_svd(R, omega, r, q)
    h = np.sqrt(s)
    return U * h[None, :], h[:, None] * Vt, s


def whitened_moment(X, damp: float = 0.0):
    """G = X^T X + damp I for activations X [n][cols] (fp64)."""
    X = np.asarray(X, np.float64)
    return X.T @ X + damp * np.eye(X.shape[1])


def weighted_factors_exact(R, X, r: int, damp: float = 0.0):
    """(A [rows, r], B [r, cols], sigma [r]) minimising ||(R - A B) X^T||_F^2 +
    damp ||R - A B||_F^2: whitening by G = L L^T, exact SVD of R L. G must be
    positive definite (damp > 0, or X of full column rank)."""
    L = np.linalg.cholesky(whitened_moment(X, damp))
    U, s, Vt = np.linalg.svd(np.asarray(R, np.float64) @ L, full_matrices=False)
    h = np.sqrt(s[:r])
    A = U[:, :r] * h[None, :]
    # B = S^(1/2) V_r^T L^(-1): solve L^T B^T = (S^(1/2) V_r^T)^T
    B = np.linalg.solve(L.T, (h[:, None] * Vt[:r]).T).T
    return A, B, s[:r]


def weighted_objective(R, X, A, B, damp: float = 0.0) -> float:
    """sqrt(||(R - A B) X^T||_F^2 + damp ||R - A B||_F^2)."""
    E = np.asarray(R, np.float64) - np.asarray(A, np.float64) @ np.asarray(B, np.float64)
    X = np.asarray(X, np.float64)
    return float(np.sqrt(np.linalg.norm(E @ X.T) ** 2 + damp * np.linalg.norm(E) ** 2))


def weighted_operator(R, X, damp: float = 0.0):
    """M = R X'^T, X' = [X; sqrt(damp) I] ([rows][n (+ cols)])."""
    X = np.asarray(X, np.float64)
    if damp > 0:
        X = np.vstack([X, np.sqrt(damp) * np.eye(X.shape[1])])
    return np.asarray(R, np.float64) @ X.T


def weighted_factors(R, X, omega, r: int, q: int = 2, damp: float = 0.0):
    """The randomized route: subspace iteration on M = R X'^T with the
    caller's test matrix omega [n (+ cols)][r + p]; A = U_r S^(1/2),
    B = S^(-1/2) U_r^T R (zero where S is 0)."""
    R = np.asarray(R, np.float64)
    U, s, _ = randomized_svd(weighted_operator(R, X, damp), omega, r, q)
    h = np.sqrt(s)
    inv = np.where(h > 0, 1.0 / np.where(h > 0, h, 1.0), 0.0)
    return U * h[None, :], inv[:, None] * (U.T @ R), s

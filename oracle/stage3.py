"""fp64 reference of Stage 3, factor production (test infrastructure).

THIS MODULE IS TEST INFRASTRUCTURE, like the rest of the package: only the
test suite, the smoke check and the benchmark's CPU-baseline leg use it.

What it follows (Sec. 3 "Compression pipeline", Stage 3, in the build's
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

"""Pins of the Stage-3 oracle: alignment cost and exact assignment against
brute force and planted permutations; the randomized truncated SVD against
exact SVDs (Eckart-Young) and exactly low-rank matrices."""
import itertools

import numpy as np
import pytest

from lxsynth import f32_to_bf16_bits
from oracle import stage3 as S


def _bf16(a):
    return f32_to_bf16_bits(np.asarray(a, np.float32))


def _expert(rng, f, d, scale=1.0):
    return tuple(_bf16(rng.standard_normal(s) * scale) for s in ((f, d), (f, d), (d, f)))


def test_cost_is_pairwise_squared_distance():
    rng = np.random.default_rng(1)
    dom, mem = _expert(rng, 5, 7), _expert(rng, 5, 7)
    C = S.align_cost(dom, mem, "bf16")
    a, b = S.neuron_vectors(*dom, "bf16"), S.neuron_vectors(*mem, "bf16")
    for i in range(5):
        for j in range(5):
            assert C[i, j] == pytest.approx(float(((a[i] - b[j]) ** 2).sum()), rel=1e-12)


def test_assignment_matches_brute_force():
    rng = np.random.default_rng(2)
    for n in (2, 5, 7):
        C = rng.random((n, n))
        perm, total = S.assign(C)
        best = min(sum(C[i, p[i]] for i in range(n)) for p in itertools.permutations(range(n)))
        assert total == pytest.approx(best, abs=1e-12)
        assert sorted(perm.tolist()) == list(range(n))


def test_planted_permutation_is_recovered_and_residual_vanishes():
    """A member that is its dominant with neurons shuffled (plus tiny noise)
    aligns back exactly; with no noise the aligned residual is zero."""
    rng = np.random.default_rng(3)
    f, d = 24, 16
    g, u, dn = (rng.standard_normal(s) for s in ((f, d), (f, d), (d, f)))
    pi = rng.permutation(f)                      # member neuron pi[i] = dominant neuron i
    inv = np.argsort(pi)
    dom = (_bf16(g), _bf16(u), _bf16(dn))
    mem = (_bf16(g[inv]), _bf16(u[inv]), _bf16(dn[:, inv]))
    perm, total = S.assign(S.align_cost(dom, mem, "bf16"))
    assert np.array_equal(perm, pi) and total == pytest.approx(0.0, abs=1e-9)
    assert np.all(S.aligned_residual(dom[0], mem[0], perm, 0, "bf16") == 0)
    assert np.all(S.aligned_residual(dom[2], mem[2], perm, 1, "bf16") == 0)


def test_randomized_svd_exact_on_low_rank_and_close_to_truncated_svd():
    rng = np.random.default_rng(4)
    rows, cols, r, p = 120, 90, 12, 10
    # exactly rank r: recovered to rounding
    R = rng.standard_normal((rows, r)) @ rng.standard_normal((r, cols))
    om = rng.standard_normal((cols, r + p))
    A, B, s = S.factors(R, om, r)
    assert np.linalg.norm(A @ B - R) <= 1e-10 * np.linalg.norm(R)
    assert np.allclose(s, np.linalg.svd(R, compute_uv=False)[:r], rtol=1e-10)
    # full rank with a decaying spectrum: close to the Eckart-Young optimum
    U0, _ = np.linalg.qr(rng.standard_normal((rows, cols)))
    V0, _ = np.linalg.qr(rng.standard_normal((cols, cols)))
    sig = 0.8 ** np.arange(cols)
    R2 = (U0 * sig) @ V0.T
    A2, B2, s2 = S.factors(R2, om, r)
    opt = np.sqrt((sig[r:] ** 2).sum())
    assert np.linalg.norm(R2 - A2 @ B2) <= 1.01 * opt
    assert np.allclose(s2, sig[:r], rtol=1e-3)
    # symmetric split: A^T A = B B^T = diag(sigma)
    assert np.allclose(A2.T @ A2, np.diag(s2), atol=1e-10)
    assert np.allclose(B2 @ B2.T, np.diag(s2), atol=1e-10)


def _decaying(rng, rows, cols, rate=0.7):
    U0, _ = np.linalg.qr(rng.standard_normal((rows, min(rows, cols))))
    V0, _ = np.linalg.qr(rng.standard_normal((cols, min(rows, cols))))
    return (U0 * rate ** np.arange(min(rows, cols))) @ V0.T


@pytest.mark.parametrize("damp", [0.0, 0.5])
def test_weighted_fit_reaches_the_closed_form_optimum(damp):
    """The fit's emitted error equals the Eckart-Young bound of R L (the tail
    of its singular values), and no perturbation of (A, B) lowers it."""
    rng = np.random.default_rng(5)
    rows, cols, n, r = 30, 20, 60, 4
    R = rng.standard_normal((rows, cols))
    X = rng.standard_normal((n, cols)) * np.linspace(0.2, 3.0, cols)[None, :]
    A, B, s = S.weighted_factors_exact(R, X, r, damp)
    L = np.linalg.cholesky(X.T @ X + damp * np.eye(cols))
    sv = np.linalg.svd(R @ L, compute_uv=False)
    best = S.weighted_objective(R, X, A, B, damp)
    assert best == pytest.approx(np.sqrt((sv[r:] ** 2).sum()), rel=1e-10)
    assert np.allclose(s, sv[:r], rtol=1e-12)
    for _ in range(20):
        dA, dB = rng.standard_normal(A.shape) * 1e-3, rng.standard_normal(B.shape) * 1e-3
        assert S.weighted_objective(R, X, A + dA, B + dB, damp) >= best * (1 - 1e-12)
    # the plain (unweighted) truncation is worse in the weighted norm
    U, sp, Vt = np.linalg.svd(R, full_matrices=False)
    assert S.weighted_objective(R, X, U[:, :r] * sp[:r], Vt[:r], damp) > best * 1.001


def test_weighted_fit_with_identity_activations_is_the_plain_truncation():
    rng = np.random.default_rng(6)
    R = rng.standard_normal((25, 18))
    A, B, s = S.weighted_factors_exact(R, np.eye(18), 5)
    U, sp, Vt = np.linalg.svd(R, full_matrices=False)
    assert np.allclose(A @ B, (U[:, :5] * sp[:5]) @ Vt[:5], atol=1e-12)
    assert np.allclose(s, sp[:5], rtol=1e-12)
    # symmetric split: A^T A = diag(s) = B G B^T
    assert np.allclose(A.T @ A, np.diag(s), atol=1e-10)
    assert np.allclose(B @ B.T, np.diag(s), atol=1e-10)


def test_weighted_fit_exact_on_low_rank_and_scale_invariant():
    """A residual of rank r is fitted exactly; scaling X by c scales the
    singular values by c and leaves A B unchanged."""
    rng = np.random.default_rng(7)
    rows, cols, n, r = 24, 16, 40, 3
    R = rng.standard_normal((rows, r)) @ rng.standard_normal((r, cols))
    X = rng.standard_normal((n, cols))
    A, B, s = S.weighted_factors_exact(R, X, r)
    assert np.linalg.norm(A @ B - R) <= 1e-10 * np.linalg.norm(R)
    A2, B2, s2 = S.weighted_factors_exact(R, 3.0 * X, r)
    assert np.allclose(s2, 3.0 * s, rtol=1e-10)
    assert np.allclose(A2 @ B2, A @ B, atol=1e-10 * np.abs(R).max())


@pytest.mark.parametrize("damp", [0.0, 2.0])
def test_weighted_randomized_route_matches_whitening(damp):
    """The operator route (randomized SVD of R X'^T, B = S^(-1/2) U^T R)
    reaches the whitened SVD's factors on a fast-decaying weighted spectrum;
    with damping the operator carries the extra sqrt(damp) I block."""
    rng = np.random.default_rng(8)
    rows, cols, n, r, p = 40, 30, 80, 6, 10
    R = _decaying(rng, rows, cols, 0.5)
    X = rng.standard_normal((n, cols))
    A0, B0, s0 = S.weighted_factors_exact(R, X, r, damp)
    om = rng.standard_normal((n + (cols if damp > 0 else 0), r + p))
    A1, B1, s1 = S.weighted_factors(R, X, om, r, q=2, damp=damp)
    assert np.allclose(s1, s0, rtol=1e-8)
    assert np.linalg.norm(A1 @ B1 - A0 @ B0) <= 1e-8 * np.linalg.norm(A0 @ B0)
    assert S.weighted_operator(R, X, damp).shape == (rows, om.shape[0])

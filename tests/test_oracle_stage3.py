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

"""Stage 3 on the GPU against the fp64 oracle: alignment cost, alignment of a
planted neuron permutation, and the randomized truncated SVD factors (same
caller-drawn test matrix on both sides, so both run the same algorithm;
compared through the basis-free products A B and the singular values)."""
import numpy as np
import pytest
import torch

from lxsynth import f32_to_bf16_bits
from oracle import stage3 as S
from oracle.moe import to_f64
from paper_2608_07814_amd import lorex as lx
from gpu_util import require_gpu, say

pytestmark = pytest.mark.gpu


def _bf(a):
    return f32_to_bf16_bits(np.asarray(a, np.float32))


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def _rel(a, b):
    return float(np.linalg.norm(np.asarray(a, np.float64) - b) / max(np.linalg.norm(b), 1e-300))


@pytest.mark.parametrize("f,d", [(96, 64), (768, 2048), (130, 70)])
def test_align_cost(f, d):
    require_gpu()
    say(f"align cost f={f} d={d}")
    rng = np.random.default_rng(f + d)
    dom = tuple(_bf(rng.standard_normal(s) / np.sqrt(d)) for s in ((f, d), (f, d), (d, f)))
    mem = tuple(_bf(rng.standard_normal(s) / np.sqrt(d)) for s in ((f, d), (f, d), (d, f)))
    got = lx.align_cost(tuple(map(_dev, dom)), tuple(map(_dev, mem))).cpu().numpy()
    ref = S.align_cost(dom, mem, "bf16")
    assert np.max(np.abs(got - ref)) <= 1e-12 * np.max(np.abs(ref))


def _member(rng, f, d, r, pi):
    """Dominant, and a member = (dominant + rank-r corrections) with its
    neurons reordered so that member neuron pi[i] is aligned neuron i."""
    s = np.sqrt(0.3 / np.sqrt(r * d))
    dg, du, dd = (rng.standard_normal(sh) / np.sqrt(d) for sh in ((f, d), (f, d), (d, f)))
    cg = (rng.standard_normal((f, r)) * s) @ (rng.standard_normal((r, d)) * s)
    cu = (rng.standard_normal((f, r)) * s) @ (rng.standard_normal((r, d)) * s)
    cd = (rng.standard_normal((d, r)) * s) @ (rng.standard_normal((r, f)) * s)
    inv = np.argsort(pi)
    dom = tuple(_bf(x) for x in (dg, du, dd))
    mem = (_bf((dg + cg)[inv]), _bf((du + cu)[inv]), _bf((dd + cd)[:, inv]))
    return dom, mem


@pytest.mark.parametrize("f,d,r,p", [(768, 2048, 64, 10), (200, 128, 16, 8)])
def test_align_and_factors_planted(f, d, r, p):
    """Neuron order recovered exactly; the factors of each aligned residual
    match the oracle's (same test matrix), and A^T A = B B^T = diag(sigma)."""
    require_gpu()
    say(f"stage 3 planted f={f} d={d} r={r} p={p}")
    rng = np.random.default_rng(7 + f)
    pi = rng.permutation(f)
    dom, mem = _member(rng, f, d, r, pi)
    ddom, dmem = tuple(map(_dev, dom)), tuple(map(_dev, mem))
    cost = lx.align_cost(ddom, dmem).cpu().numpy()
    perm, total = lx.assign(cost)
    ref_perm, ref_total = S.assign(S.align_cost(dom, mem, "bf16"))
    assert np.array_equal(perm, ref_perm) and np.array_equal(perm, pi)
    assert abs(total - ref_total) <= 1e-9 * abs(ref_total)
    permd = torch.from_numpy(perm).cuda()
    for proj, axis in ((0, 0), (1, 0), (2, 1)):
        rows, cols = dom[proj].shape
        om = rng.standard_normal((cols, r + p))
        A, B, sig = lx.lowrank_factors(ddom[proj], dmem[proj], r, torch.from_numpy(om).cuda(), q=2,
                                       perm=permd, perm_axis=axis)
        A, B, sig = A.cpu().numpy().astype(np.float64), B.cpu().numpy().astype(np.float64), sig.cpu().numpy()
        R = S.aligned_residual(dom[proj], mem[proj], perm, axis, "bf16")
        A0, B0, s0 = S.factors(R, om, r, q=2)
        e_ab, e_s = _rel(A @ B, A0 @ B0), float(np.max(np.abs(sig - s0) / s0))
        say(f"  projection {proj}: |AB - AB_oracle| / |AB_oracle| = {e_ab:.2e}, sigma rel {e_s:.2e}, "
            f"|R - AB| / |R| = {_rel(A @ B, R):.2e}")
        assert e_ab <= 1e-5 and e_s <= 1e-9
        assert np.allclose(A.T @ A, np.diag(sig), rtol=1e-5, atol=1e-6 * sig[0])
        assert np.allclose(B @ B.T, np.diag(sig), rtol=1e-5, atol=1e-6 * sig[0])


def test_factors_full_rank_residual_and_no_permutation():
    """A residual of full rank (low rank plus noise): still the oracle's
    randomized result; also fp32 weights and no permutation."""
    require_gpu()
    say("stage 3 full-rank residual")
    rng = np.random.default_rng(11)
    rows, cols, r, p = 300, 500, 32, 10
    wd = rng.standard_normal((rows, cols)).astype(np.float32)
    wm = (wd + (rng.standard_normal((rows, r)) @ rng.standard_normal((r, cols))) * 0.05
          + rng.standard_normal((rows, cols)) * 0.01).astype(np.float32)
    om = rng.standard_normal((cols, r + p))
    A, B, sig = lx.lowrank_factors(torch.from_numpy(wd).cuda(), torch.from_numpy(wm).cuda(), r,
                                   torch.from_numpy(om).cuda(), q=1)
    A, B, sig = A.cpu().numpy().astype(np.float64), B.cpu().numpy().astype(np.float64), sig.cpu().numpy()
    A0, B0, s0 = S.factors(wm.astype(np.float64) - wd, om, r, q=1)
    assert _rel(A @ B, A0 @ B0) <= 1e-5 and np.max(np.abs(sig - s0) / s0) <= 1e-9
    # q = 0 (a single sketch, no power iteration) and a member equal to its dominant
    A, B, sig = lx.lowrank_factors(torch.from_numpy(wd).cuda(), torch.from_numpy(wd).cuda(), r,
                                   torch.from_numpy(om).cuda(), q=0)
    assert float(sig.abs().max()) == 0.0 and float(A.abs().max()) == 0.0 and float(B.abs().max()) == 0.0

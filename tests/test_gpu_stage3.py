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


def _weighted_case(rng, rows, cols, n, r, noise=0.02):
    """A residual of rank r plus noise (dominant and member as bf16) and
    calibration activations with unequal column scales."""
    wd = rng.standard_normal((rows, cols)) / np.sqrt(cols)
    corr = (rng.standard_normal((rows, r)) @ rng.standard_normal((r, cols))) * (0.3 / np.sqrt(r * cols))
    wm = wd + corr + rng.standard_normal((rows, cols)) * (noise / np.sqrt(cols))
    x = rng.standard_normal((n, cols)) * np.exp(rng.standard_normal(cols) * 0.5)[None, :]
    return _bf(wd), _bf(wm), x.astype(np.float32)


@pytest.mark.parametrize("rows,cols,n,damp,xdt", [(768, 2048, 1024, 0.0, "bf16"), (768, 2048, 1024, 4.0, "f32"),
                                                  (200, 130, 300, 0.0, "f32")])
def test_weighted_factors_vs_oracle(rows, cols, n, damp, xdt):
    """Same caller-drawn test matrix on both sides: the GPU's factors equal
    the oracle's randomized route, and their emitted error is within 1% of
    the whitened SVD's optimum."""
    require_gpu()
    say(f"weighted fit rows={rows} cols={cols} n={n} damp={damp} x={xdt}")
    rng = np.random.default_rng(rows + n)
    r, p = 32, 10
    wd, wm, x = _weighted_case(rng, rows, cols, n, r)
    xb = _bf(x) if xdt == "bf16" else x
    xd = _dev(xb) if xdt == "bf16" else torch.from_numpy(x).cuda()
    xo = to_f64(xb, "bf16") if xdt == "bf16" else x.astype(np.float64)
    om = rng.standard_normal((n + (cols if damp > 0 else 0), r + p))
    # the small shape also aligns the member's columns by a permutation
    perm = rng.permutation(cols).astype(np.int32) if cols < 1000 else None
    A, B, sig = lx.weighted_factors(_dev(wd), _dev(wm), r, xd, torch.from_numpy(om).cuda(), q=2, damp=damp,
                                    perm=torch.from_numpy(perm).cuda() if perm is not None else None, perm_axis=1)
    A, B, sig = A.cpu().numpy().astype(np.float64), B.cpu().numpy().astype(np.float64), sig.cpu().numpy()
    R = (S.aligned_residual(wd, wm, perm, 1, "bf16") if perm is not None
         else to_f64(wm, "bf16") - to_f64(wd, "bf16"))
    A0, B0, s0 = S.weighted_factors(R, xo, om, r, q=2, damp=damp)
    e_ab, e_s = _rel(A @ B, A0 @ B0), float(np.max(np.abs(sig - s0) / s0))
    # the optimum: the Eckart-Young tail of the operator (R L when G is
    # positive definite; also defined for n < cols without damping)
    sv = np.linalg.svd(S.weighted_operator(R, xo, damp), compute_uv=False)
    opt = float(np.sqrt((sv[r:] ** 2).sum()))
    got = S.weighted_objective(R, xo, A, B, damp)
    U, sp, Vt = np.linalg.svd(R, full_matrices=False)
    plain = S.weighted_objective(R, xo, U[:, :r] * sp[:r], Vt[:r], damp)
    say(f"  |AB - AB_oracle| / |AB_oracle| = {e_ab:.2e}, sigma rel {e_s:.2e}; emitted error {got:.4e} "
        f"(optimum {opt:.4e}, plain SVD {plain:.4e})")
    assert e_ab <= 1e-5 and e_s <= 1e-9
    assert got <= 1.01 * opt


def test_weighted_factors_pure_damping_is_the_plain_fit():
    """No activations and damp > 0: G = damp I, so the weighted fit is the
    plain one with sigma scaled by sqrt(damp) and the same product A B
    (same test matrix for both entry points); also with a permutation."""
    require_gpu()
    say("weighted fit, damping only")
    rng = np.random.default_rng(17)
    rows, cols, r, p, damp = 300, 256, 24, 8, 2.25
    wd, wm, _ = _weighted_case(rng, rows, cols, 1, r)
    perm = torch.from_numpy(rng.permutation(rows).astype(np.int32)).cuda()
    om = torch.from_numpy(rng.standard_normal((cols, r + p))).cuda()
    x0 = torch.empty(0, cols, dtype=torch.float32, device="cuda")
    Aw, Bw, sw = lx.weighted_factors(_dev(wd), _dev(wm), r, x0, om, q=2, damp=damp, perm=perm, perm_axis=0)
    Ap, Bp, sp = lx.lowrank_factors(_dev(wd), _dev(wm), r, om, q=2, perm=perm, perm_axis=0)
    Aw, Bw, Ap, Bp = (t.cpu().numpy().astype(np.float64) for t in (Aw, Bw, Ap, Bp))
    assert np.allclose(sw.cpu().numpy(), np.sqrt(damp) * sp.cpu().numpy(), rtol=1e-10)
    assert _rel(Aw @ Bw, Ap @ Bp) <= 1e-5

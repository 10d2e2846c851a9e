"""Decode-sized batches on long-K products (split-K skinny GEMMs) and the
per-token cost example of Sec. 5 at its own shape, against the fp64 oracle.

The split-K path divides a product's weight slabs over several workgroups
when its output tiles are few; the last workgroup of each tile adds the
partial tiles in split order. Covered here: one token (every split of a tile
has one row), a few tokens, ragged splits, and repeated calls on one
workspace (the per-tile arrival counters must start from zero every call).
"""
import numpy as np
import pytest
import torch

from lxsynth import config, make_problem
from oracle import moe as O
from paper_2608_07814_amd import lorex as lx
from gpu_util import TOL_BF16, TOL_DESIGN, require_gpu, say, gpu_forward, err_ratio, dev_inputs

pytestmark = pytest.mark.gpu


def _oracle(p, tokens=None):
    return O.moe_forward(p.layer, p.x, p.routing.topk_ids, p.routing.topk_weights, tokens=tokens)


def _first(p, n):
    """The problem restricted to its first n tokens (same layer)."""
    from lxsynth import Problem, Routing
    r = p.routing
    return Problem(cfg=p.cfg, seed=p.seed, layer=p.layer, x=p.x[:n],
                   routing=Routing(r.topk_ids[:n].copy(), r.topk_weights[:n].copy()))


@pytest.mark.parametrize("f,T", [(4096, 1), (4096, 3), (1984, 5), (4096, 40)])
def test_split_k_long_down(f, T):
    """One cluster of 8, d = 256: the anchor down product has 4 column tiles
    and K = 2f, so it splits into many pieces (f = 1984: 31 weight slabs, the
    last split shorter than the others)."""
    require_gpu()
    say(f"split-K f={f} T={T}")
    p = make_problem(config(5, d=256, f=f, T=T), seed=31 + T)
    dl = lx.to_device(p.layer)
    ref = _oracle(p)
    xt, ids, w = dev_inputs(p)
    ws = lx.alloc_workspace(dl, T, 2, "flat")
    outs = []
    for _ in range(3):
        out = lx.forward(dl, xt, ids, w, workspace=ws, kind="flat")
        torch.cuda.synchronize()
        outs.append(out.cpu().numpy().astype(np.float64))
    e = err_ratio(outs[0], ref)
    say(f"  err/RMS = {e:.3e}")
    assert e <= TOL_BF16 and e <= TOL_DESIGN
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


def test_split_k_decode_levels():
    """128 experts in 16 clusters at T = 4: every level's products are split."""
    require_gpu()
    say("split-K cfg2 shape T=4")
    p = make_problem(2, T=4)
    e = err_ratio(gpu_forward(p), _oracle(p))
    say(f"  err/RMS = {e:.3e}")
    assert e <= TOL_DESIGN


@pytest.mark.timeout(400)
def test_paper_shape_cosel():
    """d = 4096, f = 14336, 8 experts in one cluster, top-2 among corrected
    members, rank 64 (the Mixtral-8x7B expert shape of the cost example):
    T = 16 against the oracle, and its first token and first 4 tokens alone."""
    require_gpu()
    say("paper shape: oracle for T=16")
    p = make_problem(5, T=16)
    ref = _oracle(p)
    dl = lx.to_device(p.layer)
    for n in (1, 4, 16):
        say(f"  T={n}")
        got = gpu_forward(_first(p, n), dev_layer=dl)
        e = err_ratio(got, ref[:n])
        say(f"  err/RMS = {e:.3e}")
        assert e <= TOL_BF16 and e <= TOL_DESIGN


@pytest.mark.parametrize("T", [1, 8, 64])
def test_tree_decode_sizes(T):
    """The BTExperts tree (d = 4096, f = 1024, 256 leaves) at decode sizes:
    every level on the skinny kernel, long-K products split."""
    require_gpu()
    say(f"tree decode T={T}")
    p = make_problem(4, T=T)
    got = gpu_forward(p)
    e = err_ratio(got, _oracle(p))
    say(f"  err/RMS = {e:.3e}")
    assert e <= TOL_BF16 and e <= TOL_DESIGN

"""Pins of the CPU oracle against brute force, library routines and invariants.

Each test names the plausible oracle mistake it would catch.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from lxsynth import make_problem, make_layer_flat, Layer, Level
from oracle import moe as O
from helpers import (rel_max_err, tiny_flat, tiny_tree, dense_layer, random_routing,
                     clone, zero_level)


def _x(T, d, seed):
    return np.random.default_rng(seed).standard_normal((T, d)).astype(np.float32)


# ---------------------------------------------------------------- brute force
@pytest.mark.parametrize("shuffle", [False, True])
def test_o1_equals_bruteforce_flat(shuffle):
    """Dense reconstruction vs scalar loops (catches any arithmetic slip in O1)."""
    layer = tiny_flat(shuffle=shuffle)
    x = _x(5, layer.d, 1)
    ids, w = random_routing(5, 3, layer.E, 2)
    ref = O.moe_forward_bruteforce(layer, x, ids, w)
    got = O.moe_forward(layer, x, ids, w)
    assert rel_max_err(got, ref) < 1e-12


def test_o1_equals_bruteforce_tree():
    """Tree path walk and nested corrections (catches a skipped level)."""
    layer = tiny_tree()
    x = _x(4, layer.d, 3)
    ids, w = random_routing(4, 3, layer.E, 4)
    ref = O.moe_forward_bruteforce(layer, x, ids, w)
    assert rel_max_err(O.moe_forward(layer, x, ids, w), ref) < 1e-12


def test_o1_equals_bruteforce_dropped_and_duplicate_ids():
    layer = tiny_flat(E=4, C=2)
    x = _x(6, layer.d, 5)
    ids, w = random_routing(6, 3, layer.E, 6, allow_dupes=True, drop_frac=0.25)
    ref = O.moe_forward_bruteforce(layer, x, ids, w)
    assert rel_max_err(O.moe_forward(layer, x, ids, w), ref) < 1e-12


def test_cfg0_bruteforce():
    """The tiny fp32 configuration end to end, against scalar loops."""
    p = make_problem(0)
    ref = O.moe_forward_bruteforce(p.layer, p.x, p.routing.topk_ids, p.routing.topk_weights)
    got = O.moe_forward(p.layer, p.x, p.routing.topk_ids, p.routing.topk_weights)
    assert rel_max_err(got, ref) < 1e-12


# ----------------------------------------------------- amortized formulation
@pytest.mark.parametrize("case", ["cfg0", "tree", "shuffled", "dupes"])
def test_amortized_equals_per_expert(case):
    """Sec. 5.1: sharing anchor/ancestor terms and applying the anchor's down
    projection to the weighted activation sum leaves the output unchanged."""
    if case == "cfg0":
        p = make_problem(0)
        layer, x, ids, w = p.layer, p.x, p.routing.topk_ids, p.routing.topk_weights
    elif case == "tree":
        layer = tiny_tree(E=16, n_roots=2, subs=2, d=16, f=8)
        x = _x(9, layer.d, 7)
        ids, w = random_routing(9, 5, layer.E, 8)
    elif case == "shuffled":
        layer = tiny_flat(E=12, C=3, shuffle=True)
        x = _x(9, layer.d, 9)
        ids, w = random_routing(9, 4, layer.E, 10)
    else:
        layer = tiny_flat(E=6, C=2)
        x = _x(9, layer.d, 11)
        ids, w = random_routing(9, 4, layer.E, 12, allow_dupes=True, drop_frac=0.2)
    a = O.moe_forward(layer, x, ids, w)
    b = O.moe_forward_amortized(layer, x, ids, w)
    assert rel_max_err(b, a) < 1e-12


# ------------------------------------------------------ textbook SwiGLU FFN
def _torch_moe(x, ids, w, experts):
    """Dense top-k SwiGLU MoE with torch library routines (fp64, CPU)."""
    xt = torch.from_numpy(np.asarray(x, dtype=np.float64))
    out = torch.zeros(xt.shape[0], experts[0][2].shape[0], dtype=torch.float64)
    for t in range(xt.shape[0]):
        for j in range(ids.shape[1]):
            e = int(ids[t, j])
            if e < 0:
                continue
            wg, wu, wd = (torch.from_numpy(np.asarray(m, dtype=np.float64)) for m in experts[e])
            h = F.silu(F.linear(xt[t], wg)) * F.linear(xt[t], wu)
            out[t] += float(w[t, j]) * F.linear(h, wd)
    return out.numpy()


def test_zero_corrections_reproduce_dominant_only_model():
    """With every factor removed each expert is its cluster's dominant
    (catches swapped gate/up, a wrong silu, a transposed down projection)."""
    layer = zero_level(tiny_flat(E=8, C=2, d=16, f=24, r=4, seed=21), 0)
    x = _x(7, layer.d, 22)
    ids, w = random_routing(7, 3, layer.E, 23)
    cl = layer.levels[0].parent
    experts = {e: (layer.anchor_gate[cl[e]], layer.anchor_up[cl[e]], layer.anchor_down[cl[e]])
               for e in range(layer.E)}
    ref = _torch_moe(x, ids, w, experts)
    assert rel_max_err(O.moe_forward(layer, x, ids, w), ref) < 1e-12


def test_single_expert_is_textbook_swiglu():
    layer = tiny_flat(E=1, C=1, d=16, f=24, r=4, seed=31)
    x = _x(5, layer.d, 32)
    ids = np.zeros((5, 1), np.int32)
    w = np.ones((5, 1), np.float32)
    xt = torch.from_numpy(x.astype(np.float64))
    g = F.linear(xt, torch.from_numpy(layer.anchor_gate[0].astype(np.float64)))
    u = F.linear(xt, torch.from_numpy(layer.anchor_up[0].astype(np.float64)))
    ref = F.linear(F.silu(g) * u, torch.from_numpy(layer.anchor_down[0].astype(np.float64)))
    assert rel_max_err(O.moe_forward(layer, x, ids, w), ref.numpy()) < 1e-12


def test_full_rank_correction_reproduces_arbitrary_expert():
    """Gate/up: A = W_target - W_dom, B = I; down: A = I, B = W_target - W_dom.
    With r = d the member becomes an arbitrary dense expert exactly
    (catches a dropped or sign-flipped correction and a wrong factor index)."""
    d, f, E, C = 64, 128, 8, 2
    rng = np.random.default_rng(41)
    base = make_layer_flat(E, C, d, f, 8, "f32", 41)
    cl, fo = base.levels[0].parent, base.levels[0].factor_of
    M = int((fo >= 0).sum())
    dg = (rng.standard_normal((M, f, d)) / np.sqrt(d)).astype(np.float32)
    du = (rng.standard_normal((M, f, d)) / np.sqrt(d)).astype(np.float32)
    dd = (rng.standard_normal((M, d, f)) / np.sqrt(d)).astype(np.float32)
    eye = np.broadcast_to(np.eye(d, dtype=np.float32), (M, d, d)).copy()
    lv = Level(parent=cl, factor_of=fo, rank=d, a_gate=dg, b_gate=eye, a_up=du, b_up=eye,
               a_down=eye, b_down=dd)
    layer = Layer(E=E, d=d, f=f, dtype="f32", anchor_gate=base.anchor_gate,
                  anchor_up=base.anchor_up, anchor_down=base.anchor_down, levels=[lv])
    experts = {}
    for e in range(E):
        c, m = cl[e], fo[e]
        g64 = base.anchor_gate[c].astype(np.float64)
        u64 = base.anchor_up[c].astype(np.float64)
        d64 = base.anchor_down[c].astype(np.float64)
        if m >= 0:   # sum of two fp32 values is exact in fp64
            g64, u64, d64 = g64 + dg[m], u64 + du[m], d64 + dd[m]
        experts[e] = (g64, u64, d64)
    x = _x(10, d, 42)
    ids, w = random_routing(10, 3, E, 43)
    ref = _torch_moe(x, ids, w, experts)
    assert rel_max_err(O.moe_forward(layer, x, ids, w), ref) < 1e-12
    assert rel_max_err(O.moe_forward_amortized(layer, x, ids, w), ref) < 1e-12


# ------------------------------------------------------------- invariants
def test_neuron_permutation_symmetry():
    """Permuting a cluster's intermediate neurons jointly (gate/up rows, down
    columns, members' A_gate/A_up rows and B_down columns) is function
    preserving (Sec. 1 neuron permutation symmetry; Sec. 3 Stage 3 (i))."""
    layer = tiny_flat(E=8, C=2, d=16, f=24, r=4, seed=51)
    x = _x(8, layer.d, 52)
    ids, w = random_routing(8, 3, layer.E, 53)
    ref = O.moe_forward(layer, x, ids, w)
    perm = np.random.default_rng(54).permutation(layer.f)
    p = clone(layer)
    c = 1
    p.anchor_gate[c] = p.anchor_gate[c][perm]
    p.anchor_up[c] = p.anchor_up[c][perm]
    p.anchor_down[c] = p.anchor_down[c][:, perm]
    lv = p.levels[0]
    for e in range(layer.E):
        m = lv.factor_of[e]
        if lv.parent[e] == c and m >= 0:
            lv.a_gate[m] = lv.a_gate[m][perm]
            lv.a_up[m] = lv.a_up[m][perm]
            lv.b_down[m] = lv.b_down[m][:, perm]
    assert rel_max_err(O.moe_forward(p, x, ids, w), ref) < 1e-12
    # permuting only the anchor (not its members' factors) must change the result
    q = clone(layer)
    q.anchor_gate[c] = q.anchor_gate[c][perm]
    assert rel_max_err(O.moe_forward(q, x, ids, w), ref) > 1e-3


def test_expert_relabeling():
    layer = tiny_flat(E=8, C=2, seed=61)
    x = _x(6, layer.d, 62)
    ids, w = random_routing(6, 3, layer.E, 63)
    ref = O.moe_forward(layer, x, ids, w)
    pi = np.random.default_rng(64).permutation(layer.E)
    p = clone(layer)
    lv = p.levels[0]
    new_parent = np.empty_like(lv.parent)
    new_fo = np.empty_like(lv.factor_of)
    new_parent[pi] = layer.levels[0].parent
    new_fo[pi] = layer.levels[0].factor_of
    lv.parent, lv.factor_of = new_parent, new_fo
    assert rel_max_err(O.moe_forward(p, x, pi[ids].astype(np.int32), w), ref) < 1e-12


def test_linear_in_routing_weights_and_dropped_slots():
    layer = tiny_flat(E=8, C=2, seed=71)
    x = _x(6, layer.d, 72)
    ids, w1 = random_routing(6, 3, layer.E, 73)
    _, w2 = random_routing(6, 3, layer.E, 74)
    o1 = O.moe_forward(layer, x, ids, w1)
    o2 = O.moe_forward(layer, x, ids, w2)
    o12 = O.moe_forward(layer, x, ids, (w1.astype(np.float64) + w2))
    assert rel_max_err(o12, o1 + o2) < 1e-12
    assert rel_max_err(O.moe_forward(layer, x, ids, 3.0 * w1.astype(np.float64)), 3 * o1) < 1e-12
    # a dropped slot (-1) equals a zero weight
    ids_d = ids.copy()
    ids_d[2, 1] = -1
    wz = w1.copy()
    wz[2, 1] = 0
    assert rel_max_err(O.moe_forward(layer, x, ids_d, w1), O.moe_forward(layer, x, ids, wz)) < 1e-12
    # every slot dropped: zero output
    assert np.all(O.moe_forward(layer, x, np.full_like(ids, -1), w1) == 0)


def test_bad_ids_flagged_and_dropped():
    layer = tiny_flat(E=8, C=2, seed=81)
    x = _x(5, layer.d, 82)
    ids, w = random_routing(5, 3, layer.E, 83)
    bad = ids.copy()
    bad[1, 0] = layer.E
    bad[3, 2] = -5
    out, flag = O.moe_forward(layer, x, bad, w, return_flag=True)
    assert flag == O.FLAG_BAD_ID
    wz = w.copy()
    wz[1, 0] = 0
    wz[3, 2] = 0
    assert rel_max_err(out, O.moe_forward(layer, x, ids, wz)) < 1e-12
    _, flag0 = O.moe_forward(layer, x, ids, w, return_flag=True)
    assert flag0 == 0


def test_token_subset_matches_full():
    p = make_problem(0)
    full = O.moe_forward(p.layer, p.x, p.routing.topk_ids, p.routing.topk_weights)
    sub = O.moe_forward(p.layer, p.x, p.routing.topk_ids, p.routing.topk_weights,
                        tokens=[3, 0, 11])
    # same arithmetic; BLAS may block a smaller batch differently
    assert rel_max_err(sub, full[[3, 0, 11]]) < 1e-13


# ------------------------------------------------------------------ tree
def test_tree_zero_sub_level_is_flat_over_roots():
    """Removing the sub-dominant corrections leaves a flat layer whose anchors
    are the roots and whose members are the leaves with their own factors."""
    tree = tiny_tree(E=16, n_roots=2, subs=2, d=16, f=8, seed=91)
    t0 = zero_level(tree, 0)
    lv1, lv2 = tree.levels
    flat_lv = Level(parent=lv1.parent[lv2.parent], factor_of=lv2.factor_of, rank=lv2.rank,
                    a_gate=lv2.a_gate, b_gate=lv2.b_gate, a_up=lv2.a_up, b_up=lv2.b_up,
                    a_down=lv2.a_down, b_down=lv2.b_down)
    flat = Layer(E=tree.E, d=tree.d, f=tree.f, dtype="f32", anchor_gate=tree.anchor_gate,
                 anchor_up=tree.anchor_up, anchor_down=tree.anchor_down, levels=[flat_lv])
    x = _x(7, tree.d, 92)
    ids, w = random_routing(7, 4, tree.E, 93)
    assert rel_max_err(O.moe_forward(t0, x, ids, w), O.moe_forward(flat, x, ids, w)) < 1e-12


def test_tree_zero_leaf_level_is_flat_over_subdominants():
    """Removing the leaf corrections makes every leaf equal to its sub-dominant
    (root + sub correction): a dense MoE over those weights."""
    tree = tiny_tree(E=16, n_roots=2, subs=2, d=16, f=8, seed=95)
    t1 = zero_level(tree, 1)
    lv1, lv2 = tree.levels
    experts = {}
    for e in range(tree.E):
        s = lv2.parent[e]
        rt = lv1.parent[s]
        m = lv1.factor_of[s]
        experts[e] = (tree.anchor_gate[rt].astype(np.float64) + lv1.a_gate[m].astype(np.float64) @ lv1.b_gate[m],
                      tree.anchor_up[rt].astype(np.float64) + lv1.a_up[m].astype(np.float64) @ lv1.b_up[m],
                      tree.anchor_down[rt].astype(np.float64) + lv1.a_down[m].astype(np.float64) @ lv1.b_down[m])
    x = _x(6, tree.d, 96)
    ids, w = random_routing(6, 4, tree.E, 97)
    assert rel_max_err(O.moe_forward(t1, x, ids, w), _torch_moe(x, ids, w, experts)) < 1e-12


def test_dense_layer_is_plain_moe():
    """L = 0 (anchors are the experts): the dense comparator's definition."""
    rng = np.random.default_rng(101)
    E, d, f = 5, 8, 12
    wg = rng.standard_normal((E, f, d)).astype(np.float32)
    wu = rng.standard_normal((E, f, d)).astype(np.float32)
    wd = rng.standard_normal((E, d, f)).astype(np.float32)
    layer = dense_layer(wg, wu, wd)
    x = _x(6, d, 102)
    ids, w = random_routing(6, 2, E, 103)
    ref = _torch_moe(x, ids, w, {e: (wg[e], wu[e], wd[e]) for e in range(E)})
    assert rel_max_err(O.moe_forward(layer, x, ids, w), ref) < 1e-12
    assert rel_max_err(O.moe_forward_bruteforce(layer, x, ids, w), ref) < 1e-12

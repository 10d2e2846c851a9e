"""Pins of the bucketing oracle, the seeded router and the FLOP/byte accounting."""
import json
import math
import os

import numpy as np
import pytest

from lxsynth import make_problem, config, route_gaussian, make_x, f32_to_bf16_bits
from oracle import bucket as B
from paper_2608_07814_amd import accounting as A
from helpers import random_routing, tiny_tree, tiny_flat


def _structure(layer):
    parents = [lv.parent for lv in layer.levels]
    n_nodes = [layer.n_anchors] + [lv.n_nodes for lv in layer.levels]
    return parents, n_nodes


def _eq(a, b):
    for la, lb in zip(a, b):
        for key in ("row_token", "offsets", "slot_row"):
            assert np.array_equal(la[key], lb[key]), key


@pytest.mark.parametrize("kind", ["flat", "flat_shuffled", "tree", "dense"])
@pytest.mark.parametrize("seed", [0, 1])
def test_bucket_definition_equals_bruteforce(kind, seed):
    if kind == "flat":
        layer = tiny_flat(E=12, C=3)
    elif kind == "flat_shuffled":
        layer = tiny_flat(E=12, C=4, shuffle=True)
    elif kind == "tree":
        layer = tiny_tree(E=16, n_roots=2, subs=2)
    else:
        layer = tiny_flat(E=5, C=5)
        layer.levels = []
    parents, n_nodes = _structure(layer)
    ids, _ = random_routing(23, 4, layer.E, 200 + seed, allow_dupes=True, drop_frac=0.15,
                            bad_frac=0.05)
    a, fa = B.bucket(parents, n_nodes, layer.E, ids)
    b, fb = B.bucket_bruteforce(parents, n_nodes, layer.E, ids)
    assert fa == fb == B.FLAG_BAD_ID
    _eq(a, b)


@pytest.mark.parametrize("T,k,hot", [(1, 2, False), (7, 3, False), (64, 8, False), (300, 8, True),
                                      (1000, 4, False)])
def test_tile_count_bound(T, k, hot):
    """The workspace's tile tables hold floor(R / bm) + min(N, R) entries per
    level (R = T * min(k, N) rows at most): the tiles the bucketing makes,
    sum over nodes of ceil(rows / bm), never exceed that."""
    layer = tiny_tree(E=32, n_roots=2, subs=4)
    parents, n_nodes = _structure(layer)
    ids, _ = random_routing(T, k, layer.E, 500 + T, allow_dupes=True, drop_frac=0.1)
    if hot:
        ids[:, :2] = [3, 4]
    lv, _ = B.bucket(parents, n_nodes, layer.E, ids)
    for li, arrs in enumerate(lv):
        cnt = np.diff(arrs["offsets"])
        R = T * min(k, n_nodes[li])
        assert cnt.sum() <= R
        for bm in (32, 128, 256):
            tiles = int(np.sum((cnt + bm - 1) // bm))
            assert tiles <= R // bm + min(n_nodes[li], R)


def test_bucket_invariants_cfg1_shape():
    p = make_problem(1, T=512)
    parents, n_nodes = _structure(p.layer)
    ids = p.routing.topk_ids
    lv, flag = B.bucket(parents, n_nodes, p.layer.E, ids)
    assert flag == 0
    T, k = ids.shape
    for li, arrs in enumerate(lv):
        off, rt, sr = arrs["offsets"], arrs["row_token"], arrs["slot_row"]
        assert off[0] == 0 and off[-1] == rt.size and np.all(np.diff(off) >= 0)
        for n in range(n_nodes[li]):
            seg = rt[off[n]:off[n + 1]]
            assert np.all(np.diff(seg) > 0)     # unique, ascending tokens per node
        tok = np.repeat(np.arange(T), k)
        assert np.all(sr >= 0)                   # Gaussian routing drops nothing
        assert np.array_equal(rt[sr], tok)       # each slot's row is its token's row
        # every row is referenced by at least one slot
        assert np.array_equal(np.unique(sr), np.arange(rt.size))
    # experts level: distinct ids per token, so every slot is its own row
    assert lv[-1]["row_token"].size == T * k
    # anchors level: row count = unique (token, cluster) pairs
    cl = p.layer.levels[0].parent[ids]
    assert lv[0]["row_token"].size == sum(len(set(r)) for r in cl.tolist())


def test_bucket_empty_and_all_dropped():
    layer = tiny_flat(E=6, C=2)
    parents, n_nodes = _structure(layer)
    for ids in (np.zeros((0, 3), np.int32), np.full((4, 3), -1, np.int32)):
        lv, flag = B.bucket(parents, n_nodes, layer.E, ids)
        assert flag == 0
        for li, arrs in enumerate(lv):
            assert arrs["row_token"].size == 0
            assert np.all(arrs["offsets"] == 0) and arrs["offsets"].size == n_nodes[li] + 1
            assert np.all(arrs["slot_row"] == -1)


def test_bucket_single_hot_expert():
    """Every token routed to the same expert: one node per level has all rows."""
    layer = tiny_flat(E=6, C=2)
    parents, n_nodes = _structure(layer)
    ids = np.full((9, 2), 4, np.int32)
    ids[:, 1] = -1
    lv, _ = B.bucket(parents, n_nodes, layer.E, ids)
    assert np.array_equal(lv[1]["offsets"], [0, 0, 0, 0, 0, 9, 9])
    assert np.array_equal(lv[0]["offsets"], [0, 0, 9])
    assert np.array_equal(lv[1]["row_token"], np.arange(9))


# ------------------------------------------------------------------ router
@pytest.mark.parametrize("cfg", [0, 1, 4])
def test_router_topk_and_weights(cfg):
    c = config(cfg, T=64)
    x = make_x(c["T"], c["d"], c["dtype"], 7)
    r = route_gaussian(x, c["dtype"], c["E"], c["k"], 7)
    ids, w = r.topk_ids, r.topk_weights
    assert ids.shape == (64, c["k"]) and w.dtype == np.float32
    assert np.all(np.abs(w.astype(np.float64).sum(1) - 1) < 1e-6)
    assert np.all(w > 0) and np.all(np.diff(w, axis=1) <= 0)
    for row in ids:
        assert len(set(row.tolist())) == c["k"]
    # brute-force top-k of the same logits
    rng = np.random.default_rng(np.random.SeedSequence(7).spawn(8)[1])
    w_r = rng.standard_normal((c["d"], c["E"])) / math.sqrt(c["d"])
    xv = (x.astype(np.uint32) << 16).view(np.float32) if c["dtype"] == "bf16" else x
    logits = xv.astype(np.float64) @ w_r
    for t in range(8):
        lst = sorted(range(c["E"]), key=lambda e: (-logits[t, e], e))[:c["k"]]
        assert ids[t].tolist() == lst
        ex = np.exp(logits[t, lst] - logits[t, lst].max())
        assert np.allclose(w[t], ex / ex.sum(), rtol=1e-6)


def test_community_routing_structure():
    p = make_problem(3, T=2000)
    ids = p.routing.topk_ids
    cl = p.layer.levels[0].parent
    assert all(len(set(r)) == 8 for r in ids.tolist())
    # most slots share the token's most common cluster (p_home = 0.7 plus chance)
    home_share = np.mean([np.bincount(cl[r], minlength=32).max() / 8 for r in ids])
    assert 0.45 < home_share < 0.75
    assert np.all(np.abs(p.routing.topk_weights.sum(1) - 1) < 1e-6)


def test_coselect_routing_structure():
    """Configuration 5's routing, at a small layer: both experts of a token are
    distinct corrected members of one cluster, uniformly spread over them."""
    p = make_problem(config(5, d=64, f=128, r=8, T=3000))
    ids = p.routing.topk_ids
    fo = p.layer.levels[0].factor_of
    assert ids.shape == (3000, 2)
    assert np.all(ids[:, 0] != ids[:, 1])
    assert np.all(fo[ids] >= 0)                       # never the dominant (expert 0)
    counts = np.bincount(ids.ravel(), minlength=8)
    assert counts[0] == 0 and np.all(np.abs(counts[1:] / 6000 - 1 / 7) < 0.02)
    assert np.all(np.abs(p.routing.topk_weights.sum(1) - 1) < 1e-6)
    # two clusters of 4: a token never mixes them
    q = make_problem(config(5, E=8, C=2, d=64, f=128, r=8, T=500))
    cl = q.layer.levels[0].parent
    assert np.all(cl[q.routing.topk_ids[:, 0]] == cl[q.routing.topk_ids[:, 1]])
    assert np.all(q.layer.levels[0].factor_of[q.routing.topk_ids] >= 0)


def test_bf16_rounding_is_rne():
    vals = np.array([1.0, 1.0 + 2**-8, 1.0 + 3 * 2**-9, -2.5, 3.0e-3], dtype=np.float32)
    bits = f32_to_bf16_bits(vals)
    back = (bits.astype(np.uint32) << 16).view(np.float32)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7 -> even mantissa (1.0)
    assert back[0] == 1.0 and back[1] == 1.0 and back[2] == np.float32(1 + 2**-7)
    assert back[3] == -2.5
    # half an ulp of bf16 in [2^-9, 2^-8): 2^-8 * 2^-9
    assert abs(float(back[4]) - float(vals[4])) <= 2.0**-17


def test_weight_scale_rule():
    """||A B||_F is about 0.3 ||W_dom||_F for every projection."""
    layer = tiny_flat(E=4, C=1, d=256, f=128, r=16, seed=3)
    lv = layer.levels[0]
    ratios = []
    for m in range(lv.n_factors):
        for a, b, w in ((lv.a_gate, lv.b_gate, layer.anchor_gate), (lv.a_down, lv.b_down, layer.anchor_down)):
            ratios.append(np.linalg.norm(a[m].astype(np.float64) @ b[m]) / np.linalg.norm(w[0]))
    assert 0.25 < np.mean(ratios) < 0.35


# -------------------------------------------------------------- accounting
def test_accounting_matches_paper_fig_flops(root):
    g = json.load(open(os.path.join(root, "tests", "golden", "paper_fig_flops.json")))
    s, pr = g["shape"], g["printed"]
    c = A.per_token_projection_cost(s["k"], s["I"], s["H"], s["r"], s["bytes_per_elem"])
    assert round(c["dense_matrix_bytes"] / 1e6) == pr["dense_matrix_MB"]
    assert round(c["factor_pair_bytes"] / 1e6, 1) == pr["factor_pair_MB"]
    assert round(c["original_flops"] / 1e6) == pr["original_MFLOPs"]
    assert round(c["original_bytes"] / 1e6) == pr["original_MB"]
    assert round(c["amortized_flops"] / 1e6) == pr["amortized_MFLOPs"]
    assert round(c["amortized_bytes"] / 1e6) == pr["amortized_MB"]
    sp = A.closed_form_speedup(s["k"], s["I"], s["H"], s["r"])
    assert round(sp, 1) == pr["speedup_approx"]
    assert abs(sp - c["original_flops"] / c["amortized_flops"]) < 1e-12
    # batch-1 arithmetic intensity of one bf16 projection: 2 FLOP per 2-byte weight
    assert round(c["original_flops"] / c["original_bytes"]) == pr["arithmetic_intensity_flop_per_byte_approx"]


def test_algorithmic_counts_from_buckets():
    p = make_problem(1, T=256)
    parents, n_nodes = _structure(p.layer)
    lv, _ = B.bucket(parents, n_nodes, p.layer.E, p.routing.topk_ids)
    rows = A.level_rows_from_buckets([l["offsets"] for l in lv],
                                     [None, p.layer.levels[0].factor_of], [0, 64])
    c = A.algorithmic_counts(2048, 768, rows, 256, 8)
    U = rows[0].rows
    S_nd = int((p.layer.levels[0].factor_of[p.routing.topk_ids] >= 0).sum())
    assert rows[1].rows == S_nd
    assert c["flops"] == 6 * 2048 * 768 * U + 6 * 64 * (2048 + 768) * S_nd
    assert c["gate_up_flops"] == 4 * 2048 * 768 * U


# ------------------------------------------------------------ router oracle
def _router_bruteforce(x64, w64, k):
    """Scalar loops: logits, selection by repeated maximum (lower index wins a
    tie), weights exp(l_j) / sum over chosen exp(l_i)."""
    T, d = x64.shape
    E = w64.shape[0]
    ids = np.zeros((T, k), np.int64)
    ws = np.zeros((T, k))
    for t in range(T):
        lg = [math.fsum(float(x64[t, i]) * float(w64[e, i]) for i in range(d)) for e in range(E)]
        left = list(range(E))
        for j in range(k):
            best = left[0]
            for e in left[1:]:
                if lg[e] > lg[best]:
                    best = e
            ids[t, j] = best
            left.remove(best)
        m = lg[ids[t, 0]]
        ex = [math.exp(lg[e] - m) for e in ids[t]]
        s = math.fsum(ex)
        ws[t] = [v / s for v in ex]
    return ids, ws


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_router_oracle_bruteforce(dtype):
    from oracle import router as R
    from lxsynth import make_router
    from oracle.moe import to_f64
    x = make_x(9, 24, dtype, 41)
    w = make_router(24, 11, dtype, 41)
    for k in (1, 3, 11):
        ids, ws, lg = R.route_topk(x, w, dtype, k)
        bi, bw = _router_bruteforce(to_f64(x, dtype), to_f64(w, dtype), k)
        assert np.array_equal(ids, bi)
        assert np.max(np.abs(ws - bw)) < 1e-14
        assert np.all(np.abs(ws.sum(1) - 1) < 1e-14)
        assert np.all(np.diff(np.take_along_axis(lg, ids.astype(np.int64), 1), axis=1) <= 0)
    # k = E: every expert once; the weights are the full softmax
    ids, ws, lg = R.route_topk(x, w, dtype, 11)
    assert np.array_equal(np.sort(ids, 1), np.tile(np.arange(11), (9, 1)))
    full = np.exp(lg - lg.max(1, keepdims=True))
    full /= full.sum(1, keepdims=True)
    assert np.max(np.abs(np.take_along_axis(full, ids.astype(np.int64), 1) - ws)) < 1e-14


def test_router_oracle_ties_and_matrix():
    """Identical router rows tie exactly: the lower expert index comes first.
    The generated router matrix is the harness router's draw (same stream)."""
    from oracle import router as R
    from lxsynth import make_router
    w = make_router(32, 6, "f32", 5)
    w[4] = w[1]                      # experts 1 and 4 always tie
    x = make_x(50, 32, "f32", 6)
    ids, ws, lg = R.route_topk(x, w, "f32", 6)
    pos = np.argsort(ids, axis=1)
    assert np.all(pos[:, 1] < pos[:, 4])
    both = ids[:, :2]
    sel = np.all(np.isin(both, [1, 4]), axis=1)
    assert np.allclose(ws[sel, 0], ws[sel, 1])
    # same draw as the Gaussian harness router: its fp64 top-k agrees with the
    # oracle on the fp32-stored matrix except at near-ties
    p = make_problem(config(1, d=64, f=64, E=16, C=4, k=4, T=400))
    wr = make_router(64, 16, "bf16", p.seed)
    lg2 = R.router_logits(p.x, wr, "bf16")
    ids2, _, _ = R.route_topk(p.x, wr, "bf16", 4)
    gap = np.sort(lg2, 1)[:, ::-1]
    # bf16 rounding of the matrix moves a logit by ~2^-9 of its scale (~0.002)
    clear = np.min(np.abs(np.diff(gap[:, :5], axis=1)), axis=1) > 0.01
    assert clear.mean() > 0.7
    assert np.array_equal(ids2[clear], p.routing.topk_ids[clear])


def test_fp32_sum_bound_covers_fp32_sums():
    from oracle import router as R
    from lxsynth import make_router
    from oracle.moe import to_f64
    x = make_x(20, 2048, "bf16", 7)
    w = make_router(2048, 8, "bf16", 7)
    exact = R.router_logits(x, w, "bf16")
    b = R.fp32_sum_bound(x, w, "bf16")
    xs, ws = to_f64(x, "bf16").astype(np.float32), to_f64(w, "bf16").astype(np.float32)
    for order in (np.arange(2048), np.random.default_rng(0).permutation(2048)):
        acc = np.zeros((20, 8), np.float32)
        for i in order:               # sequential fp32 accumulation
            acc += xs[:, i:i + 1] * ws[:, i][None, :]
        assert np.all(np.abs(acc.astype(np.float64) - exact) <= b)

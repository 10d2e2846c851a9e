"""Seeded generators: configurations, layer weights, activations and routing.

Distributions (one recipe for every configuration):

* dense anchors (cluster dominants, tree roots), gate/up/down: N(0, 1/d);
* low-rank factors: every entry of A and of B is N(0, s) with
  s^2 = 0.3 / sqrt(r * d), so that E||A B||_F^2 = 0.09 * E||W_anchor||_F^2,
  i.e. the correction carries about 0.3 of the anchor's Frobenius norm;
* activations x: N(0, 1);
* Gaussian routing: logits = x @ W_r with W_r ~ N(0, 1/d) in fp64, top-k over
  all experts (ties to the lower index, order: descending logit then index),
  weights = softmax over the chosen logits, stored fp32;
* community routing: a home cluster per token, each slot stays home with
  probability p, weights = softmax of k iid N(0, 1) logits.

Draws are fp32 (numpy PCG64, one child stream of ``SeedSequence(seed)`` per
tensor family) and are rounded to bf16 with round-to-nearest-even when the
layer is bf16. Both sides of every parity check consume the stored values.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

# Child streams of SeedSequence(seed), fixed so a change in one tensor family
# (e.g. the token count) leaves every other family's values unchanged.
_S_X, _S_ROUTER, _S_ROUTE_EXTRA, _S_ANCHOR, _S_LEVEL1, _S_SHUFFLE = 0, 1, 2, 3, 4, 7
_N_STREAMS = 8

CONFIGS = {
    0: dict(name="tiny-fp32", kind="flat", dtype="f32", E=8, C=2, k=2, d=64, f=128,
            r=8, T=16, routing="gaussian"),
    1: dict(name="prefill-d2048-f768-E128-C16-r64-T4096", kind="flat", dtype="bf16",
            E=128, C=16, k=8, d=2048, f=768, r=64, T=4096, routing="gaussian"),
    2: dict(name="decode-d2048-f768-E128-C16-r64-T64", kind="flat", dtype="bf16",
            E=128, C=16, k=8, d=2048, f=768, r=64, T=64, routing="gaussian"),
    3: dict(name="prefill-community-d2048-f768-E128-C32-r96-T16384", kind="flat",
            dtype="bf16", E=128, C=32, k=8, d=2048, f=768, r=96, T=16384,
            routing="community", p_home=0.7),
    4: dict(name="tree-d4096-f1024-E256-roots4-subs32-r128-r64-T8192", kind="tree",
            dtype="bf16", E=256, d=4096, f=1024, k=8, T=8192, n_roots=4,
            subs_per_root=8, r_sub=128, r_leaf=64, routing="gaussian"),
    # the per-token cost example of Sec. 5 (Fig. flops): Mixtral-8x7B expert
    # shape, all 8 experts in one cluster, each token's two experts co-selected
    # among the corrected members (both pay a rank-64 correction)
    5: dict(name="cosel-d4096-f14336-E8-C1-r64-k2-T1", kind="flat", dtype="bf16",
            E=8, C=1, k=2, d=4096, f=14336, r=64, T=1, routing="coselect"),
}


def config(index: int, **overrides) -> dict:
    """Copy of configuration ``index`` with ``overrides`` applied."""
    c = dict(CONFIGS[index])
    c.update(overrides)
    c["index"] = index
    return c


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); return uint16 bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    rounded = u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def _children(seed: int):
    return np.random.SeedSequence(seed).spawn(_N_STREAMS)


def _store(vals: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return f32_to_bf16_bits(vals)
    if dtype == "f32":
        return np.ascontiguousarray(vals, dtype=np.float32)
    raise ValueError(dtype)


def _normal(rng: np.random.Generator, shape, std: float, dtype: str) -> np.ndarray:
    v = rng.standard_normal(shape, dtype=np.float32)
    v *= np.float32(std)
    return _store(v, dtype)


@dataclass
class Level:
    """One correction level: nodes, their parents one level up, and factors."""
    parent: np.ndarray      # int32 [N]
    factor_of: np.ndarray   # int32 [N], -1 = node equals its parent (no factor)
    rank: int
    a_gate: np.ndarray      # [M, f, r]
    b_gate: np.ndarray      # [M, r, d]
    a_up: np.ndarray        # [M, f, r]
    b_up: np.ndarray        # [M, r, d]
    a_down: np.ndarray      # [M, d, r]
    b_down: np.ndarray      # [M, r, f]

    @property
    def n_nodes(self) -> int:
        return int(self.parent.shape[0])

    @property
    def n_factors(self) -> int:
        return int(self.a_gate.shape[0])


@dataclass
class Layer:
    E: int
    d: int
    f: int
    dtype: str                       # "bf16" (uint16 bits) or "f32"
    anchor_gate: np.ndarray          # [N0, f, d]
    anchor_up: np.ndarray            # [N0, f, d]
    anchor_down: np.ndarray          # [N0, d, f]
    levels: list = field(default_factory=list)

    @property
    def n_anchors(self) -> int:
        return int(self.anchor_gate.shape[0])

    @property
    def n_levels(self) -> int:
        return len(self.levels)

    def weight_bytes(self) -> int:
        n = self.anchor_gate.nbytes + self.anchor_up.nbytes + self.anchor_down.nbytes
        for lv in self.levels:
            n += sum(a.nbytes for a in (lv.a_gate, lv.b_gate, lv.a_up, lv.b_up,
                                        lv.a_down, lv.b_down))
        return n


@dataclass
class Routing:
    topk_ids: np.ndarray       # int32 [T, k]
    topk_weights: np.ndarray   # fp32 [T, k]


@dataclass
class Problem:
    cfg: dict
    seed: int
    layer: Layer
    x: np.ndarray              # [T, d] storage dtype
    routing: Routing

    @property
    def T(self) -> int:
        return int(self.x.shape[0])

    @property
    def k(self) -> int:
        return int(self.routing.topk_ids.shape[1])


def _factor_std(r: int, d: int, rel: float) -> float:
    # E||AB||^2 = out*in*r*s^4 and E||W||^2 = out*in/d  =>  s^2 = rel/sqrt(r*d)
    return math.sqrt(rel / math.sqrt(r * d))


def _make_factors(rng, M, d, f, r, dtype, rel=0.3):
    s = _factor_std(r, d, rel)
    return dict(
        a_gate=_normal(rng, (M, f, r), s, dtype),
        b_gate=_normal(rng, (M, r, d), s, dtype),
        a_up=_normal(rng, (M, f, r), s, dtype),
        b_up=_normal(rng, (M, r, d), s, dtype),
        a_down=_normal(rng, (M, d, r), s, dtype),
        b_down=_normal(rng, (M, r, f), s, dtype),
    )


def _make_anchors(rng, n, d, f, dtype):
    std = 1.0 / math.sqrt(d)
    return dict(
        anchor_gate=_normal(rng, (n, f, d), std, dtype),
        anchor_up=_normal(rng, (n, f, d), std, dtype),
        anchor_down=_normal(rng, (n, d, f), std, dtype),
    )


def make_layer_flat(E: int, C: int, d: int, f: int, r: int, dtype: str, seed: int,
                    shuffle: bool = False, rel: float = 0.3) -> Layer:
    """Flat LorExperts layer: C clusters of E/C experts, first member dominant.

    Cluster c holds experts [c*m, (c+1)*m) (m = E/C) unless ``shuffle``, in which
    case a seeded permutation assigns experts to clusters. The dominant is the
    lowest-indexed member and has no factor; the other members get factor
    indices 0..M-1 in ascending expert order.
    """
    if E % C:
        raise ValueError("E must be a multiple of C")
    ch = _children(seed)
    m = E // C
    cluster_of = np.repeat(np.arange(C, dtype=np.int32), m)
    if shuffle:
        perm = np.random.default_rng(ch[_S_SHUFFLE]).permutation(E)
        cluster_of = cluster_of[perm].astype(np.int32)
    factor_of = np.full(E, -1, dtype=np.int32)
    seen = set()
    nxt = 0
    for e in range(E):
        c = int(cluster_of[e])
        if c in seen:
            factor_of[e] = nxt
            nxt += 1
        else:
            seen.add(c)
    anchors = _make_anchors(np.random.default_rng(ch[_S_ANCHOR]), C, d, f, dtype)
    fac = _make_factors(np.random.default_rng(ch[_S_LEVEL1]), nxt, d, f, r, dtype, rel)
    lv = Level(parent=cluster_of, factor_of=factor_of, rank=r, **fac)
    return Layer(E=E, d=d, f=f, dtype=dtype, levels=[lv], **anchors)


def make_layer_tree(E: int, d: int, f: int, n_roots: int, subs_per_root: int,
                    r_sub: int, r_leaf: int, dtype: str, seed: int,
                    rel: float = 0.3) -> Layer:
    """Depth-2 BTExperts layer: roots, sub-dominants (root + rank r_sub), leaves.

    Sub-dominant n has parent n // subs_per_root; leaf (expert) e has parent
    e // (E / n_subs). Every sub-dominant and every leaf carries a correction,
    each drawn with the same relative scale against the root.
    """
    n_subs = n_roots * subs_per_root
    if E % n_subs:
        raise ValueError("E must be a multiple of the number of sub-dominants")
    ch = _children(seed)
    anchors = _make_anchors(np.random.default_rng(ch[_S_ANCHOR]), n_roots, d, f, dtype)
    sub_parent = (np.arange(n_subs) // subs_per_root).astype(np.int32)
    leaf_parent = (np.arange(E) // (E // n_subs)).astype(np.int32)
    f1 = _make_factors(np.random.default_rng(ch[_S_LEVEL1]), n_subs, d, f, r_sub, dtype, rel)
    f2 = _make_factors(np.random.default_rng(ch[_S_LEVEL1 + 1]), E, d, f, r_leaf, dtype, rel)
    lv1 = Level(parent=sub_parent, factor_of=np.arange(n_subs, dtype=np.int32),
                rank=r_sub, **f1)
    lv2 = Level(parent=leaf_parent, factor_of=np.arange(E, dtype=np.int32),
                rank=r_leaf, **f2)
    return Layer(E=E, d=d, f=f, dtype=dtype, levels=[lv1, lv2], **anchors)


def make_x(T: int, d: int, dtype: str, seed: int) -> np.ndarray:
    rng = np.random.default_rng(_children(seed)[_S_X])
    return _normal(rng, (T, d), 1.0, dtype)


def _decode_for_router(x: np.ndarray, dtype: str) -> np.ndarray:
    # The router sees the stored activations exactly (bf16 -> fp64 is exact).
    if dtype == "bf16":
        return (x.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


def _softmax_rows(logits: np.ndarray) -> np.ndarray:
    m = logits.max(axis=1, keepdims=True)
    e = np.exp(logits - m)
    return e / e.sum(axis=1, keepdims=True)


def make_router(d: int, E: int, dtype: str, seed: int) -> np.ndarray:
    """Router weights [E, d] in the storage dtype: the same N(0, 1/d) draw that
    ``route_gaussian`` uses (child stream of ``seed``), transposed to the
    nn.Linear layout and stored (bf16: round to nearest even from fp32)."""
    rng = np.random.default_rng(_children(seed)[_S_ROUTER])
    w_r = rng.standard_normal((d, E)) / math.sqrt(d)
    return _store(np.ascontiguousarray(w_r.T).astype(np.float32), dtype)


def route_gaussian(x: np.ndarray, dtype: str, E: int, k: int, seed: int) -> Routing:
    """Unchanged top-k router on x @ W_r (fp64), softmax over the chosen logits."""
    T, d = x.shape
    rng = np.random.default_rng(_children(seed)[_S_ROUTER])
    w_r = rng.standard_normal((d, E)) / math.sqrt(d)
    logits = _decode_for_router(x, dtype) @ w_r
    order = np.argsort(-logits, axis=1, kind="stable")[:, :k]
    chosen = np.take_along_axis(logits, order, axis=1)
    w = _softmax_rows(chosen)
    return Routing(topk_ids=order.astype(np.int32), topk_weights=w.astype(np.float32))


def route_community(T: int, members: list, k: int, p_home: float, seed: int) -> Routing:
    """Community-structured routing over clusters ``members`` (lists of experts).

    Per token a home cluster is drawn uniformly. Slots j = 0..k-1 are drawn in
    order without replacement: with probability p_home (and while the home
    cluster still has an unchosen member) uniformly among the home cluster's
    unchosen members, otherwise uniformly among all unchosen experts. Weights
    are the softmax of k iid N(0, 1) logits, in slot order.
    """
    rng = np.random.default_rng(_children(seed)[_S_ROUTE_EXTRA])
    C = len(members)
    E = sum(len(m) for m in members)
    homes = rng.integers(0, C, size=T)
    u_stay = rng.random((T, k))
    u_pick = rng.random((T, k))
    logits = rng.standard_normal((T, k))
    ids = np.empty((T, k), dtype=np.int32)
    for t in range(T):
        chosen = []
        home = members[int(homes[t])]
        for j in range(k):
            avail_home = [e for e in home if e not in chosen]
            if avail_home and u_stay[t, j] < p_home:
                pool = avail_home
            else:
                pool = [e for e in range(E) if e not in chosen]
            e = pool[min(int(u_pick[t, j] * len(pool)), len(pool) - 1)]
            chosen.append(e)
            ids[t, j] = e
    w = _softmax_rows(logits)
    return Routing(topk_ids=ids, topk_weights=w.astype(np.float32))


def route_coselect(T: int, corrected: list, k: int, seed: int) -> Routing:
    """Every token's k experts come from one cluster and all carry a correction.

    ``corrected[c]`` lists cluster c's members that carry a correction (all
    but the dominant). Per token a cluster is drawn uniformly among those with
    at least k such members; its k experts are drawn uniformly without
    replacement among them, in draw order. Weights are the softmax of k iid
    N(0, 1) logits, in slot order.
    """
    rng = np.random.default_rng(_children(seed)[_S_ROUTE_EXTRA])
    pools = [m for m in corrected if len(m) >= k]
    if not pools:
        raise ValueError("no cluster has k corrected members")
    which = rng.integers(0, len(pools), size=T)
    ids = np.empty((T, k), dtype=np.int32)
    for t in range(T):
        pool = pools[int(which[t])]
        ids[t] = np.asarray(pool)[rng.permutation(len(pool))[:k]]
    w = _softmax_rows(rng.standard_normal((T, k)))
    return Routing(topk_ids=ids, topk_weights=w.astype(np.float32))


def _cluster_members(layer: Layer) -> list:
    lv = layer.levels[-1]
    members = [[] for _ in range(layer.n_anchors)]
    for e in range(layer.E):
        members[int(lv.parent[e])].append(e)
    return members


def make_problem(cfg, seed: Optional[int] = None, T: Optional[int] = None,
                 shuffle: bool = False) -> Problem:
    """Build layer, activations and routing for a configuration.

    ``cfg`` is a configuration index or dict; ``seed`` defaults to the index;
    ``T`` overrides the token count (the layer is unchanged by ``T``).
    """
    if isinstance(cfg, int):
        cfg = config(cfg)
    cfg = dict(cfg)
    if T is not None:
        cfg["T"] = T
    if seed is None:
        seed = int(cfg.get("index", 0))
    dtype = cfg["dtype"]
    if cfg["kind"] == "flat":
        layer = make_layer_flat(cfg["E"], cfg["C"], cfg["d"], cfg["f"], cfg["r"], dtype,
                                seed, shuffle=shuffle)
    elif cfg["kind"] == "tree":
        layer = make_layer_tree(cfg["E"], cfg["d"], cfg["f"], cfg["n_roots"],
                                cfg["subs_per_root"], cfg["r_sub"], cfg["r_leaf"], dtype, seed)
    else:
        raise ValueError(cfg["kind"])
    x = make_x(cfg["T"], cfg["d"], dtype, seed)
    if cfg["routing"] == "gaussian":
        routing = route_gaussian(x, dtype, cfg["E"], cfg["k"], seed)
    elif cfg["routing"] == "community":
        routing = route_community(cfg["T"], _cluster_members(layer), cfg["k"],
                                  cfg["p_home"], seed)
    elif cfg["routing"] == "coselect":
        fo = layer.levels[-1].factor_of
        corrected = [[e for e in m if fo[e] >= 0] for m in _cluster_members(layer)]
        routing = route_coselect(cfg["T"], corrected, cfg["k"], seed)
    else:
        raise ValueError(cfg["routing"])
    return Problem(cfg=cfg, seed=seed, layer=layer, x=x, routing=routing)

"""fp64 reference forward of one compressed MoE layer (test infrastructure).

Definitions followed, stated in this library's notation (output-side factor A,
input-side factor B, weights in [out][in] layout):

* Sec. 3 "Representation" (unnumbered equation): a cluster member's weights are
  its dominant's plus a rank-r product, per projection:
  W_m = W_dom + A_m B_m.
* Sec. 3 Stage 3 (iii) "Installation": at inference the member computes with
  W_dom + A_m B_m; the router is left unchanged.
* Sec. 5 / Fig. tree: in a BTExperts tree an expert is a leaf and its weights
  are the root anchor plus the corrections of every node on path(e).
* The expert FFN is SwiGLU without biases: y = W_d (silu(W_g x) * (W_u x)),
  silu(z) = z / (1 + exp(-z)); top-k routing combines y with the router weights.
* Sec. 5.1 "Amortized forward pass": terms shared by co-selected experts (the
  anchor product and shared ancestor corrections) may be computed once per
  token; by linearity the anchor's down projection may be applied once to the
  weighted sum of the members' activations. The result is unchanged.

Routing conventions: a slot whose id is -1 is dropped (contributes 0); an id
below -1 or not below E is invalid, contributes 0 and raises the returned flag.
Duplicate ids in a row are independent slots.

Stored inputs (bf16 bit patterns or fp32) are promoted to fp64 exactly; no
rounding of the stored values is counted as error.
"""
from __future__ import annotations

import math

import numpy as np

FLAG_BAD_ID = 1


def to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact fp64 value of stored bf16 bits (uint16) or fp32 values."""
    if dtype == "bf16":
        return (np.asarray(a).astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    if dtype == "f32":
        return np.asarray(a, dtype=np.float64)
    raise ValueError(dtype)


def silu(z):
    return z / (1.0 + np.exp(-z))


def expert_path(layer, e: int):
    """Anchor index of expert e and the (level, node) pairs of path(e), leaf first."""
    nodes = []
    n = int(e)
    for li in range(layer.n_levels - 1, -1, -1):
        nodes.append((li, n))
        n = int(layer.levels[li].parent[n])
    return n, nodes


def expert_weights(layer, e: int):
    """Dense fp64 (W_gate [f,d], W_up [f,d], W_down [d,f]) of expert e.

    Anchor of the expert's tree plus, for every node on its path that carries
    a factor, the product A B of that node's factors (Sec. 3 "Representation";
    Sec. 5 path sharing).
    """
    dt = layer.dtype
    anchor, nodes = expert_path(layer, e)
    wg = to_f64(layer.anchor_gate[anchor], dt)
    wu = to_f64(layer.anchor_up[anchor], dt)
    wd = to_f64(layer.anchor_down[anchor], dt)
    for li, n in nodes:
        lv = layer.levels[li]
        m = int(lv.factor_of[n])
        if m < 0:
            continue
        wg = wg + to_f64(lv.a_gate[m], dt) @ to_f64(lv.b_gate[m], dt)
        wu = wu + to_f64(lv.a_up[m], dt) @ to_f64(lv.b_up[m], dt)
        wd = wd + to_f64(lv.a_down[m], dt) @ to_f64(lv.b_down[m], dt)
    return wg, wu, wd


def _valid(ids: np.ndarray, E: int):
    ok = (ids >= 0) & (ids < E)
    bad = bool(np.any((ids < -1) | (ids >= E)))
    return ok, bad


def moe_forward(layer, x, topk_ids, topk_weights, tokens=None, return_flag=False):
    """Binding oracle: out[t] = sum_j w[t,j] * SwiGLU_{e_tj}(x_t), fp64.

    Expert-major execution: each routed expert is reconstructed densely once
    (``expert_weights``), its FFN is applied to the tokens routed to it, and the
    per-slot outputs are then summed over j in ascending order.
    ``tokens`` restricts the computation to a subset of token indices (the
    result has one row per listed token).
    """
    x64 = to_f64(x, layer.dtype)
    ids = np.asarray(topk_ids)
    w = np.asarray(topk_weights, dtype=np.float64)
    if tokens is not None:
        tokens = np.asarray(tokens)
        x64, ids, w = x64[tokens], ids[tokens], w[tokens]
    T, k = ids.shape
    ok, bad = _valid(ids, layer.E)
    y = np.zeros((T, k, layer.d))
    for e in np.unique(ids[ok]):
        wg, wu, wd = expert_weights(layer, int(e))
        tt, jj = np.nonzero(ids == e)
        xe = x64[tt]
        h = silu(xe @ wg.T) * (xe @ wu.T)
        y[tt, jj] = h @ wd.T
    out = np.zeros((T, layer.d))
    for j in range(k):
        out += np.where(ok[:, j:j + 1], w[:, j:j + 1], 0.0) * y[:, j]
    return (out, FLAG_BAD_ID if bad else 0) if return_flag else out


def moe_forward_amortized(layer, x, topk_ids, topk_weights):
    """Amortized formulation (Sec. 5.1), fp64, one token at a time.

    For each token, the anchor products (W_gate x, W_up x) and each path node's
    input-side factor products (B x) are computed once and reused by every
    selected expert below them; the SwiGLU activations are weighted and summed
    per anchor and per factor-carrying node; the anchor's down projection and
    each node's A_down B_down are then applied once to those sums.
    No expert is ever reconstructed.
    """
    dt = layer.dtype
    x64 = to_f64(x, dt)
    ids = np.asarray(topk_ids)
    w = np.asarray(topk_weights, dtype=np.float64)
    T, k = ids.shape
    ok, _ = _valid(ids, layer.E)
    out = np.zeros((T, layer.d))
    for t in range(T):
        xt = x64[t]
        anchor_gu = {}
        node_gu = {}
        hsum = {}
        for j in range(k):
            if not ok[t, j]:
                continue
            anchor, nodes = expert_path(layer, int(ids[t, j]))
            if anchor not in anchor_gu:
                anchor_gu[anchor] = (to_f64(layer.anchor_gate[anchor], dt) @ xt,
                                     to_f64(layer.anchor_up[anchor], dt) @ xt)
            g, u = (v.copy() for v in anchor_gu[anchor])
            carriers = []
            for li, n in nodes:
                lv = layer.levels[li]
                m = int(lv.factor_of[n])
                if m < 0:
                    continue
                if (li, n) not in node_gu:
                    zg = to_f64(lv.b_gate[m], dt) @ xt
                    zu = to_f64(lv.b_up[m], dt) @ xt
                    node_gu[(li, n)] = (to_f64(lv.a_gate[m], dt) @ zg,
                                        to_f64(lv.a_up[m], dt) @ zu)
                dg, du = node_gu[(li, n)]
                g += dg
                u += du
                carriers.append((li, n, m))
            wh = w[t, j] * silu(g) * u
            key = ("anchor", anchor)
            hsum[key] = hsum.get(key, 0.0) + wh
            for li, n, m in carriers:
                key = (li, n, m)
                hsum[key] = hsum.get(key, 0.0) + wh
        acc = np.zeros(layer.d)
        for key, hs in hsum.items():
            if key[0] == "anchor":
                acc += to_f64(layer.anchor_down[key[1]], dt) @ hs
            else:
                li, _, m = key
                lv = layer.levels[li]
                acc += to_f64(lv.a_down[m], dt) @ (to_f64(lv.b_down[m], dt) @ hs)
        out[t] = acc
    return out


def moe_forward_bruteforce(layer, x, topk_ids, topk_weights):
    """Scalar Python loops (tiny shapes only): reconstruct, then per slot."""
    dt = layer.dtype
    E, d, f = layer.E, layer.d, layer.f
    x64 = to_f64(x, dt).tolist()
    ids = np.asarray(topk_ids).tolist()
    w = np.asarray(topk_weights, dtype=np.float64).tolist()
    T, k = len(ids), len(ids[0])

    def mat(a):
        return to_f64(a, dt).tolist()

    experts = {}
    for e in range(E):
        # walk the parent maps from the leaf up (independent of expert_path)
        nodes = []
        n = e
        li = layer.n_levels - 1
        while li >= 0:
            nodes.append((li, n))
            n = int(layer.levels[li].parent[n])
            li -= 1
        anchor = n
        wg = mat(layer.anchor_gate[anchor])
        wu = mat(layer.anchor_up[anchor])
        wd = mat(layer.anchor_down[anchor])
        for li, n in nodes:
            lv = layer.levels[li]
            m = int(lv.factor_of[n])
            if m < 0:
                continue
            r = lv.rank
            ag, bg = mat(lv.a_gate[m]), mat(lv.b_gate[m])
            au, bu = mat(lv.a_up[m]), mat(lv.b_up[m])
            ad, bd = mat(lv.a_down[m]), mat(lv.b_down[m])
            for i in range(f):
                for c in range(d):
                    wg[i][c] += sum(ag[i][q] * bg[q][c] for q in range(r))
                    wu[i][c] += sum(au[i][q] * bu[q][c] for q in range(r))
            for i in range(d):
                for c in range(f):
                    wd[i][c] += sum(ad[i][q] * bd[q][c] for q in range(r))
        experts[e] = (wg, wu, wd)

    out = [[0.0] * d for _ in range(T)]
    for t in range(T):
        for j in range(k):
            e = ids[t][j]
            if e < 0 or e >= E:
                continue
            wg, wu, wd = experts[e]
            h = []
            for i in range(f):
                g = sum(wg[i][c] * x64[t][c] for c in range(d))
                u = sum(wu[i][c] * x64[t][c] for c in range(d))
                h.append(g / (1.0 + math.exp(-g)) * u)
            for c in range(d):
                out[t][c] += w[t][j] * sum(wd[c][i] * h[i] for i in range(f))
    return np.array(out)

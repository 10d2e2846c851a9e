"""Routing-bucketing arrays from their definition (test infrastructure).

The amortized forward (Sec. 5.1) computes a shared term once per token for
each anchor or tree node the token's selected experts sit under. Bucketing
lists, for every tree level l = 0..L (0 = anchors, L = experts), the unique
(token, node) pairs that need that level's work:

* ``row_token[l]``: tokens of the unique pairs, sorted by (node, token);
* ``offsets[l]``  : int32 [N_l + 1], rows of node n are
                    ``offsets[n] .. offsets[n+1]-1`` (exclusive prefix sum);
* ``slot_row[l]`` : int32 [T*k], for slot s = t*k + j the row of the pair
                    (t, node_l(e_s)), or -1 if the slot is dropped or invalid.

node_l(e) is the level-l ancestor of expert e (node_L(e) = e). A slot is valid
when 0 <= id < E; ids below -1 or not below E are invalid and raise the flag.
These arrays are the bit-exact contract for the GPU bucketing.
"""
from __future__ import annotations

import numpy as np

FLAG_BAD_ID = 1


def ancestors(parents: list, E: int) -> list:
    """anc[l][e] for l = 0..L; ``parents[l-1]`` maps level-l nodes to level l-1."""
    L = len(parents)
    anc = [None] * (L + 1)
    anc[L] = np.arange(E, dtype=np.int64)
    for li in range(L - 1, -1, -1):
        anc[li] = np.asarray(parents[li], dtype=np.int64)[anc[li + 1]]
    return anc


def bucket(parents: list, n_nodes: list, E: int, topk_ids: np.ndarray):
    """Sort + unique definition. ``n_nodes[l]`` = number of nodes at level l."""
    ids = np.asarray(topk_ids, dtype=np.int64)
    T, k = ids.shape
    flat = ids.reshape(-1)
    valid = (flat >= 0) & (flat < E)
    flag = FLAG_BAD_ID if np.any((flat < -1) | (flat >= E)) else 0
    tok = np.repeat(np.arange(T, dtype=np.int64), k)
    anc = ancestors(parents, E)
    out = []
    for li in range(len(parents) + 1):
        N = int(n_nodes[li])
        node = np.where(valid, anc[li][np.where(valid, flat, 0)], -1)
        keys = node[valid] * T + tok[valid]
        uniq = np.unique(keys)
        row_token = (uniq % T).astype(np.int32)
        counts = np.bincount(uniq // T, minlength=N)
        offsets = np.zeros(N + 1, dtype=np.int32)
        offsets[1:] = np.cumsum(counts)
        slot_row = np.full(T * k, -1, dtype=np.int32)
        slot_row[valid] = np.searchsorted(uniq, keys).astype(np.int32)
        out.append(dict(row_token=row_token, offsets=offsets, slot_row=slot_row))
    return out, flag


def bucket_bruteforce(parents: list, n_nodes: list, E: int, topk_ids: np.ndarray):
    """Same arrays by explicit loops: per node, scan tokens in ascending order."""
    ids = np.asarray(topk_ids).tolist()
    T, k = len(ids), len(ids[0]) if ids else 0
    L = len(parents)
    flag = 0

    def node_at(e, li):
        n = e
        for lv in range(L - 1, li - 1, -1):
            n = int(parents[lv][n])
        return n

    out = []
    for li in range(L + 1):
        N = int(n_nodes[li])
        row_token, offsets = [], [0]
        slot_row = [-1] * (T * k)
        for n in range(N):
            for t in range(T):
                hit = False
                for j in range(k):
                    e = ids[t][j]
                    if e < -1 or e >= E:
                        flag = FLAG_BAD_ID
                    if 0 <= e < E and node_at(e, li) == n:
                        if not hit:
                            row_token.append(t)
                            hit = True
                        slot_row[t * k + j] = len(row_token) - 1
            offsets.append(len(row_token))
        out.append(dict(row_token=np.array(row_token, dtype=np.int32),
                        offsets=np.array(offsets, dtype=np.int32),
                        slot_row=np.array(slot_row, dtype=np.int32)))
    return out, flag

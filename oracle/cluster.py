"""fp64 reference of the clustering stages (test infrastructure).

THIS MODULE IS TEST INFRASTRUCTURE, like the rest of the package: only the
test suite, the smoke check and the benchmark's CPU-baseline leg use it.

What it follows (Sec. 3 "Compression pipeline"):

* Stage 1, router profiling: per-expert firing counts N_e over a calibration
  set (here: the routing ids of N tokens; an expert fires on a token when it is
  among that token's valid ids, counted once per token).
* Coact-NPMI distance (Sec. 3 "Variants"): D = 1 - NPMI of expert
  co-activation, diagonal zeroed. Readings (the paper prints no formula):
  p_i = N_i / N, p_ij = N_ij / N with N_ij the tokens on which both fire;
  NPMI = log(p_ij / (p_i p_j)) / (-log p_ij); pairs that never co-fire get
  NPMI = -1 (the limit), pairs that co-fire on every token (p_ij = 1) get 1.
* Stage 2, frequency-seeded k-medoids: the medoids start at the highest-firing
  experts; assign / update until no medoid changes. Readings: seeds in
  descending firing count (ties: lower index) and cluster c is the one seeded
  by the c-th of them; an expert joins the nearest medoid (ties: lower cluster
  index) and a medoid always stays in its own cluster; a cluster's new medoid
  is the member with the smallest sum of distances to the cluster's members,
  summed in ascending member order (ties: lower index); at most max_iter
  update rounds. Protected experts are pulled out first as singleton clusters,
  numbered after the seeded ones in ascending expert order.
* Dominant: the highest-firing member; ties by co-activation centrality, read
  as the sum of (1 - D) to the other members in ascending member order
  (larger first); then the lower index. Every other member gets a factor
  index, 0, 1, ... in ascending expert order (the layout of a flat layer).
"""
from __future__ import annotations

import numpy as np


def coact_counts(ids, E: int):
    """(N_e int64 [E], N_ij int64 [E, E] symmetric, zero diagonal)."""
    ids = np.asarray(ids)
    fire = np.zeros(E, np.int64)
    pair = np.zeros((E, E), np.int64)
    for row in ids:
        s = sorted({int(e) for e in row if 0 <= e < E})
        for a in s:
            fire[a] += 1
        for i in range(len(s)):
            for j in range(i + 1, len(s)):
                pair[s[i], s[j]] += 1
                pair[s[j], s[i]] += 1
    return fire, pair


def npmi_distance(fire, pair, N: int) -> np.ndarray:
    """D = 1 - NPMI [E, E] fp64, zero diagonal (readings above)."""
    fire = np.asarray(fire, np.float64)
    pair = np.asarray(pair, np.float64)
    E = fire.shape[0]
    D = np.zeros((E, E))
    for i in range(E):
        for j in range(E):
            if i == j:
                continue
            if pair[i, j] == 0:
                npmi = -1.0
            elif pair[i, j] == N:
                npmi = 1.0
            else:
                pij = pair[i, j] / N
                npmi = np.log(pij / ((fire[i] / N) * (fire[j] / N))) / (-np.log(pij))
            D[i, j] = 1.0 - npmi
    return D


def kmedoids(D, fire, C: int, protected=(), max_iter: int = 100):
    """(cluster_of int32 [E], factor_of int32 [E], dominant int32 [C], iterations)."""
    D = np.asarray(D, np.float64)
    fire = np.asarray(fire, np.int64)
    E = D.shape[0]
    prot = sorted(set(int(p) for p in protected))
    P = len(prot)
    K = C - P
    if K < 1 or K > E - P:
        raise ValueError("need 1 <= C - |protected| <= E - |protected|")
    free = [e for e in range(E) if e not in prot]
    # seeds: descending firing count, ties to the lower index
    order = sorted(free, key=lambda e: (-fire[e], e))
    med = order[:K]
    cluster_of = np.full(E, -1, np.int64)

    def assign():
        for e in free:
            if e in med:
                cluster_of[e] = med.index(e)
                continue
            best, bd = 0, D[e, med[0]]
            for c in range(1, K):
                if D[e, med[c]] < bd:
                    best, bd = c, D[e, med[c]]
            cluster_of[e] = best

    it = 0
    assign()
    while it < max_iter:
        it += 1
        new = list(med)
        for c in range(K):
            members = [e for e in free if cluster_of[e] == c]
            best, bs = None, None
            for m in members:
                s = 0.0
                for j in members:       # ascending member order
                    s += D[m, j]
                if bs is None or s < bs:
                    best, bs = m, s
            new[c] = best
        if new == med:
            break
        med = new
        assign()
    for i, p in enumerate(prot):
        cluster_of[p] = K + i
    dominant = np.zeros(C, np.int64)
    for c in range(C):
        members = [e for e in range(E) if cluster_of[e] == c]

        def key(e):
            cent = 0.0
            for j in members:
                if j != e:
                    cent += 1.0 - D[e, j]
            return (-fire[e], -cent, e)
        dominant[c] = min(members, key=key)
    factor_of = np.full(E, -1, np.int64)
    nxt = 0
    for e in range(E):
        if dominant[cluster_of[e]] != e:
            factor_of[e] = nxt
            nxt += 1
    return cluster_of.astype(np.int32), factor_of.astype(np.int32), dominant.astype(np.int32), it

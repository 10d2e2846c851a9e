"""Pins of the clustering oracle (firing / co-activation counts, NPMI
distance, frequency-seeded k-medoids, dominant choice)."""
import math

import numpy as np
import pytest

from oracle import cluster as K
from helpers import random_routing


def test_counts_match_one_hot_products():
    ids, _ = random_routing(300, 6, 20, 3, allow_dupes=True, drop_frac=0.1, bad_frac=0.02)
    fire, pair = K.coact_counts(ids, 20)
    X = np.zeros((300, 20), np.int64)
    for t, row in enumerate(ids):
        for e in row:
            if 0 <= e < 20:
                X[t, e] = 1           # fires once per token, duplicates or not
    G = X.T @ X
    assert np.array_equal(fire, np.diag(G))
    np.fill_diagonal(G, 0)
    assert np.array_equal(pair, G)


def test_npmi_closed_forms():
    N = 100
    fire = np.array([50, 20, 30, 30, 40])
    pair = np.zeros((5, 5), np.int64)
    pair[0, 1] = pair[1, 0] = 10          # p01 = 0.1 = 0.5 * 0.2: independent -> NPMI 0
    pair[2, 3] = pair[3, 2] = 30          # always together -> NPMI 1
    pair[0, 2] = pair[2, 0] = 15          # 0.15 vs 0.5 * 0.3 = 0.15: independent
    pair[0, 4] = pair[4, 0] = 5           # below independence: negative NPMI
    D = K.npmi_distance(fire, pair, N)
    assert D[0, 1] == pytest.approx(1.0, abs=1e-15)
    assert D[2, 3] == pytest.approx(0.0, abs=1e-15)
    assert D[0, 2] == pytest.approx(1.0, abs=1e-15)
    assert D[1, 4] == 2.0                 # never co-fire: NPMI -1
    npmi04 = math.log(0.05 / (0.5 * 0.4)) / -math.log(0.05)
    assert D[0, 4] == pytest.approx(1 - npmi04, rel=1e-14) and D[0, 4] > 1
    assert np.array_equal(D, D.T) and np.all(np.diag(D) == 0)
    # a pair firing on every token
    D2 = K.npmi_distance(np.array([10, 10]), np.array([[0, 10], [10, 0]]), 10)
    assert D2[0, 1] == 0.0


def _planted(E=24, G=4, seed=0):
    rng = np.random.default_rng(seed)
    grp = np.repeat(np.arange(G), E // G)
    rng.shuffle(grp)
    D = np.where(grp[:, None] == grp[None, :], rng.uniform(0.1, 0.3, (E, E)),
                 rng.uniform(1.5, 1.9, (E, E)))
    D = (D + D.T) / 2
    np.fill_diagonal(D, 0)
    fire = rng.integers(10, 1000, E)
    return D, fire, grp


def test_kmedoids_recovers_planted_groups_from_frequency_seeds():
    D, fire, grp = _planted()
    # make every group's most-fired expert one of the four seeds
    for g in range(4):
        fire[np.where(grp == g)[0][0]] = 5000 + g
    cl, fo, dom, it = K.kmedoids(D, fire, 4)
    for g in range(4):
        assert len(set(cl[grp == g].tolist())) == 1
    assert len(set(cl.tolist())) == 4
    # cluster c is seeded by the c-th most fired expert
    seeds = np.argsort(-fire, kind="stable")[:4]
    assert np.array_equal(cl[seeds], np.arange(4))
    # the dominant is the most-fired member, and the only factor-less one
    for c in range(4):
        m = np.where(cl == c)[0]
        assert dom[c] == m[np.argmax(fire[m])]
        assert fo[dom[c]] == -1
    assert np.array_equal(np.sort(fo[fo >= 0]), np.arange(24 - 4))
    assert np.all(np.diff(fo[fo >= 0]) > 0)       # ascending expert order


def test_kmedoids_fixed_point_and_single_cluster():
    rng = np.random.default_rng(5)
    X = rng.standard_normal((30, 3))
    D = np.sqrt(((X[:, None] - X[None]) ** 2).sum(-1))
    fire = rng.integers(0, 50, 30)
    cl, _, dom, it = K.kmedoids(D, fire, 5)
    assert it < 100
    # fixed point: every cluster's medoid minimises its in-cluster distance sum,
    # and every non-medoid is nearest (ties: lower cluster) to its own medoid
    med = []
    for c in range(5):
        m = np.where(cl == c)[0]
        sums = [sum(D[a, j] for j in m) for a in m]
        med.append(m[int(np.argmin(sums))])
    for e in range(30):
        if e in med:
            assert cl[e] == med.index(e)
        else:
            assert cl[e] == int(np.argmin([D[e, q] for q in med]))
    # C = 1: everything in one cluster; dominant = most fired (ties: centrality)
    cl1, fo1, dom1, _ = K.kmedoids(D, fire, 1)
    assert np.all(cl1 == 0) and fire[dom1[0]] == fire.max()
    assert np.sum(fo1 == -1) == 1


def test_dominant_ties_and_protection():
    E = 6
    D = np.full((E, E), 1.5)
    np.fill_diagonal(D, 0)
    D[0, 1] = D[1, 0] = 0.2
    D[0, 2] = D[2, 0] = 0.2
    D[1, 2] = D[2, 1] = 0.9        # 0 is the most central of {0, 1, 2}
    fire = np.array([7, 9, 9, 1, 1, 1])
    # 1 and 2 tie on firing and on centrality (both sum(1 - D) = -0.1)
    cl, fo, dom, _ = K.kmedoids(D, fire, 2, protected=[4])
    assert cl[4] == 1                          # protected: singleton after the seeded
    assert np.sum(cl == 1) == 1
    members0 = np.where(cl == 0)[0]
    assert set(members0.tolist()) == {0, 1, 2, 3, 5}
    # firing tie between 1 and 2 with equal centrality: lower index
    assert dom[0] == 1 and dom[1] == 4
    D[1, 3] = D[3, 1] = 0.1                    # now 1 is more central than 2
    D[2, 3] = D[3, 2] = 1.9
    cl, fo, dom, _ = K.kmedoids(D, fire, 2, protected=[4])
    assert dom[0] == 1
    D[1, 3] = D[3, 1] = 1.9
    D[2, 3] = D[3, 2] = 0.1                    # 2 more central than 1
    cl, fo, dom, _ = K.kmedoids(D, fire, 2, protected=[4])
    assert dom[0] == 2
    assert fo[2] == -1 and fo[4] == -1 and np.sum(fo >= 0) == 4

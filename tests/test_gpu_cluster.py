"""GPU router profiling, NPMI distance and k-medoids against the clustering
oracle. Counts are exact integers (bit-exact); the distance is fp64 whose log
may differ from the host's in the last bits (compared to 1e-13); the
clustering decisions are compared bit-exactly with the oracle run on the
GPU's own distance matrix, so both sides decide on the same fp64 values."""
import numpy as np
import pytest
import torch

from lxsynth import Layer, Level, Problem, Routing, make_x, route_community
from lxsynth.gen import _make_factors, _make_anchors
from oracle import cluster as K
from oracle import moe as O
from paper_2608_07814_amd import lorex as lx
from gpu_util import TOL_BF16, TOL_DESIGN, require_gpu, say, gpu_forward, err_ratio
from helpers import random_routing

pytestmark = pytest.mark.gpu


def _calib(E, groups, N, k, seed):
    members = [list(range(g * (E // groups), (g + 1) * (E // groups))) for g in range(groups)]
    return route_community(N, members, k, 0.7, seed).topk_ids


def _gpu_counts(ids, E):
    fire, pair, dist = lx.coact_distance(torch.from_numpy(np.ascontiguousarray(ids, np.int32)).cuda(), E)
    torch.cuda.synchronize()
    return (fire.cpu().numpy().view(np.uint32).astype(np.int64), pair.cpu().numpy().view(np.uint32).astype(np.int64),
            dist.cpu().numpy(), dist)


@pytest.mark.parametrize("E,groups,N,k", [(128, 32, 4096, 8), (256, 16, 2000, 8), (20, 4, 300, 6)])
def test_counts_and_distance(E, groups, N, k):
    require_gpu()
    say(f"coact E={E} N={N} k={k}")
    ids = _calib(E, groups, N, k, 40 + E)
    if E == 20:  # dropped, invalid and repeated ids are ignored
        ids, _ = random_routing(N, k, E, 41, allow_dupes=True, drop_frac=0.1, bad_frac=0.05)
    fire, pair, dist, _ = _gpu_counts(ids, E)
    f0, p0 = K.coact_counts(ids, E)
    assert np.array_equal(fire, f0) and np.array_equal(pair, p0)
    d0 = K.npmi_distance(f0, p0, N)
    assert np.max(np.abs(dist - d0)) <= 1e-13
    assert np.array_equal(dist, dist.T) and np.all(np.diag(dist) == 0)


@pytest.mark.parametrize("E,C,prot", [(128, 32, ()), (128, 64, (3, 77)), (256, 96, (0, 255, 100)),
                                      (20, 5, (7,))])
def test_kmedoids_matches_oracle(E, C, prot):
    require_gpu()
    say(f"kmedoids E={E} C={C} protected={prot}")
    ids = _calib(E, min(E // 4, 32), 3000, 8, 50 + C)
    fire, _, dist, dist_d = _gpu_counts(ids, E)
    fire_d = torch.from_numpy(fire.astype(np.int32)).cuda()
    cl, fo, dom, it = (t.cpu().numpy() for t in lx.kmedoids(dist_d, fire_d, C, protected=prot))
    c0, f0, d0, it0 = K.kmedoids(dist, fire, C, protected=prot)
    say(f"  {int(it[0])} update rounds (oracle {it0})")
    assert np.array_equal(cl, c0) and np.array_equal(fo, f0) and np.array_equal(dom, d0) and it[0] == it0


def test_kmedoids_metric_large_and_max_iter():
    """E = 1024 points of a Euclidean metric (ties improbable), then the
    iteration cap: max_iter = 0 keeps the seeds' assignment, 1 one update."""
    require_gpu()
    say("kmedoids E=1024 metric")
    rng = np.random.default_rng(9)
    X = rng.standard_normal((1024, 6))
    D = np.sqrt(((X[:, None] - X[None]) ** 2).sum(-1))
    np.fill_diagonal(D, 0)
    fire = rng.integers(0, 10000, 1024)
    Dd = torch.from_numpy(D).cuda()
    fd = torch.from_numpy(fire.astype(np.int32)).cuda()
    for C, mi in ((40, 100), (40, 0), (40, 1)):
        got = [t.cpu().numpy() for t in lx.kmedoids(Dd, fd, C, max_iter=mi)]
        ref = K.kmedoids(D, fire, C, max_iter=mi)
        for g, r in zip(got[:3], ref[:3]):
            assert np.array_equal(g, r)
        assert got[3][0] == ref[3]


def test_clusters_drive_the_forward():
    """Profiling -> distance -> k-medoids on the GPU, then a flat layer built
    on the resulting cluster map runs through lx_moe_forward (oracle parity)."""
    require_gpu()
    say("cluster -> forward")
    E, C, d, f, r, k = 64, 16, 256, 128, 64, 4
    ids = _calib(E, 16, 2000, k, 61)
    fire, _, _, dist_d = _gpu_counts(ids, E)
    cl, fo, dom, _ = (t.cpu().numpy() for t in lx.kmedoids(dist_d, torch.from_numpy(fire.astype(np.int32)).cuda(), C))
    rng = np.random.default_rng(62)
    anchors = _make_anchors(rng, C, d, f, "bf16")
    fac = _make_factors(rng, E - C, d, f, r, "bf16", 0.3)
    layer = Layer(E=E, d=d, f=f, dtype="bf16",
                  levels=[Level(parent=cl.astype(np.int32), factor_of=fo.astype(np.int32), rank=r, **fac)],
                  **anchors)
    T = 200
    x = make_x(T, d, "bf16", 63)
    rids, rw = random_routing(T, k, E, 64)
    p = Problem(cfg={}, seed=63, layer=layer, x=x, routing=Routing(rids, rw))
    e = err_ratio(gpu_forward(p), O.moe_forward(layer, x, rids, rw))
    say(f"  err/RMS = {e:.3e}")
    assert e <= TOL_BF16 and e <= TOL_DESIGN


def _final_margins(D, Dg, cl, C):
    """Smallest gap between the best and the second-best choice among the
    final decisions of a k-medoids result: a member's nearest medoid, and a
    cluster's medoid (smallest in-cluster distance sum). An exact tie that
    both matrices hold exactly (e.g. D = 2 for pairs that never co-fire, no
    rounding involved) is decided by the index on both sides and is skipped."""
    med = []
    gap = np.inf
    for c in range(C):
        mem = np.nonzero(cl == c)[0]
        s = np.array([sum(D[m, j] for j in mem) for m in mem])
        sg = np.array([sum(Dg[m, j] for j in mem) for m in mem])
        med.append(int(mem[np.argmin(s)]))
        if len(mem) > 1:
            o = np.argsort(s, kind="stable")
            g = s[o[1]] - s[o[0]]
            if not (g == 0 and sg[o[1]] == sg[o[0]]):
                gap = min(gap, g)
    med = np.array(med)
    for e in range(D.shape[0]):
        if e in med:
            continue
        o = np.argsort(D[e, med], kind="stable")
        g = D[e, med[o[1]]] - D[e, med[o[0]]]
        if g == 0 and Dg[e, med[o[1]]] == Dg[e, med[o[0]]]:
            continue
        gap = min(gap, g)
    return gap


@pytest.mark.parametrize("E,C,N", [(128, 32, 4096), (64, 16, 2000)])
def test_cluster_chain_against_oracle_only_chain(E, C, N):
    """ids -> counts -> distance -> k-medoids on the GPU against the same chain
    run by the oracle alone (oracle counts, oracle distance, oracle k-medoids).
    The two distance matrices agree to 1e-13; a decision may legitimately
    differ only where two candidates are closer than that bound, so the test
    first shows that every final decision of the oracle's run has a margin far
    above it, and then requires identical clusterings."""
    require_gpu()
    say(f"cluster chain E={E} C={C} N={N}")
    ids = _calib(E, min(E // 4, 32), N, 8, 70 + E)
    fire, _, dist, dist_d = _gpu_counts(ids, E)
    cl, fo, dom, it = (t.cpu().numpy() for t in
                       lx.kmedoids(dist_d, torch.from_numpy(fire.astype(np.int32)).cuda(), C))
    f0, p0 = K.coact_counts(ids, E)
    d0 = K.npmi_distance(f0, p0, N)
    c0, fo0, dom0, it0 = K.kmedoids(d0, f0, C)
    bound = float(np.max(np.abs(dist - d0)))
    margin = _final_margins(d0, dist, c0, C)
    say(f"  distance bound {bound:.2e}, smallest final decision margin {margin:.2e}, rounds {int(it[0])}/{it0}")
    assert bound <= 1e-13
    assert margin > 1e3 * E * max(bound, 1e-16)
    assert np.array_equal(cl, c0) and np.array_equal(fo, fo0) and np.array_equal(dom, dom0) and it[0] == it0

"""GPU bucketing vs the oracle's definition: bit-exact arrays at every level."""
import numpy as np
import pytest
import torch

from lxsynth import make_problem
from oracle import bucket as B
from paper_2608_07814_amd import lorex as lx
from gpu_util import require_gpu, say
from helpers import tiny_flat, tiny_tree, random_routing

pytestmark = pytest.mark.gpu


def _structure(layer):
    return [lv.parent for lv in layer.levels], [layer.n_anchors] + [lv.n_nodes for lv in layer.levels]


def _check(layer, ids, expect_flag=0):
    require_gpu()
    dl = lx.to_device(layer)
    ids_d = torch.from_numpy(np.ascontiguousarray(ids, dtype=np.int32)).cuda()
    T, k = ids.shape
    ws = lx.alloc_workspace(dl, T, k, "tree")
    parents, n_nodes = _structure(layer)
    ref, rflag = B.bucket(parents, n_nodes, layer.E, ids)
    assert rflag == expect_flag
    for li in range(layer.n_levels + 1):
        rt, off, sr = lx.bucket(dl, ids_d, li, workspace=ws)
        assert np.array_equal(off.cpu().numpy(), ref[li]["offsets"]), f"offsets level {li}"
        assert np.array_equal(rt.cpu().numpy(), ref[li]["row_token"]), f"row_token level {li}"
        assert np.array_equal(sr.cpu().numpy(), ref[li]["slot_row"]), f"slot_row level {li}"
    assert lx.read_device_status(ws) & lx.LX_DEVFLAG_BAD_ID == expect_flag


@pytest.mark.parametrize("cfg,T", [(0, 16), (1, 4096), (2, 64), (3, 2000), (3, 16384), (4, 1000), (4, 4096),
                                   (4, 8192), (4, 16384)])
def test_bucket_configs(cfg, T):
    """Full sizes included: cfg3 at T=16384 and the cfg4 tree at T=8192. The
    scan keeps 8, 16 or 32 histogram entries per thread in registers (the
    largest level's entries / 1024 threads, rounded up to a multiple of 4):
    cfg0 at T=16 has fewer token tiles than that block (several node starts
    per block); the tree at T=4096 takes 16; the tree at T=16384 (256 leaves x
    256 token tiles: 64 entries per thread) reads its chunk in two blocks."""
    say(f"bucket cfg{cfg} T={T}")
    p = make_problem(cfg, T=T)
    _check(p.layer, p.routing.topk_ids)


# Batches of at most 64 tokens take the single-workgroup path, larger ones
# the four-pass path; the "small_" cases cover the former.
@pytest.mark.parametrize("case", ["dupes_drops_bad", "all_dropped", "one_hot_expert", "T1", "ragged",
                                  "shuffled", "dense", "small_dupes_drops_bad", "small_all_dropped",
                                  "small_one_hot_expert", "small_tree", "small_k32"])
def test_bucket_adversarial(case):
    say(f"bucket adversarial {case}")
    flag = 0
    small = case.startswith("small_")
    if small:
        case = case[len("small_"):]
    if case == "dupes_drops_bad":
        layer = tiny_flat(E=12, C=3)
        ids, _ = random_routing(50 if small else 150, 6, 12, 9, allow_dupes=True, drop_frac=0.2, bad_frac=0.05)
        flag = lx.LX_DEVFLAG_BAD_ID
    elif case == "all_dropped":
        layer = tiny_flat(E=12, C=3)
        ids = np.full((40 if small else 70, 4), -1, np.int32)
    elif case == "one_hot_expert":
        layer = tiny_flat(E=12, C=3)
        T = 64 if small else 300
        ids = np.full((T, 3), 7, np.int32)
        ids[:, 1] = 2
        ids[::3, 2] = -1
    elif case == "tree":
        layer = tiny_tree(E=16, n_roots=2, subs=2)
        ids, _ = random_routing(33, 5, 16, 13, allow_dupes=True, drop_frac=0.1)
    elif case == "k32":
        layer = tiny_flat(E=40, C=8, shuffle=True)
        ids, _ = random_routing(64, 32, 40, 14, allow_dupes=True)
    elif case == "T1":
        layer = tiny_tree(E=16, n_roots=2, subs=2)
        ids = np.array([[3, 15, 4, 3]], np.int32)
    elif case == "ragged":
        layer = tiny_tree(E=16, n_roots=2, subs=2)
        ids, _ = random_routing(129, 5, 16, 10)
    elif case == "shuffled":
        layer = tiny_flat(E=40, C=8, shuffle=True)
        ids, _ = random_routing(333, 8, 40, 11)
    else:
        layer = tiny_flat(E=10, C=10)
        layer.levels = []
        ids, _ = random_routing(100, 4, 10, 12)
    _check(layer, ids, flag)


def test_bucket_deterministic():
    require_gpu()
    p = make_problem(1, T=4096)
    dl = lx.to_device(p.layer)
    ids_d = torch.from_numpy(p.routing.topk_ids).cuda()
    ws = lx.alloc_workspace(dl, 4096, 8, "tree")
    a = [t.cpu().numpy() for t in lx.bucket(dl, ids_d, 0, workspace=ws)]
    for _ in range(3):
        b = [t.cpu().numpy() for t in lx.bucket(dl, ids_d, 0, workspace=ws)]
        for x, y in zip(a, b):
            assert np.array_equal(x, y)

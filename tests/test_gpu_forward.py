"""GPU forward vs the fp64 oracle, element by element.

Bar: max|diff| <= 1e-2 * RMS(oracle output) for bf16 inputs (fp32 output);
fp32 layers additionally meet 1e-4 * RMS. The full-size configurations compare
every one of the T x d outputs with the oracle, in the launch configuration the
benchmark times.
"""
import numpy as np
import pytest
import torch

from lxsynth import config, make_problem, make_layer_flat
from oracle import moe as O
from paper_2608_07814_amd import lorex as lx
from gpu_util import TOL_BF16, TOL_F32, TOL_DESIGN, require_gpu, say, gpu_forward, err_ratio, dev_inputs
from helpers import tiny_flat, tiny_tree, random_routing, zero_level

pytestmark = pytest.mark.gpu


def _oracle(p, tokens=None):
    return O.moe_forward(p.layer, p.x, p.routing.topk_ids, p.routing.topk_weights, tokens=tokens)


def test_cfg0_fp32_full():
    require_gpu()
    say("forward cfg0 fp32")
    p = make_problem(0)
    got = gpu_forward(p)
    e = err_ratio(got, _oracle(p))
    say(f"  cfg0 err/RMS = {e:.3e}")
    assert e <= TOL_F32


@pytest.mark.parametrize("seed", [1, 101, 201])
def test_cfg1_shapes_full_compare(seed):
    """30B-A3B-class flat layer at T=256 (several tiles, ragged last tile)."""
    require_gpu()
    say(f"forward cfg1 T=256 seed={seed}")
    p = make_problem(1, seed=seed, T=256)
    got = gpu_forward(p)
    e = err_ratio(got, _oracle(p))
    say(f"  err/RMS = {e:.3e}")
    assert e <= TOL_BF16
    assert e <= TOL_DESIGN


def _full_size(cfg):
    """Every output of configuration cfg at its full T against the oracle."""
    require_gpu()
    p = make_problem(cfg)
    say(f"forward cfg{cfg} T={p.T} full compare ({p.T * p.layer.d} outputs)")
    got = gpu_forward(p)
    assert np.all(np.isfinite(got))
    ref = _oracle(p)
    e = err_ratio(got, ref)
    rms = float(np.sqrt(np.mean(ref * ref)))
    # where the largest error sits, and the error of the sampled rows alone
    t_worst = int(np.argmax(np.max(np.abs(got - ref), axis=1)))
    say(f"  cfg{cfg} max|diff|/RMS = {e:.3e} (RMS {rms:.4e}, worst token {t_worst}, "
        f"mean|diff|/RMS {float(np.mean(np.abs(got - ref))) / rms:.3e})")
    assert e <= TOL_BF16
    assert e <= TOL_DESIGN


def test_cfg1_full_size():
    """T=4096, the prefill workload: all 4096 x 2048 outputs."""
    _full_size(1)


def test_cfg2_decode_full():
    require_gpu()
    say("forward cfg2 T=64")
    p = make_problem(2)
    got = gpu_forward(p)
    e = err_ratio(got, _oracle(p))
    say(f"  err/RMS = {e:.3e}")
    assert e <= TOL_BF16
    assert e <= TOL_DESIGN


def test_decode_shape_duplicates_and_drops():
    """Decode-sized batch on fast levels (skinny GEMMs, single-workgroup
    bucketing) with duplicate and dropped slots."""
    require_gpu()
    say("forward decode dupes/drops")
    layer = make_layer_flat(32, 4, 256, 192, 64, "bf16", 21)
    p = _tiny_problem(layer, 48, 8, 22, allow_dupes=True, drop_frac=0.15)
    e = err_ratio(gpu_forward(p), _oracle(p))
    say(f"  err/RMS = {e:.3e}")
    assert e <= TOL_BF16
    assert e <= TOL_DESIGN


def test_cfg3_community():
    require_gpu()
    say("forward cfg3 T=300")
    p = make_problem(3, T=300)
    got = gpu_forward(p)
    e = err_ratio(got, _oracle(p))
    say(f"  err/RMS = {e:.3e}")
    assert e <= TOL_BF16
    assert e <= TOL_DESIGN


def test_cfg3_full_size():
    """T=16384 with community routing: all 16384 x 2048 outputs."""
    _full_size(3)


@pytest.mark.parametrize("cfg,over,T", [(3, {"d": 512, "f": 256}, 40), (1, {"r": 32}, 600),
                                          (1, {"r": 96, "d": 512, "f": 320}, 900),
                                          (3, {"r": 160, "d": 512, "f": 256}, 200)])
def test_rank_not_multiple_of_64(cfg, over, T):
    """Ranks 32, 96 and 160 on the bf16 (hi, lo) path: the low-rank output
    products' 64-wide K-slabs cross from the hi to the lo half of their
    operand (weight columns taken modulo r); small batches of such levels
    stay on the large-tile kernel."""
    require_gpu()
    say(f"rank {over.get('r', 96)} cfg{cfg} {over} T={T}")
    p = make_problem(config(cfg, **over), seed=5 + T)
    e = err_ratio(gpu_forward(p), _oracle(p))
    say(f"  err/RMS = {e:.3e}")
    assert e <= TOL_BF16 and e <= TOL_DESIGN


def test_cfg4_tree_small():
    require_gpu()
    say("forward cfg4 T=8")
    p = make_problem(4, T=8)
    got = gpu_forward(p)
    e = err_ratio(got, _oracle(p))
    say(f"  err/RMS = {e:.3e}")
    assert e <= TOL_BF16
    assert e <= TOL_DESIGN


def test_cfg4_tree_mixed_kernels():
    """T=100: the root level runs on the large-tile kernel while the sub and
    leaf levels (few rows per node) run on the skinny kernel."""
    require_gpu()
    say("forward cfg4 T=100")
    p = make_problem(4, T=100)
    got = gpu_forward(p)
    e = err_ratio(got, _oracle(p))
    say(f"  err/RMS = {e:.3e}")
    assert e <= TOL_BF16
    assert e <= TOL_DESIGN


def test_cfg4_tree_full_size():
    """The BTExperts tree at T=8192: all 8192 x 4096 outputs (the sub and leaf
    levels run on the large-tile kernel at this size)."""
    _full_size(4)


# ------------------------------------------------------------ edge cases
def _tiny_problem(layer, T, k, seed, dtype=None, **kw):
    from lxsynth import Problem, Routing
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, layer.d)).astype(np.float32)
    if layer.dtype == "bf16":
        from lxsynth import f32_to_bf16_bits
        x = f32_to_bf16_bits(x)
    ids, w = random_routing(T, k, layer.E, seed + 1, **kw)
    return Problem(cfg={}, seed=seed, layer=layer, x=x, routing=Routing(ids, w))


@pytest.mark.parametrize("dtype,T", [("f32", 77), ("bf16", 77), ("bf16", 40)])
def test_dropped_duplicate_and_bad_ids(dtype, T):
    """T=40 takes the single-workgroup bucketing, T=77 the four-pass one."""
    require_gpu()
    say(f"edge ids {dtype} T={T}")
    layer = make_layer_flat(12, 3, 64, 96, 16, dtype, 5)
    p = _tiny_problem(layer, T, 5, 3, allow_dupes=True, drop_frac=0.2, bad_frac=0.05)
    got, ws = gpu_forward(p, return_ws=True)
    ref, flag = O.moe_forward(p.layer, p.x, p.routing.topk_ids, p.routing.topk_weights,
                              return_flag=True)
    assert flag == O.FLAG_BAD_ID
    assert lx.read_device_status(ws) & lx.LX_DEVFLAG_BAD_ID
    assert err_ratio(got, ref) <= (TOL_F32 if dtype == "f32" else TOL_BF16)


def test_all_dropped_gives_zero_and_T1():
    require_gpu()
    say("edge all dropped / T=1")
    layer = make_layer_flat(8, 2, 64, 128, 8, "bf16", 6)
    p = _tiny_problem(layer, 9, 2, 4)
    got = gpu_forward(p, ids=np.full((9, 2), -1, np.int32))
    assert np.all(got == 0)
    p1 = _tiny_problem(layer, 1, 2, 5)
    assert err_ratio(gpu_forward(p1), _oracle(p1)) <= TOL_BF16


def test_T0_is_noop():
    require_gpu()
    layer = make_layer_flat(8, 2, 64, 128, 8, "bf16", 6)
    dl = lx.to_device(layer)
    x = torch.empty(0, 64, dtype=torch.bfloat16, device="cuda")
    ids = torch.empty(0, 2, dtype=torch.int32, device="cuda")
    w = torch.empty(0, 2, dtype=torch.float32, device="cuda")
    out = lx.forward(dl, x, ids, w)
    torch.cuda.synchronize()
    assert out.shape == (0, 64)


def test_hot_expert_and_empty_clusters():
    """Every token on the same two experts: most clusters and experts empty,
    one group spans many tiles."""
    require_gpu()
    say("edge hot expert")
    layer = make_layer_flat(16, 4, 128, 256, 16, "bf16", 7)
    p = _tiny_problem(layer, 700, 2, 6)
    ids = np.stack([np.full(700, 5), np.full(700, 6)], 1).astype(np.int32)
    p.routing.topk_ids[:] = ids
    assert err_ratio(gpu_forward(p), _oracle(p)) <= TOL_BF16


def test_shuffled_clusters_and_bf16_output():
    require_gpu()
    say("edge shuffled clusters, bf16 out")
    layer = make_layer_flat(32, 8, 256, 128, 32, "bf16", 8, shuffle=True)
    p = _tiny_problem(layer, 200, 6, 9)
    ref = _oracle(p)
    assert err_ratio(gpu_forward(p), ref) <= TOL_BF16
    got16 = gpu_forward(p, out_dtype=lx.LX_BF16)
    # bf16 rounding of the output alone is ~2^-9 relative per element
    assert err_ratio(got16, ref) <= 4e-2


def test_flat_tree_and_determinism():
    """lx_moe_forward and lx_moe_forward_tree on the same flat layer agree
    bitwise, and repeated calls are bitwise identical (no atomics)."""
    require_gpu()
    say("flat vs tree api, determinism")
    p = make_problem(1, T=512)
    dl = lx.to_device(p.layer)
    a = gpu_forward(p, kind="flat", dev_layer=dl)
    b = gpu_forward(p, kind="tree", dev_layer=dl)
    c = gpu_forward(p, kind="flat", dev_layer=dl)
    assert np.array_equal(a, b) and np.array_equal(a, c)


def test_zero_corrections_on_gpu():
    require_gpu()
    say("zero corrections")
    p = make_problem(1, T=128)
    p.layer = zero_level(p.layer, 0)
    assert err_ratio(gpu_forward(p), _oracle(p)) <= TOL_BF16


def test_tree_generic_levels():
    """A three-level tree with some factor-less nodes, fp32 and bf16."""
    require_gpu()
    say("generic tree")
    for dtype in ("f32", "bf16"):
        layer = tiny_tree(E=32, d=64, f=48, n_roots=2, subs=2, r_sub=16, r_leaf=8, dtype=dtype, seed=12)
        layer.levels[0].factor_of[1] = -1
        layer.levels[1].factor_of[3:9] = -1
        p = _tiny_problem(layer, 90, 6, 13, drop_frac=0.1)
        assert err_ratio(gpu_forward(p), _oracle(p)) <= (TOL_F32 if dtype == "f32" else TOL_BF16)


def test_general_token_kernels():
    """k > 8 slots and a three-level correction tree take the general SwiGLU
    and combine kernels (the fast ones cover k <= 8 with at most two
    correction levels), here on bf16 shapes whose levels all keep f24 rows."""
    require_gpu()
    from lxsynth import Level
    from lxsynth.gen import _make_factors
    say("general token kernels: k=12 flat, three-level tree")
    layer = make_layer_flat(32, 4, 64, 128, 64, "bf16", 21)
    p = _tiny_problem(layer, 70, 12, 22, drop_frac=0.1)
    assert err_ratio(gpu_forward(p), _oracle(p)) <= TOL_DESIGN
    # depth-2 tree over 16 nodes, then 2 leaves (rank 64) under each of them
    base = tiny_tree(E=16, d=64, f=64, n_roots=2, subs=2, r_sub=64, r_leaf=64, dtype="bf16", seed=23)
    f3 = _make_factors(np.random.default_rng(24), 32, 64, 64, 64, "bf16", 0.3)
    base.levels.append(Level(parent=(np.arange(32) // 2).astype(np.int32),
                             factor_of=np.arange(32, dtype=np.int32), rank=64, **f3))
    base.levels[2].factor_of[5] = -1
    base.E = 32
    p3 = _tiny_problem(base, 50, 6, 25)
    assert err_ratio(gpu_forward(p3), _oracle(p3)) <= TOL_DESIGN


def test_dense_comparator():
    """L = 0: the uncompressed MoE through lx_dense_moe_forward."""
    require_gpu()
    say("dense comparator")
    layer = make_layer_flat(16, 16, 256, 128, 8, "bf16", 14)
    layer.levels = []
    p = _tiny_problem(layer, 300, 4, 15)
    assert err_ratio(gpu_forward(p, kind="dense"), _oracle(p)) <= TOL_BF16


def test_aux_stream_switch_bitwise():
    """With the auxiliary stream turned on (lx_set_aux_stream(1)) the
    correction chains fork onto it; the results are bitwise those of the
    default single-stream run, flat and tree."""
    require_gpu()
    say("aux stream on/off")
    for cfg, T in ((1, 700), (4, 300), (4, 2304)):
        p = make_problem(cfg, T=T)
        dl = lx.to_device(p.layer)
        a = gpu_forward(p, dev_layer=dl)
        prev = lx.set_aux_stream(True)
        try:
            b = gpu_forward(p, dev_layer=dl)
        finally:
            lx.set_aux_stream(prev)
        assert np.array_equal(a, b), f"cfg{cfg} T={T}"


def _merged_layer(case):
    from lxsynth import Level, make_layer_tree
    from lxsynth.gen import _make_factors
    if case == "three_levels":
        base = tiny_tree(E=16, d=512, f=256, n_roots=2, subs=2, r_sub=128, r_leaf=64, dtype="bf16", seed=31)
        f3 = _make_factors(np.random.default_rng(32), 32, 512, 256, 64, "bf16", 0.3)
        base.levels.append(Level(parent=(np.arange(32) // 2).astype(np.int32),
                                 factor_of=np.arange(32, dtype=np.int32), rank=64, **f3))
        base.levels[1].factor_of[5] = -1
        base.levels[2].factor_of[[0, 9, 17]] = -1
        base.E = 32
        return base, 1024
    layer = make_layer_tree(64, 512, 256, 2, 4, 128, 64, "bf16", 33)
    if case == "holes":
        layer.levels[0].factor_of[1] = -1          # a sub-dominant without a correction
        layer.levels[1].factor_of[3:11] = -1       # leaves without one (some under that sub)
    return layer, 2048


@pytest.mark.parametrize("case", ["all_factors", "holes", "three_levels"])
def test_merged_tree_products(case):
    """Trees whose correction levels all run on the large-tile kernel compute
    every level's gate|up and down corrections as one product over the leaf
    rows (K concatenated over the levels; an intermediate level's down term
    rides on the leaf row of its first slot). Leaves and sub-dominants without
    factors, dropped and duplicate slots; three levels take the general token
    kernels. The merged launches must be the ones that ran."""
    require_gpu()
    say(f"merged tree products: {case}")
    layer, T = _merged_layer(case)
    p = _tiny_problem(layer, T, 4, 34, allow_dupes=(case == "holes"), drop_frac=0.1 if case == "holes" else 0.0)
    lx.profile_reset()
    lx.profile_enable(True)
    try:
        got = gpu_forward(p)
        names = set(lx.profile_read())
    finally:
        lx.profile_enable(False)
    assert "lowrank_gate_up_out_merged" in names and "lowrank_down_out_merged" in names, names
    assert not any(n.startswith("lowrank_down_out_l") for n in names)
    e = err_ratio(got, _oracle(p))
    say(f"  err/RMS = {e:.3e}")
    assert e <= TOL_BF16 and e <= TOL_DESIGN
    # a second call gives the same bits
    assert np.array_equal(got, gpu_forward(p))


@pytest.mark.parametrize("cfg,T", [(2, 64), (1, 700), (4, 2304)])
def test_hip_graph_capture_replays(cfg, T):
    """The forward captured into a HIP graph (torch's CUDAGraph API; every
    launch on the caller's stream, no allocation, memset or host sync inside
    the call) replays to the eager result bitwise, several times, with eager
    forwards on other routing run between the replays."""
    require_gpu()
    import torch
    say(f"graph capture cfg{cfg} T={T}")
    p = make_problem(cfg, T=T)
    dl = lx.to_device(p.layer)
    xt, ids_d, w_d = dev_inputs(p)
    kind = {1: "flat"}.get(len(dl.levels), "tree")
    ws = lx.alloc_workspace(dl, p.T, p.k, kind)
    out = torch.empty(p.T, p.layer.d, dtype=torch.float32, device="cuda")
    eager = gpu_forward(p, dev_layer=dl)
    call = lx.PreparedCall(dl, xt, ids_d, w_d, out, ws, kind)
    call()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        lx.PreparedCall(dl, xt, ids_d, w_d, out, ws, kind)()
    rng = np.random.default_rng(7)
    out2 = torch.empty_like(out)
    for rep in range(3):
        out.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy().astype(np.float64), eager), f"replay {rep}"
        # eager work on another routing between replays, in the same workspace
        perm = torch.from_numpy(rng.permutation(p.T)).cuda()
        lx.PreparedCall(dl, xt, ids_d[perm].contiguous(), w_d[perm].contiguous(), out2, ws, kind)()
        torch.cuda.synchronize()

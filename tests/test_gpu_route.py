"""GPU top-k router (lx_route_topk) against the fp64 router oracle.

The GPU takes its decisions on fp32 logits; the oracle's are fp64. Where two
logits are closer than the fp32 summation bound of both (oracle.router.
fp32_sum_bound), either order is correct, so the comparison is tie-aware:
every chosen expert must beat every unchosen one, and each chosen one its
successor, up to the two bounds; tokens whose top-(k+1) logits are all
farther apart than that must match the oracle exactly. Weights are compared
with the softmax of the oracle's fp64 logits over the GPU's chosen experts.
"""
import numpy as np
import pytest
import torch

from lxsynth import config, make_problem, make_router, make_x
from oracle import moe as O
from oracle import router as R
from paper_2608_07814_amd import lorex as lx
from gpu_util import TOL_BF16, TOL_DESIGN, require_gpu, say, err_ratio

pytestmark = pytest.mark.gpu


def _bf16_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)


def _check(x, w, k, ids, wts):
    T, E = x.shape[0], w.shape[0]
    ref_ids, _, lg = R.route_topk(x, w, "bf16", k)
    b = R.fp32_sum_bound(x, w, "bf16")
    assert ids.shape == (T, k) and ids.min() >= 0 and ids.max() < E
    for t in range(T):
        assert len(set(ids[t].tolist())) == k
    rows = np.arange(T)[:, None]
    lc, bc = lg[rows, ids], b[rows, ids]
    # ordered within the bounds
    assert np.all(lc[:, :-1] + bc[:, :-1] + bc[:, 1:] >= lc[:, 1:])
    # every chosen beats every unchosen within the bounds
    mask = np.ones((T, E), bool)
    mask[rows, ids] = False
    lu = np.where(mask, lg, -np.inf)
    bu = np.where(mask, b, 0.0)
    worst_chosen = np.min(lc + bc, axis=1)
    best_unchosen = np.max(lu - bu, axis=1)
    assert np.all(worst_chosen >= best_unchosen)
    # clear tokens match exactly
    srt = np.sort(lg, axis=1)[:, ::-1][:, :k + 1]
    gaps = -np.diff(srt, axis=1)
    clear = np.all(gaps > 2 * b.max(axis=1, keepdims=True), axis=1)
    assert np.array_equal(ids[clear], ref_ids[clear])
    # weights: softmax of the fp64 logits over the GPU's chosen experts
    ex = np.exp(lc - lc.max(axis=1, keepdims=True))
    w64 = ex / ex.sum(axis=1, keepdims=True)
    tol = w64 * (2 * b.max(axis=1, keepdims=True) + 4e-7) + 1e-7
    assert np.all(np.abs(wts - w64) <= tol)
    return float(clear.mean()), float(np.mean(np.all(ids == ref_ids, axis=1)))


@pytest.mark.parametrize("T,d,E,k", [(1, 2048, 128, 8), (64, 2048, 128, 8), (100, 256, 8, 2),
                                     (4096, 2048, 128, 8), (33, 4096, 256, 8), (50, 128, 512, 32),
                                     (7, 512, 40, 32), (45, 1024, 64, 1), (5, 1216, 100, 6)])
def test_route_matches_oracle(T, d, E, k):
    require_gpu()
    say(f"route T={T} d={d} E={E} k={k}")
    x = make_x(T, d, "bf16", 70 + T)
    w = make_router(d, E, "bf16", 70 + T)
    ids, wts = lx.route_topk(_bf16_dev(x), _bf16_dev(w), k)
    torch.cuda.synchronize()
    clear, same = _check(x, w, k, ids.cpu().numpy(), wts.cpu().numpy().astype(np.float64))
    # the worst-case bound is loose (d u sum|x w|): few tokens are provably
    # unambiguous at large d, but in practice the ids match the oracle's
    say(f"  provably unambiguous {clear:.3f} (all exact); identical to the oracle on {same:.3f}")
    assert clear > 0.1 and same > 0.95


def test_route_ties_determinism_and_edges():
    """Equal router rows give bitwise equal logits: the lower index goes
    first. Repeated calls are bitwise identical. Extreme activations stay
    finite and the weights sum to 1."""
    require_gpu()
    say("route ties / determinism")
    x = make_x(300, 512, "bf16", 3)
    w = make_router(512, 64, "bf16", 3)
    w[37] = w[5]
    w[6] = w[5]
    xd, wd = _bf16_dev(x), _bf16_dev(w)
    a = [lx.route_topk(xd, wd, 6) for _ in range(3)]
    torch.cuda.synchronize()
    ids = a[0][0].cpu().numpy()
    for i, v in a[1:]:
        assert torch.equal(i, a[0][0]) and torch.equal(v, a[0][1])
    pos = {e: np.where(ids == e, np.arange(6)[None, :], 99).min(1) for e in (5, 6, 37)}
    has = pos[37] < 99
    assert np.all(pos[5][has] < pos[6][has]) and np.all(pos[6][has] < pos[37][has])
    wts = a[0][1].cpu().numpy()
    sel = (pos[5] < 99) & (pos[6] < 99)
    assert np.all(wts[sel, pos[5][sel]] == wts[sel, pos[6][sel]])
    _check(x, w, 6, ids, wts.astype(np.float64))
    # large activations: logits of order 1e3, softmax saturates to one expert
    xb = (make_x(20, 512, "f32", 4) * 512).astype(np.float32)
    from lxsynth import f32_to_bf16_bits
    xb = f32_to_bf16_bits(xb)
    i2, w2 = lx.route_topk(_bf16_dev(xb), wd, 4)
    w2 = w2.cpu().numpy()
    assert np.all(np.isfinite(w2)) and np.all(np.abs(w2.sum(1) - 1) < 1e-5)


def test_route_then_forward_on_one_stream():
    """Routing on the GPU feeding the compressed forward (no host round trip),
    against the oracle forward on the same ids and weights."""
    require_gpu()
    say("route -> forward, cfg1 shapes T=256")
    p = make_problem(1, T=256)
    w = make_router(p.layer.d, p.layer.E, "bf16", p.seed)
    dl = lx.to_device(p.layer)
    xd = _bf16_dev(p.x)
    ids, wts = lx.route_topk(xd, _bf16_dev(w), p.k)
    out = lx.forward(dl, xd, ids, wts)
    torch.cuda.synchronize()
    ids_h, w_h = ids.cpu().numpy(), wts.cpu().numpy()
    _check(p.x, w, p.k, ids_h, w_h.astype(np.float64))
    ref = O.moe_forward(p.layer, p.x, ids_h, w_h)
    e = err_ratio(out.cpu().numpy().astype(np.float64), ref)
    say(f"  err/RMS = {e:.3e}")
    assert e <= TOL_BF16 and e <= TOL_DESIGN


@pytest.mark.parametrize("cfg,T", [(2, 64), (1, 300), (4, 100), (4, 2500)])
def test_route_fused_into_bucketing(cfg, T):
    """lx_route_moe_forward_tree: the router's top-k runs inside the first
    bucketing kernel, the histogram pass (batches of at most 64 tokens keep
    the router's own top-k launch ahead of the single-workgroup bucketing;
    split-K router logits at these sizes). Its ids and weights are
    bitwise those of lx_route_topk, tie-aware against the fp64 router oracle;
    the bucketing of those ids is byte-equal to the bucketing oracle's; the
    output is bitwise that of lx_moe_forward_tree on the same ids and meets
    the oracle bar; no separate top-k launch runs."""
    require_gpu()
    from oracle import bucket as B
    say(f"route fused into bucketing cfg{cfg} T={T}")
    p = make_problem(cfg, T=T)
    w = make_router(p.layer.d, p.layer.E, "bf16", p.seed)
    dl = lx.to_device(p.layer)
    xd, wd = _bf16_dev(p.x), _bf16_dev(w)
    lx.profile_reset()
    lx.profile_enable(True)
    try:
        out, ids, wts = lx.route_forward(dl, xd, wd, p.k)
        names = list(lx.profile_read())
    finally:
        lx.profile_enable(False)
    assert "router_logits" in names
    if T <= 64:  # the single-workgroup bucketing keeps the router's own top-k launch
        assert "router_topk" in names and "bucket_small" in names, names
    else:
        assert "router_topk" not in names and "router_topk+bucket_hist" in names, names
    ids_r, wts_r = lx.route_topk(xd, wd, p.k)
    torch.cuda.synchronize()
    assert torch.equal(ids, ids_r) and torch.equal(wts, wts_r)
    ids_h, w_h = ids.cpu().numpy(), wts.cpu().numpy()
    _check(p.x, w, p.k, ids_h, w_h.astype(np.float64))
    # the bucketing of the GPU's own ids against the bucketing oracle
    parents = [lv.parent for lv in p.layer.levels]
    n_nodes = [p.layer.n_anchors] + [lv.n_nodes for lv in p.layer.levels]
    ref, _ = B.bucket(parents, n_nodes, p.layer.E, ids_h)
    ws = lx.alloc_workspace(dl, T, p.k, "tree")
    for li in range(p.layer.n_levels + 1):
        rt, off, sr = (t.cpu().numpy() for t in lx.bucket(dl, ids, li, workspace=ws))
        assert np.array_equal(off, ref[li]["offsets"]) and np.array_equal(rt, ref[li]["row_token"])
        assert np.array_equal(sr, ref[li]["slot_row"])
    # the forward on those ids: bitwise the unfused call, and the oracle bar
    plain = lx.forward(dl, xd, ids, wts, kind="tree")
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    assert np.array_equal(got, plain.cpu().numpy())
    e = err_ratio(got.astype(np.float64), O.moe_forward(p.layer, p.x, ids_h, w_h))
    say(f"  err/RMS = {e:.3e}")
    assert e <= TOL_BF16 and e <= TOL_DESIGN

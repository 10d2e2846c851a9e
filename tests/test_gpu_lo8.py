"""The anchor down projection's precision modes: the fp8 lo half and fp16.

lx_quantize_f8 is checked byte for byte against an encoder written here from
the format definitions (OCP e4m3: sign, 4 exponent bits with bias 7, 3
mantissa bits, subnormals below 2^-6, 0x7E = 448 the largest finite value;
E8M0: value 2^(byte - 127)), and the forward with the fp8 copy against the
oracle and against the bf16 (hi, lo) path.
"""
import numpy as np
import pytest
import torch

from lxsynth import config, make_problem
from oracle import moe as O
from paper_2608_07814_amd import lorex as lx
from gpu_util import TOL_BF16, TOL_DESIGN, require_gpu, say, gpu_forward, err_ratio, sample_tokens

pytestmark = pytest.mark.gpu


def _e4m3_table():
    codes = np.arange(0x7F)  # 0x00 .. 0x7E (0x7F is NaN)
    e, m = codes >> 3, codes & 7
    return np.where(e == 0, m / 8.0 * 2.0 ** -6, (1 + m / 8.0) * 2.0 ** (e - 7.0))


def _encode_e4m3(x):
    """Nearest e4m3 code (ties to the even code) of |x| <= 448, with x's sign."""
    tab = _e4m3_table()
    a = np.abs(x).ravel()
    hi = np.searchsorted(tab, a, side="left").clip(1, len(tab) - 1)
    lo = hi - 1
    dlo, dhi = a - tab[lo], tab[hi] - a
    pick = np.where(dlo < dhi, lo, np.where(dhi < dlo, hi, np.where(lo % 2 == 0, lo, hi)))
    pick = np.where(a >= tab[-1], len(tab) - 1, pick)
    return (pick | np.where(np.signbit(x.ravel()), 0x80, 0)).reshape(x.shape).astype(np.uint8)


def _reference_quantize(w):
    """w float64 [rows][cols] (bf16 values) -> codes [rows][cols], words [rows][cols // 64]."""
    rows, cols = w.shape
    blocks = w.reshape(rows, cols // 32, 32)
    amax = np.abs(blocks).max(axis=2)
    e = np.where(amax > 0, np.floor(np.log2(np.where(amax > 0, amax, 1.0))), -127)
    b = np.clip(e - 7 + 127, 1, 254).astype(np.int64)
    scaled = blocks * 2.0 ** (127 - b)[:, :, None]
    codes = _encode_e4m3(scaled).reshape(rows, cols)
    words = (b[:, 0::2] | (b[:, 1::2] << 8)).astype(np.int64)
    return codes, words


def test_quantize_f8_bytes():
    require_gpu()
    rng = np.random.default_rng(31)
    w = (rng.standard_normal((2, 8, 192)) * 0.02).astype(np.float32)
    w[0, 1, :32] = 0.0                    # an all-zero block
    w[0, 2, 5] = 3.0                      # one large value in a block of small ones
    w[1, 3, 64:96] *= 1e-4                # tiny block
    w[1, 4, 7] = -w[1, 4, 7]
    wt = torch.from_numpy(w).cuda().to(torch.bfloat16)
    w8, sc = lx.quantize_f8(wt)
    torch.cuda.synchronize()
    wv = wt.float().cpu().numpy().astype(np.float64)
    for n in range(2):
        codes, words = _reference_quantize(wv[n])
        assert np.array_equal(w8[n].cpu().numpy(), codes), n
        assert np.array_equal(sc[n].cpu().numpy().astype(np.int64) & 0xFFFFFFFF, words), n


@pytest.mark.parametrize("cfg,T", [(1, 384), (4, 96)])
def test_lo8_forward_vs_oracle_and_bf16_pair(cfg, T):
    """Both anchor-down paths meet the bar; the fp8 lo half stays within the
    design bound (a lost lo half would give ~1e-2)."""
    require_gpu()
    p = make_problem(cfg, T=T)
    ref = O.moe_forward(p.layer, p.x, p.routing.topk_ids, p.routing.topk_weights)
    e8 = err_ratio(gpu_forward(p, dev_layer=lx.to_device(p.layer, lo8=True, f16=False)), ref)
    e16 = err_ratio(gpu_forward(p, dev_layer=lx.to_device(p.layer, lo8=False, f16=False)), ref)
    say(f"cfg{cfg} T={T}: fp8-lo err/RMS {e8:.3e}, bf16-pair err/RMS {e16:.3e}")
    assert e16 <= TOL_DESIGN
    assert e8 <= TOL_DESIGN


def test_lo8_dense_comparator():
    require_gpu()
    from lxsynth import make_layer_flat
    from helpers import random_routing
    from lxsynth import Problem, Routing, f32_to_bf16_bits
    layer = make_layer_flat(16, 16, 256, 128, 8, "bf16", 14)
    layer.levels = []
    rng = np.random.default_rng(15)
    x = f32_to_bf16_bits(rng.standard_normal((300, 256)).astype(np.float32))
    ids, w = random_routing(300, 4, 16, 16)
    p = Problem(cfg={}, seed=15, layer=layer, x=x, routing=Routing(ids, w))
    got = gpu_forward(p, kind="dense", dev_layer=lx.to_device(layer, lo8=True, f16=False))
    ref = O.moe_forward(layer, x, ids, w)
    assert err_ratio(got, ref) <= TOL_DESIGN


def test_convert_f16_exact():
    """lx_convert_f16: per matrix the exponent puts the largest magnitude in
    [2^14, 2^15), and every value is the bf16 value times 2^exp exactly (all
    of these are within fp16's normal range after scaling); an all-zero
    matrix gets exponent 0."""
    require_gpu()
    rng = np.random.default_rng(41)
    w = (rng.standard_normal((4, 16, 320)) * 0.02).astype(np.float32)
    w[1] *= 3000.0           # large weights
    w[2] = 0.0               # all zero
    w[3] *= 1e-6             # tiny weights
    w[3, 0, 0] = 2.0 ** -20  # an exact power of two as the maximum
    wt = torch.from_numpy(w).cuda().to(torch.bfloat16)
    w16, ex = lx.convert_f16(wt)
    torch.cuda.synchronize()
    wv = wt.float().cpu().numpy().astype(np.float64)
    ex = ex.cpu().numpy()
    for i in range(4):
        m = np.abs(wv[i]).max()
        want = 0 if m == 0 else 14 - int(np.floor(np.log2(m)))
        assert ex[i] == want, (i, ex[i], want)
        got = w16[i].float().cpu().numpy().astype(np.float64) * 2.0 ** -int(ex[i])
        assert np.array_equal(got, wv[i]), i


def test_paired_down_launch_small_grid():
    """The tree's fp16 anchor down projection and merged down-in share one
    persistent launch, whose schedule spreads the second product's items over
    the XCDs from the last one down. With one anchor, one sub-node and two
    leaves at T = 512, k = 1 the launch bound is 7 work items: the grid is
    rounded up to a multiple of 8 so that every XCD has a workgroup. Every
    output against the oracle, and the paired launch ran."""
    require_gpu()
    p = make_problem(config(4, E=2, d=256, f=256, n_roots=1, subs_per_root=1, r_sub=64, r_leaf=64, k=1), T=512)
    ref = O.moe_forward(p.layer, p.x, p.routing.topk_ids, p.routing.topk_weights)
    lx.profile_reset()
    lx.profile_enable(True)
    try:
        got = gpu_forward(p)
        names = lx.profile_read()
    finally:
        lx.profile_enable(False)
        lx.profile_reset()
    assert "anchor_down+lowrank_down_in_merged" in names, sorted(names)
    e = err_ratio(got, ref)
    say(f"small paired launch: err/RMS {e:.3e}")
    assert e <= TOL_DESIGN


def test_padded_copies_exact():
    """lx_convert_f16_padded equals lx_convert_f16 in the original rows and
    columns (same values, same exponents) and is exactly zero in the padding;
    lx_pad_bf16 copies the bf16 values unchanged and zero-fills the rest."""
    require_gpu()
    rng = np.random.default_rng(43)
    w = (rng.standard_normal((3, 96, 200)) * 0.02).astype(np.float32)
    w[1] *= 1e3
    w[2] = 0.0
    wt = torch.from_numpy(w).cuda().to(torch.bfloat16)
    w16, ex = lx.convert_f16(wt)
    for rows_out, cols_out in ((128, 200), (96, 256), (100, 264)):
        p16, pex = lx.convert_f16_padded(wt, rows_out, cols_out)
        pb = lx.pad_bf16(wt, rows_out, cols_out)
        torch.cuda.synchronize()
        assert torch.equal(pex, ex)
        assert torch.equal(p16[:, :96, :200].view(torch.int16), w16.view(torch.int16))
        assert torch.equal(pb[:, :96, :200].view(torch.int16), wt.view(torch.int16))
        mask = torch.ones(rows_out, cols_out, dtype=torch.bool, device=wt.device)
        mask[:96, :200] = False
        assert int(p16.view(torch.int16)[:, mask].abs().max()) == 0 if mask.any() else True
        assert int(pb.view(torch.int16)[:, mask].abs().max()) == 0 if mask.any() else True


@pytest.mark.parametrize("cfg,T,kind", [(1, 1024, None), (4, 600, None), ("dense", 600, "dense")])
def test_f16_forward(cfg, T, kind):
    """With the fp16 copy the anchor down projection multiplies fp16 sums
    (a different result from the fp8-lo path: the path ran) within the
    design bound, and the output meets the bar, flat, tree and uncompressed."""
    require_gpu()
    if cfg == "dense":
        from lxsynth import make_layer_flat, Problem, Routing, f32_to_bf16_bits
        from helpers import random_routing
        layer = make_layer_flat(16, 16, 256, 256, 8, "bf16", 44)
        layer.levels = []
        rng = np.random.default_rng(45)
        x = f32_to_bf16_bits(rng.standard_normal((T, 256)).astype(np.float32))
        ids, w = random_routing(T, 4, 16, 46)
        p = Problem(cfg={}, seed=45, layer=layer, x=x, routing=Routing(ids, w))
    else:
        p = make_problem(cfg, T=T)
    ref = O.moe_forward(p.layer, p.x, p.routing.topk_ids, p.routing.topk_weights)
    g16 = gpu_forward(p, kind=kind, dev_layer=lx.to_device(p.layer, lo8=True, f16=True))
    g8 = gpu_forward(p, kind=kind, dev_layer=lx.to_device(p.layer, lo8=True, f16=False))
    e16, e8 = err_ratio(g16, ref), err_ratio(g8, ref)
    say(f"{cfg} T={T}: fp16 err/RMS {e16:.3e}, fp8-lo err/RMS {e8:.3e}")
    assert not np.array_equal(g16, g8)
    assert e16 <= TOL_DESIGN and e16 <= TOL_BF16


@pytest.mark.parametrize("cfg,T,used", [(1, 2048, True), (4, 2304, True), (3, 2048, True)])
def test_f16_correction_products(cfg, T, used):
    """With the fp16 copies of the factors every correction product runs once
    in fp16 (tile-scaled fp16 intermediates, token-scaled fp16 activation
    sums): a different result from the same layer without those copies (the
    path ran), and both meet the design bound against the oracle. Rank 96
    (not a multiple of 64) runs on copies padded with zeros to rank 128.
    (Sizes with more than 64 rows per expert at every level: smaller batches
    take the skinny kernel, which keeps the pairs.)"""
    require_gpu()
    p = make_problem(cfg, T=T)
    ref = O.moe_forward(p.layer, p.x, p.routing.topk_ids, p.routing.topk_weights)
    full = lx.to_device(p.layer, lo8=True, f16=True)
    assert all(lv.b_down_f16 is not None for lv in full.levels if lv.n_factors > 0)
    if cfg == 3:
        assert all(lv.rank_f16 == 128 and lv.b_gate_pad is not None for lv in full.levels)
    anchor_only = lx.to_device(p.layer, lo8=True, f16=True)
    for lv in anchor_only.levels:
        for n in lx.FACTOR_F16 + lx.FACTOR_PAD:
            setattr(lv, n, None)
        lv.rank_f16 = 0
    g_full = gpu_forward(p, dev_layer=full)
    g_anchor = gpu_forward(p, dev_layer=anchor_only)
    e_full, e_anchor = err_ratio(g_full, ref), err_ratio(g_anchor, ref)
    say(f"cfg{cfg} T={T}: fp16 corrections err/RMS {e_full:.3e}, bf16-pair corrections {e_anchor:.3e}")
    assert np.array_equal(g_full, g_anchor) != used
    assert e_full <= TOL_DESIGN and e_anchor <= TOL_DESIGN

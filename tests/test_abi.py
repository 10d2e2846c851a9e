"""The C ABI on the CPU: library loads, exports every declared entry point, and
host-side validation and workspace planning behave as documented. No call
here reaches a kernel launch (no GPU in this environment)."""
import ctypes
import os
import re

import pytest

from paper_2608_07814_amd import lorex as lx

FAKE = 0x10000  # a 16-byte-aligned address that is never dereferenced


@pytest.fixture(scope="module")
def L(root):
    if not os.path.exists(lx.LIB_PATH):
        from paper_2608_07814_amd import build
        build.build()
    return lx.lib()


def _declared(root):
    src = open(os.path.join(root, "include", "lorex.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(lx_[a-z0-9_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported(L, root):
    names = _declared(root)
    assert len(names) == len(lx.EXPORTS) == 35
    for n in names:
        assert hasattr(L, n), n
        assert n in lx.EXPORTS, n


def test_status_strings_and_version(L):
    assert lx.status_string(lx.LX_OK) == "LX_OK"
    assert lx.status_string(lx.LX_ERR_WORKSPACE_TOO_SMALL) == "LX_ERR_WORKSPACE_TOO_SMALL"
    assert L.lx_version() >= 100


def _tree(E=128, C=16, d=2048, f=768, r=64, levels=1, dtype=lx.LX_BF16, M=None):
    s = lx.LxTreeLayer()
    s.E, s.d, s.f, s.dtype = E, d, f, dtype
    s.n_anchors = C if levels else E
    s.anchor_gate = s.anchor_up = s.anchor_down = FAKE
    s.n_levels = levels
    for i in range(levels):
        c = s.levels[i]
        c.n_nodes = E
        c.rank = r
        c.n_factors = E - C if M is None else M
        c.parent = c.factor_of = FAKE
        c.a_gate = c.b_gate = c.a_up = c.b_up = c.a_down = c.b_down = FAKE
    return s


def test_workspace_bytes_valid_and_monotone(L):
    s = _tree()
    sizes = [L.lx_moe_tree_workspace_bytes(ctypes.byref(s), T, 8) for T in (0, 1, 64, 4096)]
    assert all(n > 0 for n in sizes)
    assert sizes == sorted(sizes) and sizes[3] > sizes[2] > sizes[1]
    # a flat descriptor plans the same workspace as its one-level tree
    f = lx.LxFlatLayer()
    f.E, f.C, f.d, f.f, f.r, f.M, f.dtype = 128, 16, 2048, 768, 64, 112, lx.LX_BF16
    for n in ("cluster_of", "factor_of", "dom_gate", "dom_up", "dom_down", "a_gate", "b_gate",
              "a_up", "b_up", "a_down", "b_down"):
        setattr(f, n, FAKE)
    assert L.lx_moe_workspace_bytes(ctypes.byref(f), 4096, 8) == sizes[3]
    dn = lx.LxDenseLayer()
    dn.E, dn.d, dn.f, dn.dtype = 128, 2048, 768, lx.LX_BF16
    dn.w_gate = dn.w_up = dn.w_down = FAKE
    assert L.lx_dense_moe_workspace_bytes(ctypes.byref(dn), 4096, 8) > 0


@pytest.mark.parametrize("mut,code", [
    (lambda s: setattr(s, "d", 2044), lx.LX_ERR_UNSUPPORTED),          # d % 8
    (lambda s: setattr(s.levels[0], "rank", 60), lx.LX_ERR_UNSUPPORTED),  # bf16 rank % 8
    (lambda s: setattr(s.levels[0], "n_nodes", 127), lx.LX_ERR_INVALID_ARGUMENT),  # last level != E
    (lambda s: setattr(s, "anchor_up", FAKE + 4), lx.LX_ERR_INVALID_ARGUMENT),     # misaligned
    (lambda s: setattr(s.levels[0], "a_down", None), lx.LX_ERR_INVALID_ARGUMENT),  # null factor
    (lambda s: setattr(s, "n_levels", 5), lx.LX_ERR_INVALID_ARGUMENT),
    (lambda s: setattr(s, "E", 9000), lx.LX_ERR_UNSUPPORTED),
    # fp8 down copy: both pointers or neither, aligned, bf16 with f % 64 == 0
    (lambda s: setattr(s, "anchor_down_f8", FAKE), lx.LX_ERR_INVALID_ARGUMENT),
    (lambda s: (setattr(s, "anchor_down_f8", FAKE + 8), setattr(s, "anchor_down_f8_scale", FAKE)),
     lx.LX_ERR_INVALID_ARGUMENT),
    (lambda s: (setattr(s, "anchor_down_f8", FAKE), setattr(s, "anchor_down_f8_scale", FAKE),
                setattr(s, "f", 776)), lx.LX_ERR_UNSUPPORTED),
    (lambda s: (setattr(s, "anchor_down_f8", FAKE), setattr(s, "anchor_down_f8_scale", FAKE),
                setattr(s, "dtype", lx.LX_F32)), lx.LX_ERR_UNSUPPORTED),
])
def test_descriptor_validation(L, mut, code):
    s = _tree()
    mut(s)
    assert L.lx_moe_tree_workspace_bytes(ctypes.byref(s), 64, 8) == 0
    st = L.lx_moe_forward_tree(ctypes.byref(s), 64, 8, FAKE, FAKE, FAKE, FAKE, lx.LX_F32, FAKE,
                               1 << 40, None)
    assert st == code, (lx.status_string(st), L.lx_last_error())
    assert L.lx_last_error().decode()


def test_call_validation(L):
    s = _tree()
    need = L.lx_moe_tree_workspace_bytes(ctypes.byref(s), 64, 8)
    call = lambda T, k, x=FAKE, ids=FAKE, w=FAKE, out=FAKE, od=lx.LX_F32, ws=FAKE, n=need: \
        L.lx_moe_forward_tree(ctypes.byref(s), T, k, x, ids, w, out, od, ws, n, None)
    assert call(64, 0) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(64, 33) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(-1, 8) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(64, 8, x=None) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(64, 8, ids=None) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(64, 8, out=FAKE + 8) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(64, 8, od=7) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(64, 8, ws=None) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(64, 8, n=need - 1) == lx.LX_ERR_WORKSPACE_TOO_SMALL
    assert L.lx_bucket(ctypes.byref(s), 64, 8, FAKE, 2, None, None, None, FAKE, need, None) \
        == lx.LX_ERR_INVALID_ARGUMENT
    assert L.lx_read_device_status(None, None, None) == lx.LX_ERR_INVALID_ARGUMENT


def test_fp8_copy_planned_like_bf16_and_quantize_validation(L):
    s = _tree()
    plain = L.lx_moe_tree_workspace_bytes(ctypes.byref(s), 4096, 8)
    s.anchor_down_f8, s.anchor_down_f8_scale = FAKE, FAKE
    assert L.lx_moe_tree_workspace_bytes(ctypes.byref(s), 4096, 8) == plain
    q = L.lx_quantize_f8
    assert q(FAKE, 2, 8, 96, FAKE, FAKE, None) == lx.LX_ERR_UNSUPPORTED        # cols % 64
    assert q(FAKE, -1, 8, 64, FAKE, FAKE, None) == lx.LX_ERR_INVALID_ARGUMENT
    assert q(None, 2, 8, 64, FAKE, FAKE, None) == lx.LX_ERR_INVALID_ARGUMENT
    assert q(FAKE, 2, 8, 64, FAKE + 4, FAKE, None) == lx.LX_ERR_INVALID_ARGUMENT
    assert q(None, 0, 8, 64, None, None, None) == lx.LX_OK                      # empty: no launch


def test_profile_entries_empty(L):
    assert L.lx_profile_reset() == lx.LX_OK
    assert L.lx_profile_count() == 0
    assert L.lx_profile_entry(0, None, None, None) == lx.LX_ERR_INVALID_ARGUMENT


def test_route_validation(L):
    r = L.lx_route_topk
    need = L.lx_route_workspace_bytes(64, 2048, 128)
    # logits, then the partial tiles of the split logits GEMM: 4 items (two
    # 32-row tiles x two 64-expert tiles) x 8 splits (32 weight slabs / 4)
    assert need == 64 * 128 * 4 + 4 * 8 * 32 * 64 * 4
    # enough items to fill the machine: no split, logits only
    assert L.lx_route_workspace_bytes(32768, 2048, 128) == 32768 * 128 * 4
    assert L.lx_route_workspace_bytes(64, 2000, 128) == 0
    ok = dict(x=FAKE, w=FAKE, dt=lx.LX_BF16, T=64, d=2048, E=128, k=8, ids=FAKE, wt=FAKE, ws=FAKE, n=need)

    def call(**kw):
        a = dict(ok, **kw)
        return r(a["x"], a["w"], a["dt"], a["T"], a["d"], a["E"], a["k"], a["ids"], a["wt"], a["ws"], a["n"], None)
    assert call(dt=lx.LX_F32) == lx.LX_ERR_UNSUPPORTED
    assert call(d=2000) == lx.LX_ERR_UNSUPPORTED           # d % 64
    assert call(E=513) == lx.LX_ERR_UNSUPPORTED
    assert call(E=42) == lx.LX_ERR_UNSUPPORTED             # E % 4
    assert call(n=need - 1) == lx.LX_ERR_WORKSPACE_TOO_SMALL
    assert call(ws=None) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(k=0) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(k=33) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(E=4, k=5) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(T=-1) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(x=None) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(w=FAKE + 8) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(ids=FAKE + 2) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(T=0, x=None, ids=None, ws=None) == lx.LX_OK  # empty: no launch


def test_cluster_validation(L):
    import ctypes as C
    co = L.lx_coact_distance
    assert co(FAKE, 10, 0, 8, FAKE, FAKE, FAKE, None) == lx.LX_ERR_INVALID_ARGUMENT   # k
    assert co(FAKE, 10, 2, 1025, FAKE, FAKE, FAKE, None) == lx.LX_ERR_UNSUPPORTED      # E
    assert co(FAKE, -1, 2, 8, FAKE, FAKE, FAKE, None) == lx.LX_ERR_INVALID_ARGUMENT
    assert co(FAKE, 10, 2, 8, FAKE, FAKE, FAKE + 4, None) == lx.LX_ERR_INVALID_ARGUMENT  # dist 8-aligned
    km = L.lx_kmedoids
    none = (C.c_int32 * 1)(0)

    def call(E=8, Cn=3, prot=(), it=10):
        arr = (C.c_int32 * max(len(prot), 1))(*prot)
        return km(FAKE, FAKE, E, Cn, arr, len(prot), it, FAKE, FAKE, FAKE, FAKE, None)
    assert call(E=0) == lx.LX_ERR_UNSUPPORTED
    assert call(Cn=0) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(Cn=9) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(Cn=2, prot=(1, 2)) == lx.LX_ERR_INVALID_ARGUMENT          # no seeded cluster left
    assert call(prot=(1, 1)) == lx.LX_ERR_INVALID_ARGUMENT                # repeated
    assert call(prot=(8,)) == lx.LX_ERR_INVALID_ARGUMENT                  # out of range
    assert call(it=-1) == lx.LX_ERR_INVALID_ARGUMENT
    assert km(FAKE, FAKE, 8, 3, none, 0, 10, None, FAKE, FAKE, FAKE, None) == lx.LX_ERR_INVALID_ARGUMENT


def test_assign_on_host_matches_brute_force():
    """lx_assign is host code: checked here against every permutation."""
    import itertools
    import numpy as np
    rng = np.random.default_rng(7)
    for n in (1, 3, 6, 8):
        C = rng.random((n, n))
        if n == 6:
            C = np.round(C * 4) / 4              # many ties among optima
        perm, total = lx.assign(C)
        best = min(sum(C[i, p[i]] for i in range(n)) for p in itertools.permutations(range(n)))
        assert sorted(perm.tolist()) == list(range(n))
        assert abs(total - best) < 1e-12 and abs(total - C[np.arange(n), perm].sum()) < 1e-12
    perm, total = lx.assign(np.zeros((0, 0)))
    assert perm.size == 0 and total == 0.0


def test_stage3_validation(L):
    need = L.lx_align_workspace_bytes(768, 2048)
    assert need == 2 * 768 * (3 * 2048 + 1) * 8
    args = [FAKE] * 6
    assert L.lx_align_cost(*args, lx.LX_BF16, 768, 2048, FAKE, FAKE, need - 1, None) == lx.LX_ERR_WORKSPACE_TOO_SMALL
    assert L.lx_align_cost(*args, 7, 768, 2048, FAKE, FAKE, need, None) == lx.LX_ERR_INVALID_ARGUMENT
    assert L.lx_align_cost(FAKE + 1, *args[1:], lx.LX_BF16, 768, 2048, FAKE, FAKE, need, None) \
        == lx.LX_ERR_INVALID_ARGUMENT
    assert L.lx_lowrank_workspace_bytes(768, 2048, 120, 10) == 0          # r + p > 128
    n = L.lx_lowrank_workspace_bytes(768, 2048, 64, 10)
    lr = L.lx_lowrank_factors
    base = dict(t=lx.LX_BF16, rows=768, cols=2048, perm=None, ax=0, r=64, p=10, q=2, n=n)

    def call(**kw):
        a = dict(base, **kw)
        return lr(FAKE, FAKE, a["t"], a["rows"], a["cols"], a["perm"], a["ax"], a["r"], a["p"], a["q"], FAKE, FAKE,
                  FAKE, FAKE, FAKE, a["n"], None)
    assert call(r=120) == lx.LX_ERR_UNSUPPORTED
    assert call(rows=50) == lx.LX_ERR_UNSUPPORTED                          # r + p > rows
    assert call(q=-1) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(ax=2) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(n=n - 1) == lx.LX_ERR_WORKSPACE_TOO_SMALL
    assert call(perm=FAKE + 2) == lx.LX_ERR_INVALID_ARGUMENT


def test_weighted_fit_validation(L):
    """Host-side checks of lx_weighted_factors (no kernel is launched)."""
    ws = L.lx_weighted_workspace_bytes
    assert ws(768, 2048, 512, 0, 120, 10) == 0                  # r + p > 128
    assert ws(768, 2048, 40, 0, 64, 10) == 0                    # r + p > activation rows
    assert ws(768, 2048, 40, 1, 64, 10) > 0                     # damping adds cols rows
    assert ws(768, 2048, 4096, 1, 64, 10) > ws(768, 2048, 4096, 0, 64, 10)
    n = ws(768, 2048, 512, 0, 64, 10)
    base = dict(t=lx.LX_BF16, xt=lx.LX_BF16, rows=768, cols=2048, n_act=512, damp=0.0, r=64, p=10, q=2, n=n,
                x=FAKE, ax=0)

    def call(**kw):
        a = dict(base, **kw)
        return L.lx_weighted_factors(FAKE, FAKE, a["t"], a["rows"], a["cols"], None, a["ax"], a["x"], a["xt"],
                                     a["n_act"], a["damp"], a["r"], a["p"], a["q"], FAKE, FAKE, FAKE, FAKE, FAKE,
                                     a["n"], None)
    assert call(damp=-1.0) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(damp=float("nan")) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(damp=float("inf")) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(xt=7) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(n_act=-1) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(n_act=40) == lx.LX_ERR_UNSUPPORTED                 # r + p > n'
    assert call(x=None) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(x=FAKE + 1) == lx.LX_ERR_INVALID_ARGUMENT          # misaligned bf16
    assert call(ax=3) == lx.LX_ERR_INVALID_ARGUMENT
    assert call(n=n - 1) == lx.LX_ERR_WORKSPACE_TOO_SMALL
    # damping: the same call needs the larger workspace
    assert call(damp=0.1) == lx.LX_ERR_WORKSPACE_TOO_SMALL


def test_binding_error_paths_raise_lorex_error(L):
    """The binding's own shape checks raise LorexError with a status (no kernel
    is launched: every shape below is refused by a workspace-size query)."""
    import torch
    with pytest.raises(lx.LorexError) as e:
        lx.route_workspace(16, 100, 128, device="cpu")              # d not a multiple of 64
    assert e.value.status == lx.LX_ERR_UNSUPPORTED and "router shape" in str(e.value)
    with pytest.raises(lx.LorexError) as e:
        lx.route_workspace(16, 2048, 6, device="cpu")               # E not a multiple of 4
    assert e.value.status == lx.LX_ERR_UNSUPPORTED
    w = torch.zeros(200, 200, dtype=torch.float32)
    with pytest.raises(lx.LorexError) as e:                        # r + p > 128
        lx.lowrank_factors(w, w, 120, torch.zeros(200, 130, dtype=torch.float64))
    assert e.value.status == lx.LX_ERR_UNSUPPORTED and "lx_lowrank_factors" in str(e.value)
    x = torch.zeros(300, 200, dtype=torch.float32)
    with pytest.raises(lx.LorexError) as e:                        # r + p > 128
        lx.weighted_factors(w, w, 120, x, torch.zeros(300, 130, dtype=torch.float64))
    assert e.value.status == lx.LX_ERR_UNSUPPORTED and "lx_weighted_factors" in str(e.value)
    with pytest.raises(lx.LorexError) as e:                        # r + p > activation rows
        lx.weighted_factors(w, w, 60, x[:50], torch.zeros(50, 70, dtype=torch.float64))
    assert e.value.status == lx.LX_ERR_UNSUPPORTED


def test_aux_stream_switch(L):
    """lx_set_aux_stream is a plain process-wide switch that returns the
    previous setting (off by default) and touches no device."""
    assert lx.set_aux_stream(False) is False
    assert L.lx_set_aux_stream(7) == 0          # any non-zero value enables
    assert lx.set_aux_stream(True) is True
    assert lx.set_aux_stream(False) is True
    assert lx.set_aux_stream(False) is False


def test_static_forward_refuses_batches_beyond_its_scratch(L):
    """lx_moe_forward_tree_static: a batch whose workspace exceeds the static
    scratch is refused on the host, before any device call (T = 4096 at the
    30B-A3B shape needs about 1.1 GB); invalid arguments likewise."""
    s = _tree()
    assert L.lx_moe_tree_workspace_bytes(ctypes.byref(s), 4096, 8) > lx.STATIC_SCRATCH_BYTES
    st = L.lx_moe_forward_tree_static(ctypes.byref(s), 4096, 8, FAKE, FAKE, FAKE, FAKE, lx.LX_F32, None)
    assert st == lx.LX_ERR_WORKSPACE_TOO_SMALL
    msg = L.lx_last_error().decode()
    assert "static scratch" in msg and str(lx.STATIC_SCRATCH_BYTES) in msg
    assert L.lx_moe_forward_tree_static(None, 4, 8, FAKE, FAKE, FAKE, FAKE, lx.LX_F32, None) == \
        lx.LX_ERR_INVALID_ARGUMENT
    assert L.lx_moe_forward_tree_static(ctypes.byref(s), 4, 0, FAKE, FAKE, FAKE, FAKE, lx.LX_F32, None) == \
        lx.LX_ERR_INVALID_ARGUMENT
    assert L.lx_moe_tree_workspace_bytes(ctypes.byref(s), 64, 8) <= lx.STATIC_SCRATCH_BYTES


def test_convert_f16_validation(L):
    assert L.lx_convert_f16(FAKE, 0, 4, 4, FAKE, FAKE, None) == lx.LX_ERR_INVALID_ARGUMENT
    assert L.lx_convert_f16(FAKE, 1, 4, 4, FAKE + 8, FAKE, None) == lx.LX_ERR_INVALID_ARGUMENT  # w_f16 % 16
    assert L.lx_convert_f16(None, 1, 4, 4, FAKE, FAKE, None) == lx.LX_ERR_INVALID_ARGUMENT
    # a layer whose fp16 down copy lacks its exponents is refused
    s = _tree()
    s.anchor_down_f16 = FAKE
    assert L.lx_moe_tree_workspace_bytes(ctypes.byref(s), 64, 8) == 0
    s.anchor_down_f16_exp = FAKE
    assert L.lx_moe_tree_workspace_bytes(ctypes.byref(s), 64, 8) > 0


def test_factor_f16_copies_validation(L):
    """The fp16 factor copies of a level come as all eight arrays or none,
    aligned, and only in bf16 layers (checked on the host, no device access);
    the flat layer carries them the same way."""
    s = _tree()
    lv = s.levels[0]
    names = lx.FACTOR_F16
    lv.a_gate_f16 = FAKE
    assert L.lx_moe_tree_workspace_bytes(ctypes.byref(s), 64, 8) == 0
    assert "fp16 factor copies" in L.lx_last_error().decode()
    for n in names:
        setattr(lv, n, FAKE)
    assert L.lx_moe_tree_workspace_bytes(ctypes.byref(s), 64, 8) > 0
    lv.b_down_f16 = FAKE + 8  # not 16-byte aligned
    assert L.lx_moe_tree_workspace_bytes(ctypes.byref(s), 64, 8) == 0
    lv.b_down_f16 = FAKE
    s.dtype = lx.LX_F32
    assert L.lx_moe_tree_workspace_bytes(ctypes.byref(s), 64, 8) == 0
    f = lx.LxFlatLayer()
    f.E, f.C, f.d, f.f, f.r, f.M, f.dtype = 128, 16, 2048, 768, 64, 112, lx.LX_BF16
    for n in ("cluster_of", "factor_of", "dom_gate", "dom_up", "dom_down", "a_gate", "b_gate",
              "a_up", "b_up", "a_down", "b_down"):
        setattr(f, n, FAKE)
    f.a_down_f16 = FAKE
    assert L.lx_moe_workspace_bytes(ctypes.byref(f), 64, 8) == 0
    for n in names:
        setattr(f, n, FAKE)
    assert L.lx_moe_workspace_bytes(ctypes.byref(f), 64, 8) > 0


def test_padded_rank_validation(L):
    """rank_f16 (the padded rank of a level's fp16 copies): 0, or a multiple
    of 64 in [rank, 128], only with the fp16 copies, and above the rank only
    with both zero-padded bf16 input factors (checked on the host); the flat
    layer carries it as r_f16; the padded-copy entry points check their
    sizes and pointers."""
    s = _tree(r=96)
    lv = s.levels[0]
    for n in lx.FACTOR_F16:
        setattr(lv, n, FAKE)
    assert L.lx_moe_tree_workspace_bytes(ctypes.byref(s), 64, 8) > 0
    for bad in (100, 64, 192):  # not a multiple of 64, below the rank, above 128
        lv.rank_f16 = bad
        assert L.lx_moe_tree_workspace_bytes(ctypes.byref(s), 64, 8) == 0
        assert "multiple of 64" in L.lx_last_error().decode()
    lv.rank_f16 = 128
    assert L.lx_moe_tree_workspace_bytes(ctypes.byref(s), 64, 8) == 0
    assert "b_gate_pad" in L.lx_last_error().decode()
    lv.b_gate_pad = FAKE
    lv.b_up_pad = FAKE + 8  # not 16-byte aligned
    assert L.lx_moe_tree_workspace_bytes(ctypes.byref(s), 64, 8) == 0
    lv.b_up_pad = FAKE
    assert L.lx_moe_tree_workspace_bytes(ctypes.byref(s), 64, 8) > 0
    for n in lx.FACTOR_F16:
        setattr(lv, n, None)
    assert L.lx_moe_tree_workspace_bytes(ctypes.byref(s), 64, 8) == 0
    assert "without fp16 factor copies" in L.lx_last_error().decode()
    f = lx.LxFlatLayer()
    f.E, f.C, f.d, f.f, f.r, f.M, f.dtype = 128, 16, 2048, 768, 96, 112, lx.LX_BF16
    for n in ("cluster_of", "factor_of", "dom_gate", "dom_up", "dom_down", "a_gate", "b_gate",
              "a_up", "b_up", "a_down", "b_down") + lx.FACTOR_F16:
        setattr(f, n, FAKE)
    f.r_f16 = 128
    assert L.lx_moe_workspace_bytes(ctypes.byref(f), 64, 8) == 0
    f.b_gate_pad = f.b_up_pad = FAKE
    assert L.lx_moe_workspace_bytes(ctypes.byref(f), 64, 8) > 0
    # entry points: sizes and pointers (no device work is queued)
    E = lx.LX_ERR_INVALID_ARGUMENT
    assert L.lx_convert_f16_padded(FAKE, 1, 96, 64, 64, 64, FAKE, FAKE, None) == E  # rows_out < rows
    assert L.lx_convert_f16_padded(FAKE, 1, 96, 64, 128, 32, FAKE, FAKE, None) == E  # cols_out < cols
    assert L.lx_convert_f16_padded(None, 1, 96, 64, 128, 64, FAKE, FAKE, None) == E
    assert L.lx_convert_f16_padded(FAKE, 1, 96, 64, 128, 64, FAKE + 8, FAKE, None) == E
    assert L.lx_pad_bf16(FAKE, 0, 96, 64, 128, 64, FAKE, None) == E
    assert L.lx_pad_bf16(FAKE, 1, 96, 64, 128, 64, None, None) == E
    assert L.lx_pad_bf16(FAKE, 1, 96, 64, 128, 64, FAKE + 8, None) == E

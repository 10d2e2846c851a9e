"""lx_moe_forward_tree_static (no allocation, static per-GPU scratch) against
lx_moe_forward_tree with a caller workspace: two calls in a row on the static
scratch, the second with a smaller batch, each equal to the workspace entry
point's output (same kernels and launch plan: bitwise), which itself meets the
oracle bar in the forward tests."""
import numpy as np
import pytest
import torch

from lxsynth import make_problem
from oracle import moe as O
from paper_2608_07814_amd import lorex as lx
from gpu_util import TOL_BF16, require_gpu, say, dev_inputs, err_ratio

pytestmark = pytest.mark.gpu


def _inputs(p, T):
    xt, ids, w = dev_inputs(p)
    return xt[:T].contiguous(), ids[:T].contiguous(), w[:T].contiguous()


@pytest.mark.parametrize("cfg,T1,T2", [(2, 64, 23), (4, 48, 9)])
def test_static_scratch_matches_workspace_entry_point(cfg, T1, T2):
    require_gpu()
    p = make_problem(cfg, T=T1)
    dl = lx.to_device(p.layer)
    for T in (T1, T2):
        say(f"static scratch cfg{cfg} T={T}")
        x, ids, w = _inputs(p, T)
        ref = lx.forward(dl, x, ids, w, kind="tree")
        out = torch.full((T, p.layer.d), float("nan"), dtype=torch.float32, device="cuda")
        torch.cuda.synchronize()
        before = torch.cuda.memory_allocated()
        lx.forward_static(dl, x, ids, w, out)
        torch.cuda.synchronize()
        assert torch.cuda.memory_allocated() == before
        got, want = out.cpu().numpy(), ref.cpu().numpy()
        assert np.all(np.isfinite(got))
        assert np.array_equal(got, want), f"max |diff| {np.max(np.abs(got - want))}"
        # and the bar of the parity tests against the oracle
        orc = O.moe_forward(p.layer, p.x[:T], p.routing.topk_ids[:T], p.routing.topk_weights[:T])
        e = err_ratio(got.astype(np.float64), orc)
        say(f"  err/RMS = {e:.3e}")
        assert e <= TOL_BF16


def test_static_scratch_refuses_large_batch():
    require_gpu()
    p = make_problem(1, T=512)
    dl = lx.to_device(p.layer)
    x, ids, w = _inputs(p, 512)
    out = torch.empty(512, p.layer.d, dtype=torch.float32, device="cuda")
    with pytest.raises(lx.LorexError) as e:
        lx.forward_static(dl, x, ids, w, out)
    assert e.value.status == lx.LX_ERR_WORKSPACE_TOO_SMALL

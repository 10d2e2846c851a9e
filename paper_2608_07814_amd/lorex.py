"""Thin Python binding of liblorex.so (ctypes): argument marshalling only.

Every step of the forward runs in the library's HIP kernels; torch is used for
device memory (tensors whose ``data_ptr()`` is passed down) and for the
current stream. The library is loaded on first use; a missing library raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field
from typing import Optional

import numpy as np
import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "liblorex.so")

LX_OK, LX_ERR_INVALID_ARGUMENT, LX_ERR_UNSUPPORTED, LX_ERR_WORKSPACE_TOO_SMALL, LX_ERR_HIP = range(5)
LX_F32, LX_BF16 = 0, 1
LX_MAX_LEVELS = 4
LX_MAX_K = 32
LX_MAX_NODES = 8192
LX_DEVFLAG_BAD_ID = 1
LX_DEVFLAG_BAD_TREE = 2

_c_void = ctypes.c_void_p
_c_i32 = ctypes.c_int32


class LxLevel(ctypes.Structure):
    _fields_ = [("n_nodes", _c_i32), ("rank", _c_i32), ("n_factors", _c_i32),
                ("parent", _c_void), ("factor_of", _c_void),
                ("a_gate", _c_void), ("b_gate", _c_void), ("a_up", _c_void), ("b_up", _c_void),
                ("a_down", _c_void), ("b_down", _c_void),
                ("a_gate_f16", _c_void), ("a_gate_f16_exp", _c_void), ("a_up_f16", _c_void),
                ("a_up_f16_exp", _c_void), ("a_down_f16", _c_void), ("a_down_f16_exp", _c_void),
                ("b_down_f16", _c_void), ("b_down_f16_exp", _c_void),
                ("rank_f16", _c_i32), ("b_gate_pad", _c_void), ("b_up_pad", _c_void)]

# the optional fp16 factor copies of a level (lx_convert_f16), with exponents
FACTOR_F16 = ("a_gate_f16", "a_gate_f16_exp", "a_up_f16", "a_up_f16_exp", "a_down_f16", "a_down_f16_exp",
              "b_down_f16", "b_down_f16_exp")
# the zero-padded bf16 input factors that go with copies of a padded rank
FACTOR_PAD = ("b_gate_pad", "b_up_pad")


class LxTreeLayer(ctypes.Structure):
    _fields_ = [("E", _c_i32), ("d", _c_i32), ("f", _c_i32), ("dtype", _c_i32),
                ("n_anchors", _c_i32), ("anchor_gate", _c_void), ("anchor_up", _c_void),
                ("anchor_down", _c_void), ("n_levels", _c_i32),
                ("levels", LxLevel * LX_MAX_LEVELS),
                ("anchor_down_f8", _c_void), ("anchor_down_f8_scale", _c_void),
                ("anchor_down_f16", _c_void), ("anchor_down_f16_exp", _c_void)]


class LxFlatLayer(ctypes.Structure):
    _fields_ = [("E", _c_i32), ("C", _c_i32), ("d", _c_i32), ("f", _c_i32), ("r", _c_i32),
                ("M", _c_i32), ("dtype", _c_i32), ("cluster_of", _c_void), ("factor_of", _c_void),
                ("dom_gate", _c_void), ("dom_up", _c_void), ("dom_down", _c_void),
                ("a_gate", _c_void), ("b_gate", _c_void), ("a_up", _c_void), ("b_up", _c_void),
                ("a_down", _c_void), ("b_down", _c_void),
                ("dom_down_f8", _c_void), ("dom_down_f8_scale", _c_void),
                ("dom_down_f16", _c_void), ("dom_down_f16_exp", _c_void),
                ("a_gate_f16", _c_void), ("a_gate_f16_exp", _c_void), ("a_up_f16", _c_void),
                ("a_up_f16_exp", _c_void), ("a_down_f16", _c_void), ("a_down_f16_exp", _c_void),
                ("b_down_f16", _c_void), ("b_down_f16_exp", _c_void),
                ("r_f16", _c_i32), ("b_gate_pad", _c_void), ("b_up_pad", _c_void)]


class LxDenseLayer(ctypes.Structure):
    _fields_ = [("E", _c_i32), ("d", _c_i32), ("f", _c_i32), ("dtype", _c_i32),
                ("w_gate", _c_void), ("w_up", _c_void), ("w_down", _c_void),
                ("w_down_f8", _c_void), ("w_down_f8_scale", _c_void),
                ("w_down_f16", _c_void), ("w_down_f16_exp", _c_void)]


EXPORTS = {
    "lx_status_string": (ctypes.c_char_p, [_c_i32]),
    "lx_last_error": (ctypes.c_char_p, []),
    "lx_version": (_c_i32, []),
    "lx_set_aux_stream": (_c_i32, [_c_i32]),
    "lx_moe_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(LxFlatLayer), _c_i32, _c_i32]),
    "lx_moe_tree_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(LxTreeLayer), _c_i32, _c_i32]),
    "lx_dense_moe_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(LxDenseLayer), _c_i32, _c_i32]),
    "lx_moe_forward": (_c_i32, [ctypes.POINTER(LxFlatLayer), _c_i32, _c_i32, _c_void, _c_void, _c_void,
                                _c_void, _c_i32, _c_void, ctypes.c_size_t, _c_void]),
    "lx_moe_forward_tree": (_c_i32, [ctypes.POINTER(LxTreeLayer), _c_i32, _c_i32, _c_void, _c_void,
                                     _c_void, _c_void, _c_i32, _c_void, ctypes.c_size_t, _c_void]),
    "lx_route_moe_tree_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(LxTreeLayer), _c_i32, _c_i32]),
    "lx_route_moe_forward_tree": (_c_i32, [ctypes.POINTER(LxTreeLayer), _c_i32, _c_i32, _c_void, _c_void, _c_void,
                                           _c_void, _c_void, _c_i32, _c_void, ctypes.c_size_t, _c_void]),
    "lx_moe_forward_tree_static": (_c_i32, [ctypes.POINTER(LxTreeLayer), _c_i32, _c_i32, _c_void, _c_void,
                                            _c_void, _c_void, _c_i32, _c_void]),
    "lx_dense_moe_forward": (_c_i32, [ctypes.POINTER(LxDenseLayer), _c_i32, _c_i32, _c_void, _c_void,
                                      _c_void, _c_void, _c_i32, _c_void, ctypes.c_size_t, _c_void]),
    "lx_bucket": (_c_i32, [ctypes.POINTER(LxTreeLayer), _c_i32, _c_i32, _c_void, _c_i32, _c_void,
                           _c_void, _c_void, _c_void, ctypes.c_size_t, _c_void]),
    "lx_read_device_status": (_c_i32, [_c_void, _c_void, ctypes.POINTER(ctypes.c_uint32)]),
    "lx_convert_f16": (_c_i32, [_c_void, _c_i32, _c_i32, _c_i32, _c_void, _c_void, _c_void]),
    "lx_convert_f16_padded": (_c_i32, [_c_void, _c_i32, _c_i32, _c_i32, _c_i32, _c_i32, _c_void, _c_void, _c_void]),
    "lx_pad_bf16": (_c_i32, [_c_void, _c_i32, _c_i32, _c_i32, _c_i32, _c_i32, _c_void, _c_void]),
    "lx_quantize_f8": (_c_i32, [_c_void, _c_i32, _c_i32, _c_i32, _c_void, _c_void, _c_void]),
    "lx_route_workspace_bytes": (ctypes.c_size_t, [_c_i32, _c_i32, _c_i32]),
    "lx_coact_distance": (_c_i32, [_c_void, _c_i32, _c_i32, _c_i32, _c_void, _c_void, _c_void, _c_void]),
    "lx_kmedoids": (_c_i32, [_c_void, _c_void, _c_i32, _c_i32, ctypes.POINTER(ctypes.c_int32), _c_i32, _c_i32,
                             _c_void, _c_void, _c_void, _c_void, _c_void]),
    "lx_align_workspace_bytes": (ctypes.c_size_t, [_c_i32, _c_i32]),
    "lx_align_cost": (_c_i32, [_c_void] * 6 + [_c_i32, _c_i32, _c_i32, _c_void, _c_void, ctypes.c_size_t, _c_void]),
    "lx_assign": (_c_i32, [_c_void, _c_i32, _c_void, _c_void]),
    "lx_lowrank_workspace_bytes": (ctypes.c_size_t, [_c_i32, _c_i32, _c_i32, _c_i32]),
    "lx_lowrank_factors": (_c_i32, [_c_void, _c_void, _c_i32, _c_i32, _c_i32, _c_void, _c_i32, _c_i32, _c_i32,
                                    _c_i32, _c_void, _c_void, _c_void, _c_void, _c_void, ctypes.c_size_t, _c_void]),
    "lx_weighted_workspace_bytes": (ctypes.c_size_t, [_c_i32] * 6),
    "lx_weighted_factors": (_c_i32, [_c_void, _c_void, _c_i32, _c_i32, _c_i32, _c_void, _c_i32, _c_void, _c_i32,
                                     _c_i32, ctypes.c_double, _c_i32, _c_i32, _c_i32, _c_void, _c_void, _c_void,
                                     _c_void, _c_void, ctypes.c_size_t, _c_void]),
    "lx_route_topk": (_c_i32, [_c_void, _c_void, _c_i32, _c_i32, _c_i32, _c_i32, _c_i32, _c_void, _c_void,
                               _c_void, ctypes.c_size_t, _c_void]),
    "lx_profile_enable": (_c_i32, [_c_i32]),
    "lx_profile_collect": (_c_i32, []),
    "lx_profile_count": (_c_i32, []),
    "lx_profile_entry": (_c_i32, [_c_i32, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_int64),
                                  ctypes.POINTER(ctypes.c_double)]),
    "lx_profile_reset": (_c_i32, []),
}

_LIB: Optional[ctypes.CDLL] = None


class LorexError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{status_string(status)}: {msg}")
        self.status = status


def lib() -> ctypes.CDLL:
    """Load liblorex.so (once). Raises if it has not been built."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2608_07814_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in EXPORTS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = L
    return _LIB


def status_string(s: int) -> str:
    return lib().lx_status_string(s).decode()


def _check(status: int):
    if status != LX_OK:
        raise LorexError(status, lib().lx_last_error().decode())


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream=None) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


# ----------------------------------------------------------- device layers
def _dev_array(a, dtype: str, device) -> torch.Tensor:
    """numpy host array (bf16 bits as uint16, fp32, int32) -> device tensor."""
    if isinstance(a, torch.Tensor):
        return a.to(device).contiguous()
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(a).to(device)


@dataclass
class DeviceLevel:
    parent: torch.Tensor
    factor_of: torch.Tensor
    rank: int
    a_gate: torch.Tensor
    b_gate: torch.Tensor
    a_up: torch.Tensor
    b_up: torch.Tensor
    a_down: torch.Tensor
    b_down: torch.Tensor
    # optional fp16 copies of the factors (lx_convert_f16): fp16 tensors of
    # the same shapes and int32 exponents [n_factors]
    a_gate_f16: Optional[torch.Tensor] = None
    a_gate_f16_exp: Optional[torch.Tensor] = None
    a_up_f16: Optional[torch.Tensor] = None
    a_up_f16_exp: Optional[torch.Tensor] = None
    a_down_f16: Optional[torch.Tensor] = None
    a_down_f16_exp: Optional[torch.Tensor] = None
    b_down_f16: Optional[torch.Tensor] = None
    b_down_f16_exp: Optional[torch.Tensor] = None
    # rank of the fp16 copies when padded to a multiple of 64 (0: rank), with
    # the zero-padded bf16 b_gate / b_up [n_factors][rank_f16][d]
    rank_f16: int = 0
    b_gate_pad: Optional[torch.Tensor] = None
    b_up_pad: Optional[torch.Tensor] = None

    @property
    def n_nodes(self) -> int:
        return int(self.parent.shape[0])

    @property
    def n_factors(self) -> int:
        return int(self.a_gate.shape[0])


@dataclass
class DeviceLayer:
    """A layer's arrays in device memory plus the C descriptor that points at them."""
    E: int
    d: int
    f: int
    dtype: str
    anchor_gate: torch.Tensor
    anchor_up: torch.Tensor
    anchor_down: torch.Tensor
    levels: list = field(default_factory=list)
    # optional fp8 copy of anchor_down (lx_quantize_f8): uint8 [n][d][f] and
    # int32 scale words [n][d][f // 64]
    anchor_down_f8: Optional[torch.Tensor] = None
    anchor_down_f8_scale: Optional[torch.Tensor] = None
    # optional fp16 copy of anchor_down (lx_convert_f16): fp16 [n][d][f] and
    # int32 scale exponents [n]
    anchor_down_f16: Optional[torch.Tensor] = None
    anchor_down_f16_exp: Optional[torch.Tensor] = None

    @property
    def lx_dtype(self) -> int:
        return LX_BF16 if self.dtype == "bf16" else LX_F32

    @property
    def n_anchors(self) -> int:
        return int(self.anchor_gate.shape[0])

    def tree_struct(self) -> LxTreeLayer:
        s = LxTreeLayer()
        s.E, s.d, s.f, s.dtype = self.E, self.d, self.f, self.lx_dtype
        s.n_anchors = self.n_anchors
        s.anchor_gate, s.anchor_up, s.anchor_down = (_ptr(self.anchor_gate), _ptr(self.anchor_up),
                                                     _ptr(self.anchor_down))
        s.anchor_down_f8, s.anchor_down_f8_scale = _ptr(self.anchor_down_f8), _ptr(self.anchor_down_f8_scale)
        s.anchor_down_f16, s.anchor_down_f16_exp = _ptr(self.anchor_down_f16), _ptr(self.anchor_down_f16_exp)
        s.n_levels = len(self.levels)
        for i, lv in enumerate(self.levels):
            c = s.levels[i]
            c.n_nodes, c.rank, c.n_factors = lv.n_nodes, lv.rank, lv.n_factors
            c.parent, c.factor_of = _ptr(lv.parent), _ptr(lv.factor_of)
            c.a_gate, c.b_gate, c.a_up, c.b_up, c.a_down, c.b_down = (
                _ptr(lv.a_gate), _ptr(lv.b_gate), _ptr(lv.a_up), _ptr(lv.b_up),
                _ptr(lv.a_down), _ptr(lv.b_down))
            for n in FACTOR_F16 + FACTOR_PAD:
                setattr(c, n, _ptr(getattr(lv, n)))
            c.rank_f16 = lv.rank_f16
        return s

    def flat_struct(self) -> LxFlatLayer:
        if len(self.levels) != 1:
            raise ValueError("a flat layer has exactly one correction level")
        lv = self.levels[0]
        s = LxFlatLayer()
        s.E, s.C, s.d, s.f, s.r, s.M, s.dtype = (self.E, self.n_anchors, self.d, self.f, lv.rank,
                                                 lv.n_factors, self.lx_dtype)
        s.cluster_of, s.factor_of = _ptr(lv.parent), _ptr(lv.factor_of)
        s.dom_gate, s.dom_up, s.dom_down = (_ptr(self.anchor_gate), _ptr(self.anchor_up),
                                            _ptr(self.anchor_down))
        s.dom_down_f8, s.dom_down_f8_scale = _ptr(self.anchor_down_f8), _ptr(self.anchor_down_f8_scale)
        s.dom_down_f16, s.dom_down_f16_exp = _ptr(self.anchor_down_f16), _ptr(self.anchor_down_f16_exp)
        s.a_gate, s.b_gate, s.a_up, s.b_up, s.a_down, s.b_down = (
            _ptr(lv.a_gate), _ptr(lv.b_gate), _ptr(lv.a_up), _ptr(lv.b_up), _ptr(lv.a_down),
            _ptr(lv.b_down))
        for n in FACTOR_F16 + FACTOR_PAD:
            setattr(s, n, _ptr(getattr(lv, n)))
        s.r_f16 = lv.rank_f16
        return s

    def dense_struct(self) -> LxDenseLayer:
        if self.levels:
            raise ValueError("a dense layer has no correction levels")
        s = LxDenseLayer()
        s.E, s.d, s.f, s.dtype = self.E, self.d, self.f, self.lx_dtype
        s.w_gate, s.w_up, s.w_down = _ptr(self.anchor_gate), _ptr(self.anchor_up), _ptr(self.anchor_down)
        s.w_down_f8, s.w_down_f8_scale = _ptr(self.anchor_down_f8), _ptr(self.anchor_down_f8_scale)
        s.w_down_f16, s.w_down_f16_exp = _ptr(self.anchor_down_f16), _ptr(self.anchor_down_f16_exp)
        return s


def quantize_f8(w: torch.Tensor, stream=None):
    """fp8 copy of bf16 weights [n][rows][cols] (lx_quantize_f8): returns
    (uint8 [n][rows][cols], int32 scale words [n][rows][cols // 64])."""
    if w.dtype != torch.bfloat16 or not w.is_contiguous() or w.dim() != 3:
        raise ValueError("w must be a contiguous bf16 [n][rows][cols] tensor")
    n, rows, cols = (int(v) for v in w.shape)
    w8 = torch.empty(n, rows, cols, dtype=torch.uint8, device=w.device)
    sc = torch.empty(n, rows, max(cols // 64, 1), dtype=torch.int32, device=w.device)
    _check(lib().lx_quantize_f8(_ptr(w), n, rows, cols, _ptr(w8), _ptr(sc), _stream(stream)))
    return w8, sc


def route_workspace(T: int, d: int, E: int, device="cuda") -> torch.Tensor:
    n = int(lib().lx_route_workspace_bytes(T, d, E))
    if n == 0:
        raise LorexError(LX_ERR_UNSUPPORTED, f"unsupported router shape T={T} d={d} E={E}")
    return torch.empty(n, dtype=torch.uint8, device=device)


def route_topk(x: torch.Tensor, w_r: torch.Tensor, k: int, ids: Optional[torch.Tensor] = None,
               weights: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None, stream=None):
    """The top-k router on the GPU (lx_route_topk): bf16 x [T][d] and router
    weights [E][d] -> (int32 ids [T][k], fp32 weights [T][k]), ready for
    ``forward`` on the same stream."""
    if x.dtype != torch.bfloat16 or w_r.dtype != torch.bfloat16:
        raise ValueError("x and w_r must be bf16")
    if not (x.is_contiguous() and w_r.is_contiguous()) or x.dim() != 2 or w_r.dim() != 2:
        raise ValueError("x [T][d] and w_r [E][d] must be contiguous 2-d tensors")
    T, d = (int(v) for v in x.shape)
    E = int(w_r.shape[0])
    if int(w_r.shape[1]) != d:
        raise ValueError("w_r must be [E][d]")
    if ids is None:
        ids = torch.empty(T, k, dtype=torch.int32, device=x.device)
    if weights is None:
        weights = torch.empty(T, k, dtype=torch.float32, device=x.device)
    if workspace is None:
        workspace = route_workspace(T, d, E, x.device)
    _check(lib().lx_route_topk(_ptr(x), _ptr(w_r), LX_BF16, T, d, E, k, _ptr(ids), _ptr(weights),
                               _ptr(workspace), workspace.numel(), _stream(stream)))
    return ids, weights


def coact_distance(topk_ids: torch.Tensor, E: int, stream=None):
    """Router profiling counts and the Coact-NPMI distance (lx_coact_distance):
    int32 ids [N][k] on the device -> (fire uint32-as-int32 [E], pair [E][E],
    dist fp64 [E][E])."""
    if topk_ids.dtype != torch.int32 or topk_ids.dim() != 2 or not topk_ids.is_contiguous():
        raise ValueError("topk_ids must be a contiguous int32 [N][k] tensor")
    N, k = (int(v) for v in topk_ids.shape)
    dev = topk_ids.device
    fire = torch.empty(E, dtype=torch.int32, device=dev)
    pair = torch.empty(E, E, dtype=torch.int32, device=dev)
    dist = torch.empty(E, E, dtype=torch.float64, device=dev)
    _check(lib().lx_coact_distance(_ptr(topk_ids), N, k, E, _ptr(fire), _ptr(pair), _ptr(dist), _stream(stream)))
    return fire, pair, dist


def kmedoids(dist: torch.Tensor, fire: torch.Tensor, C: int, protected=(), max_iter: int = 100, stream=None):
    """Frequency-seeded k-medoids and dominants (lx_kmedoids) -> (cluster_of,
    factor_of, dominant, iterations) int32 device tensors."""
    if dist.dtype != torch.float64 or not dist.is_contiguous() or dist.dim() != 2:
        raise ValueError("dist must be a contiguous fp64 [E][E] tensor")
    E = int(dist.shape[0])
    dev = dist.device
    cl = torch.empty(E, dtype=torch.int32, device=dev)
    fo = torch.empty(E, dtype=torch.int32, device=dev)
    dom = torch.empty(max(C, 1), dtype=torch.int32, device=dev)
    it = torch.empty(1, dtype=torch.int32, device=dev)
    prot = (ctypes.c_int32 * max(len(protected), 1))(*[int(p) for p in protected])
    _check(lib().lx_kmedoids(_ptr(dist), _ptr(fire), E, C, prot, len(protected), max_iter, _ptr(cl), _ptr(fo),
                             _ptr(dom), _ptr(it), _stream(stream)))
    return cl, fo, dom, it


def align_cost(dom, mem, stream=None) -> torch.Tensor:
    """Neuron-alignment cost (lx_align_cost): dom and mem are (gate, up, down)
    device tensors of one dtype -> fp64 [f][f]."""
    g = dom[0]
    f, d = (int(v) for v in g.shape)
    dt = LX_BF16 if g.dtype == torch.bfloat16 else LX_F32
    for t in (*dom, *mem):
        if not t.is_contiguous() or t.dtype != g.dtype:
            raise ValueError("expert tensors must be contiguous and of one dtype")
    cost = torch.empty(f, f, dtype=torch.float64, device=g.device)
    n = int(lib().lx_align_workspace_bytes(f, d))
    ws = torch.empty(n, dtype=torch.uint8, device=g.device)
    _check(lib().lx_align_cost(*[_ptr(t) for t in (*dom, *mem)], dt, f, d, _ptr(cost), _ptr(ws), n,
                               _stream(stream)))
    return cost


def assign(cost) -> tuple:
    """Exact assignment on the host (lx_assign): fp64 numpy [n][n] ->
    (int32 perm [n], total cost)."""
    import numpy as np
    c = np.ascontiguousarray(cost, dtype=np.float64)
    n = int(c.shape[0])
    perm = np.empty(n, np.int32)
    total = ctypes.c_double(0.0)
    _check(lib().lx_assign(c.ctypes.data, n, perm.ctypes.data, ctypes.addressof(total)))
    return perm, total.value


def lowrank_factors(w_dom: torch.Tensor, w_mem: torch.Tensor, r: int, omega: torch.Tensor, q: int = 2,
                    perm: Optional[torch.Tensor] = None, perm_axis: int = 0, stream=None):
    """Rank-r factors of the aligned residual (lx_lowrank_factors) ->
    (A fp32 [rows][r], B fp32 [r][cols], sigma fp64 [r])."""
    rows, cols = (int(v) for v in w_dom.shape)
    p = int(omega.shape[1]) - r
    dt = LX_BF16 if w_dom.dtype == torch.bfloat16 else LX_F32
    if omega.dtype != torch.float64 or not omega.is_contiguous() or int(omega.shape[0]) != cols:
        raise ValueError("omega must be a contiguous fp64 [cols][r + p] tensor")
    dev = w_dom.device
    A = torch.empty(rows, r, dtype=torch.float32, device=dev)
    B = torch.empty(r, cols, dtype=torch.float32, device=dev)
    sig = torch.empty(r, dtype=torch.float64, device=dev)
    n = int(lib().lx_lowrank_workspace_bytes(rows, cols, r, p))
    if n == 0:
        raise LorexError(LX_ERR_UNSUPPORTED, f"unsupported shape for lx_lowrank_factors: rows={rows} cols={cols} r={r} p={p}")
    ws = torch.empty(n, dtype=torch.uint8, device=dev)
    _check(lib().lx_lowrank_factors(_ptr(w_dom), _ptr(w_mem), dt, rows, cols, _ptr(perm) if perm is not None else None,
                                    perm_axis, r, p, q, _ptr(omega), _ptr(A), _ptr(B), _ptr(sig), _ptr(ws), n,
                                    _stream(stream)))
    return A, B, sig


def weighted_factors(w_dom: torch.Tensor, w_mem: torch.Tensor, r: int, x: torch.Tensor, omega: torch.Tensor,
                     q: int = 2, damp: float = 0.0, perm: Optional[torch.Tensor] = None, perm_axis: int = 0,
                     stream=None):
    """Activation-weighted rank-r factors of the aligned residual on
    calibration activations x [n][cols] (lx_weighted_factors) ->
    (A fp32 [rows][r], B fp32 [r][cols], sigma fp64 [r]); omega fp64
    [n (+ cols when damp > 0)][r + p]."""
    rows, cols = (int(v) for v in w_dom.shape)
    n = int(x.shape[0])
    if x.dim() != 2 or int(x.shape[1]) != cols or not x.is_contiguous() or x.dtype not in (torch.bfloat16,
                                                                                           torch.float32):
        raise ValueError("x must be a contiguous bf16 or fp32 [n][cols] tensor")
    np_rows = n + (cols if damp > 0 else 0)
    p = int(omega.shape[1]) - r
    if omega.dtype != torch.float64 or not omega.is_contiguous() or int(omega.shape[0]) != np_rows:
        raise ValueError("omega must be a contiguous fp64 [n (+ cols when damp > 0)][r + p] tensor")
    dt = LX_BF16 if w_dom.dtype == torch.bfloat16 else LX_F32
    xdt = LX_BF16 if x.dtype == torch.bfloat16 else LX_F32
    dev = w_dom.device
    A = torch.empty(rows, r, dtype=torch.float32, device=dev)
    B = torch.empty(r, cols, dtype=torch.float32, device=dev)
    sig = torch.empty(r, dtype=torch.float64, device=dev)
    nb = int(lib().lx_weighted_workspace_bytes(rows, cols, n, 1 if damp > 0 else 0, r, p))
    if nb == 0:
        raise LorexError(LX_ERR_UNSUPPORTED, f"unsupported shape for lx_weighted_factors: rows={rows} cols={cols} n={n} r={r} p={p}")
    ws = torch.empty(nb, dtype=torch.uint8, device=dev)
    _check(lib().lx_weighted_factors(_ptr(w_dom), _ptr(w_mem), dt, rows, cols,
                                     _ptr(perm) if perm is not None else None, perm_axis, _ptr(x), xdt, n,
                                     float(damp), r, p, q, _ptr(omega), _ptr(A), _ptr(B), _ptr(sig), _ptr(ws), nb,
                                     _stream(stream)))
    return A, B, sig


def convert_f16(w: torch.Tensor, stream=None):
    """fp16 copy of bf16 weights [n][rows][cols] (lx_convert_f16): returns
    (fp16 [n][rows][cols] = w * 2^exps[i] per matrix, int32 exps [n])."""
    if w.dtype != torch.bfloat16 or not w.is_contiguous() or w.dim() != 3:
        raise ValueError("w must be a contiguous bf16 [n][rows][cols] tensor")
    n, rows, cols = (int(v) for v in w.shape)
    w16 = torch.empty(n, rows, cols, dtype=torch.float16, device=w.device)
    ex = torch.empty(n, dtype=torch.int32, device=w.device)
    _check(lib().lx_convert_f16(_ptr(w), n, rows, cols, _ptr(w16), _ptr(ex), _stream(stream)))
    return w16, ex


def convert_f16_padded(w: torch.Tensor, rows_out: int, cols_out: int, stream=None):
    """lx_convert_f16 into a zero-padded [n][rows_out][cols_out] layout
    (lx_convert_f16_padded): returns (fp16 tensor, int32 exps [n])."""
    if w.dtype != torch.bfloat16 or not w.is_contiguous() or w.dim() != 3:
        raise ValueError("w must be a contiguous bf16 [n][rows][cols] tensor")
    n, rows, cols = (int(v) for v in w.shape)
    w16 = torch.empty(n, rows_out, cols_out, dtype=torch.float16, device=w.device)
    ex = torch.empty(n, dtype=torch.int32, device=w.device)
    _check(lib().lx_convert_f16_padded(_ptr(w), n, rows, cols, rows_out, cols_out, _ptr(w16), _ptr(ex),
                                       _stream(stream)))
    return w16, ex


def pad_bf16(w: torch.Tensor, rows_out: int, cols_out: int, stream=None) -> torch.Tensor:
    """Zero-padded copy [n][rows_out][cols_out] of bf16 weights (lx_pad_bf16)."""
    if w.dtype != torch.bfloat16 or not w.is_contiguous() or w.dim() != 3:
        raise ValueError("w must be a contiguous bf16 [n][rows][cols] tensor")
    n, rows, cols = (int(v) for v in w.shape)
    out = torch.empty(n, rows_out, cols_out, dtype=torch.bfloat16, device=w.device)
    _check(lib().lx_pad_bf16(_ptr(w), n, rows, cols, rows_out, cols_out, _ptr(out), _stream(stream)))
    return out


def attach_down_f16(layer: "DeviceLayer") -> "DeviceLayer":
    """Give a bf16 layer the fp16 copy of its anchor down weights; a no-op
    for fp32 layers."""
    if layer.dtype == "bf16":
        layer.anchor_down_f16, layer.anchor_down_f16_exp = convert_f16(layer.anchor_down)
    return layer


def attach_factors_f16(layer: "DeviceLayer") -> "DeviceLayer":
    """Give every level of a bf16 layer the fp16 copies of its factors (used,
    with the anchor down fp16 copy, by the fp16 path of the correction
    products); a rank that is not a multiple of 64 gets copies padded with
    zeros to the next one (rank_f16, with padded bf16 b_gate / b_up); a no-op
    for fp32 layers, levels without factors and padded ranks above 128."""
    if layer.dtype == "bf16":
        for lv in layer.levels:
            if lv.n_factors == 0:
                continue
            r = lv.rank
            rf = -(-r // 64) * 64  # the fp16 path takes ranks that are multiples of 64
            if rf > 128:
                continue
            for n in ("a_gate", "a_up", "a_down"):  # [n][rows][r]: zero columns
                w = getattr(lv, n)
                w16, ex = convert_f16(w) if rf == r else convert_f16_padded(w, w.shape[1], rf)
                setattr(lv, n + "_f16", w16)
                setattr(lv, n + "_f16_exp", ex)
            w = lv.b_down  # [n][r][f]: zero rows
            lv.b_down_f16, lv.b_down_f16_exp = convert_f16(w) if rf == r else convert_f16_padded(w, rf, w.shape[2])
            if rf > r:
                lv.rank_f16 = rf
                lv.b_gate_pad = pad_bf16(lv.b_gate, rf, lv.b_gate.shape[2])
                lv.b_up_pad = pad_bf16(lv.b_up, rf, lv.b_up.shape[2])
    return layer


def attach_down_f8(layer: "DeviceLayer") -> "DeviceLayer":
    """Give a bf16 layer the fp8 copy of its anchor down weights (used by the
    anchor down projection where applicable); a no-op for other layers."""
    if layer.dtype == "bf16" and layer.f % 64 == 0:
        layer.anchor_down_f8, layer.anchor_down_f8_scale = quantize_f8(layer.anchor_down)
    return layer


def to_device(layer, device="cuda", lo8: bool = True, f16: bool = True) -> DeviceLayer:
    """Copy a host layer (fields as in ``lxsynth.Layer``) to device tensors.
    ``lo8``: also prepare the fp8 copy of the anchor down weights (bf16 layers
    with f a multiple of 64), so the anchor down projection can take its
    fp8-lo path; ``f16``: also prepare their fp16 copy and the fp16 copies of
    every level's factors (bf16 layers), for the fp16 path (preferred where it
    applies)."""
    dt = layer.dtype
    levels = []
    for lv in layer.levels:
        levels.append(DeviceLevel(
            parent=_dev_array(np.asarray(lv.parent, dtype=np.int32), dt, device),
            factor_of=_dev_array(np.asarray(lv.factor_of, dtype=np.int32), dt, device),
            rank=int(lv.rank),
            **{n: _dev_array(getattr(lv, n), dt, device)
               for n in ("a_gate", "b_gate", "a_up", "b_up", "a_down", "b_down")}))
    dl = DeviceLayer(E=int(layer.E), d=int(layer.d), f=int(layer.f), dtype=dt,
                     anchor_gate=_dev_array(layer.anchor_gate, dt, device),
                     anchor_up=_dev_array(layer.anchor_up, dt, device),
                     anchor_down=_dev_array(layer.anchor_down, dt, device), levels=levels)
    if lo8:
        dl = attach_down_f8(dl)
    if f16:
        dl = attach_factors_f16(attach_down_f16(dl))
    return dl


# ----------------------------------------------------------------- calls
def workspace_bytes(layer: DeviceLayer, T: int, k: int, kind: str = "tree") -> int:
    L = lib()
    if kind == "flat":
        n = L.lx_moe_workspace_bytes(ctypes.byref(layer.flat_struct()), T, k)
    elif kind == "dense":
        n = L.lx_dense_moe_workspace_bytes(ctypes.byref(layer.dense_struct()), T, k)
    else:
        n = L.lx_moe_tree_workspace_bytes(ctypes.byref(layer.tree_struct()), T, k)
    if n == 0:
        raise LorexError(LX_ERR_INVALID_ARGUMENT, L.lx_last_error().decode())
    return int(n)


def alloc_workspace(layer: DeviceLayer, T: int, k: int, kind: str = "tree", device="cuda"):
    return torch.empty(workspace_bytes(layer, T, k, kind), dtype=torch.uint8, device=device)


def forward(layer: DeviceLayer, x: torch.Tensor, topk_ids: torch.Tensor, topk_weights: torch.Tensor,
            out: Optional[torch.Tensor] = None, out_dtype: int = LX_F32,
            workspace: Optional[torch.Tensor] = None, kind: Optional[str] = None, stream=None):
    """One MoE-layer forward. ``kind``: "flat" (lx_moe_forward), "tree"
    (lx_moe_forward_tree) or "dense" (lx_dense_moe_forward); default: flat
    for one correction level, dense for none, tree otherwise."""
    T, k = int(topk_ids.shape[0]), int(topk_ids.shape[1]) if topk_ids.dim() == 2 else 1
    if kind is None:
        kind = {0: "dense", 1: "flat"}.get(len(layer.levels), "tree")
    if out is None:
        out = torch.empty(T, layer.d, device=x.device,
                          dtype=torch.float32 if out_dtype == LX_F32 else torch.bfloat16)
    if workspace is None:
        workspace = alloc_workspace(layer, T, k, kind, x.device)
    for name, t in (("x", x), ("topk_ids", topk_ids), ("topk_weights", topk_weights), ("out", out)):
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    if topk_ids.dtype != torch.int32 or topk_weights.dtype != torch.float32:
        raise ValueError("topk_ids must be int32 and topk_weights float32")
    L = lib()
    args = (T, k, _ptr(x), _ptr(topk_ids), _ptr(topk_weights), _ptr(out), out_dtype,
            _ptr(workspace), workspace.numel(), _stream(stream))
    if kind == "flat":
        st = L.lx_moe_forward(ctypes.byref(layer.flat_struct()), *args)
    elif kind == "dense":
        st = L.lx_dense_moe_forward(ctypes.byref(layer.dense_struct()), *args)
    else:
        st = L.lx_moe_forward_tree(ctypes.byref(layer.tree_struct()), *args)
    _check(st)
    return out


def route_forward(layer: DeviceLayer, x: torch.Tensor, w_r: torch.Tensor, k: int,
                  out: Optional[torch.Tensor] = None, ids: Optional[torch.Tensor] = None,
                  weights: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                  out_dtype: int = LX_F32, stream=None):
    """The router fused into the tree forward (lx_route_moe_forward_tree):
    bf16 x [T][d] and router weights [E][d] -> (out, int32 ids [T][k], fp32
    weights [T][k]). Flat layers run as their one-level tree."""
    if x.dtype != torch.bfloat16 or w_r.dtype != torch.bfloat16:
        raise ValueError("x and w_r must be bf16")
    if not (x.is_contiguous() and w_r.is_contiguous()):
        raise ValueError("x and w_r must be contiguous")
    T = int(x.shape[0])
    desc = layer.tree_struct()
    L = lib()
    if ids is None:
        ids = torch.empty(T, k, dtype=torch.int32, device=x.device)
    if weights is None:
        weights = torch.empty(T, k, dtype=torch.float32, device=x.device)
    if out is None:
        out = torch.empty(T, layer.d, device=x.device,
                          dtype=torch.float32 if out_dtype == LX_F32 else torch.bfloat16)
    if workspace is None:
        n = int(L.lx_route_moe_tree_workspace_bytes(ctypes.byref(desc), T, k))
        if n == 0:
            raise LorexError(LX_ERR_INVALID_ARGUMENT, L.lx_last_error().decode())
        workspace = torch.empty(n, dtype=torch.uint8, device=x.device)
    _check(L.lx_route_moe_forward_tree(ctypes.byref(desc), T, k, _ptr(x), _ptr(w_r), _ptr(ids), _ptr(weights),
                                       _ptr(out), out_dtype, _ptr(workspace), workspace.numel(), _stream(stream)))
    return out, ids, weights


STATIC_SCRATCH_BYTES = 64 << 20  # LX_STATIC_SCRATCH_BYTES


def forward_static(layer: DeviceLayer, x: torch.Tensor, topk_ids: torch.Tensor, topk_weights: torch.Tensor,
                   out: torch.Tensor, out_dtype: int = LX_F32, stream=None) -> torch.Tensor:
    """The tree forward on the library's static per-GPU scratch
    (lx_moe_forward_tree_static): no workspace, nothing allocated by the
    call; ``out`` is caller-provided. Flat layers run as their one-level
    tree."""
    T, k = int(topk_ids.shape[0]), int(topk_ids.shape[1])
    for name, t in (("x", x), ("topk_ids", topk_ids), ("topk_weights", topk_weights), ("out", out)):
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    if topk_ids.dtype != torch.int32 or topk_weights.dtype != torch.float32:
        raise ValueError("topk_ids must be int32 and topk_weights float32")
    _check(lib().lx_moe_forward_tree_static(ctypes.byref(layer.tree_struct()), T, k, _ptr(x), _ptr(topk_ids),
                                            _ptr(topk_weights), _ptr(out), out_dtype, _stream(stream)))
    return out


def bucket(layer: DeviceLayer, topk_ids: torch.Tensor, level: int,
           workspace: Optional[torch.Tensor] = None, stream=None):
    """Bucketing arrays of one tree level: (row_token, node_offsets, slot_row).
    ``row_token`` is trimmed to the row count."""
    T, k = int(topk_ids.shape[0]), int(topk_ids.shape[1])
    N = layer.n_anchors if level == 0 else layer.levels[level - 1].n_nodes
    dev = topk_ids.device
    if workspace is None:
        workspace = alloc_workspace(layer, T, k, "tree", dev)
    row_token = torch.empty(max(T * min(k, N), 1), dtype=torch.int32, device=dev)
    offsets = torch.empty(N + 1, dtype=torch.int32, device=dev)
    slot_row = torch.empty(max(T * k, 1), dtype=torch.int32, device=dev)
    st = lib().lx_bucket(ctypes.byref(layer.tree_struct()), T, k, _ptr(topk_ids), level,
                         _ptr(row_token), _ptr(offsets), _ptr(slot_row), _ptr(workspace),
                         workspace.numel(), _stream(stream))
    _check(st)
    torch.cuda.current_stream().synchronize() if stream is None else stream.synchronize()
    n = int(offsets[-1].item())
    return row_token[:n], offsets, slot_row[:T * k]


def set_aux_stream(enable: bool) -> bool:
    """Allow (True) or forbid (False, the default) the forward's auxiliary
    stream (lx_set_aux_stream); returns the previous setting."""
    return bool(lib().lx_set_aux_stream(1 if enable else 0))


def read_device_status(workspace: torch.Tensor, stream=None) -> int:
    v = ctypes.c_uint32(0)
    _check(lib().lx_read_device_status(_ptr(workspace), _stream(stream), ctypes.byref(v)))
    return int(v.value)


# ------------------------------------------------------------ kernel timing
def profile_enable(on: bool = True):
    _check(lib().lx_profile_enable(1 if on else 0))


def profile_reset():
    _check(lib().lx_profile_reset())


def profile_read() -> dict:
    """{kernel name: (launches, total ms)} after waiting for pending events."""
    L = lib()
    _check(L.lx_profile_collect())
    out = {}
    for i in range(L.lx_profile_count()):
        name = ctypes.c_char_p()
        n = ctypes.c_int64()
        ms = ctypes.c_double()
        _check(L.lx_profile_entry(i, ctypes.byref(name), ctypes.byref(n), ctypes.byref(ms)))
        out[name.value.decode()] = (int(n.value), float(ms.value))
    return out


class PreparedCall:
    """A forward call with every argument marshalled once; ``__call__`` only
    re-issues the C call (for timing loops)."""

    def __init__(self, layer: DeviceLayer, x: torch.Tensor, topk_ids: torch.Tensor,
                 topk_weights: torch.Tensor, out: torch.Tensor, workspace: torch.Tensor,
                 kind: str, out_dtype: int = LX_F32, stream=None):
        L = lib()
        self._keep = (layer, x, topk_ids, topk_weights, out, workspace)
        if kind == "flat":
            self._desc, self._fn = layer.flat_struct(), L.lx_moe_forward
        elif kind == "dense":
            self._desc, self._fn = layer.dense_struct(), L.lx_dense_moe_forward
        else:
            self._desc, self._fn = layer.tree_struct(), L.lx_moe_forward_tree
        T, k = int(topk_ids.shape[0]), int(topk_ids.shape[1])
        self._args = (ctypes.byref(self._desc), T, k, _ptr(x), _ptr(topk_ids), _ptr(topk_weights),
                      _ptr(out), out_dtype, _ptr(workspace), workspace.numel(), _stream(stream))

    def __call__(self):
        st = self._fn(*self._args)
        if st != LX_OK:
            _check(st)

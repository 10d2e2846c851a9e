"""fp64 reference of the unchanged top-k router (test infrastructure).

THIS MODULE IS TEST INFRASTRUCTURE, like the rest of the package: only the
test suite, the smoke check and the benchmark's CPU-baseline leg use it.

What it follows: the compressed layer keeps the model's router as it is
(Sec. 3 "Stage 1" and Fig. overview: top-k over all E experts, so every expert
stays addressable). The paper gives no formula for the router; the reading
used throughout this repository:

* logits_e = sum_i W_r[e, i] x_i, with W_r stored in [E][d] layout (the
  nn.Linear layout of the gate), promoted to fp64 exactly;
* the k largest logits, in descending order; equal logits put the lower
  expert index first;
* weights = the softmax over all E logits, restricted to the k chosen experts
  and renormalised to sum 1 (which equals the softmax of the chosen logits).
"""
from __future__ import annotations

import numpy as np

from .moe import to_f64


def router_logits(x, w_r, dtype: str) -> np.ndarray:
    """fp64 logits [T, E] of stored activations x [T, d] and router weights
    w_r [E, d] (both in the storage dtype ``dtype``). One matrix-vector
    product per expert, so experts with equal weight rows get bitwise equal
    logits (a blocked matrix product may sum their columns in different
    orders)."""
    x64 = to_f64(x, dtype)
    w64 = to_f64(w_r, dtype)
    return np.stack([x64 @ w64[e] for e in range(w64.shape[0])], axis=1)


def route_topk(x, w_r, dtype: str, k: int):
    """(ids int32 [T, k], weights fp64 [T, k], logits fp64 [T, E])."""
    logits = router_logits(x, w_r, dtype)
    T, E = logits.shape
    if not 1 <= k <= E:
        raise ValueError("need 1 <= k <= E")
    # stable sort of the negated logits: ties keep ascending expert order
    order = np.argsort(-logits, axis=1, kind="stable")[:, :k]
    full = np.exp(logits - logits.max(axis=1, keepdims=True))
    full /= full.sum(axis=1, keepdims=True)
    chosen = np.take_along_axis(full, order, axis=1)
    weights = chosen / chosen.sum(axis=1, keepdims=True)
    return order.astype(np.int32), weights, logits


def fp32_sum_bound(x, w_r, dtype: str) -> np.ndarray:
    """Bound [T, E] on |fl32(logit) - logit| for any order of fp32 summation of
    the d exact products x_i W_r[e, i] (bf16 x bf16 products are exact in
    fp32): gamma_(d-1) * sum_i |x_i W_r[e, i]|, gamma_n = n u / (1 - n u),
    u = 2^-24, plus the rounding of the final value."""
    a = np.abs(to_f64(x, dtype)) @ np.abs(to_f64(w_r, dtype)).T
    d = np.asarray(x).shape[1]
    u = 2.0 ** -24
    g = (d - 1) * u / (1 - (d - 1) * u)
    return g * a + u * a

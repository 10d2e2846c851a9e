"""Algorithmic work of the compressed MoE forward: FLOPs and HBM bytes.

These are the counts the method must do, used for roofline fractions. They
exclude executed overhead (the hi+lo split of the down-projection input, tile
padding, elementwise SwiGLU work) and workspace traffic.

Per-token model of Sec. 5 "Inference cost" (gate projection, two co-selected
experts sharing a dominant, Fig. flops): the original pays k * 2IH FLOPs and
loads k full matrices; the amortized form pays 2IH once plus k * 2r(I+H) for
the rank-r corrections; their ratio is the closed-form speedup of that section.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


def closed_form_speedup(k: int, I: int, H: int, r: int) -> float:
    """k*2IH / (2IH + k*2r(I+H)): amortized vs original per-token cost."""
    return (k * 2 * I * H) / (2 * I * H + k * 2 * r * (I + H))


def per_token_projection_cost(k: int, I: int, H: int, r: int, bytes_per_elem: int = 2):
    """FLOPs and weight bytes of one projection for one token (Fig. flops).

    Returns a dict with ``original_flops``, ``original_bytes`` (k full matrices),
    ``amortized_flops``, ``amortized_bytes`` (one shared matrix plus k factor
    pairs), ``dense_matrix_bytes`` and ``factor_pair_bytes``.
    """
    full = I * H
    pair = r * (I + H)
    return dict(
        original_flops=k * 2 * full,
        original_bytes=k * full * bytes_per_elem,
        amortized_flops=2 * full + k * 2 * pair,
        amortized_bytes=(full + k * pair) * bytes_per_elem,
        dense_matrix_bytes=full * bytes_per_elem,
        factor_pair_bytes=pair * bytes_per_elem,
    )


@dataclass
class LevelRows:
    """Row counts of one tree level, from the bucketing."""
    rank: int          # 0 for the anchor level
    rows: int          # unique (token, node) pairs whose node does work
    nodes_touched: int  # distinct nodes with at least one such row


def algorithmic_counts(d: int, f: int, levels: list, T: int, k: int,
                       weight_bytes: int = 2, x_bytes: int = 2, out_bytes: int = 4):
    """FLOPs and bytes of one layer forward.

    ``levels[0]`` is the anchor level (dense gate/up/down per row);
    ``levels[l>0]`` are correction levels (rank-r gate/up/down per row, only
    rows whose node carries a factor). FLOPs count 2 per multiply-add:
    anchor rows 6*d*f each, correction rows 6*r*(d+f) each. Bytes count every
    touched weight once, x once, the output once, and ids + weights.
    """
    a = levels[0]
    flops = 6 * d * f * a.rows
    wbytes = 3 * d * f * a.nodes_touched * weight_bytes
    for lv in levels[1:]:
        flops += 6 * lv.rank * (d + f) * lv.rows
        wbytes += 3 * lv.rank * (d + f) * lv.nodes_touched * weight_bytes
    io = T * d * (x_bytes + out_bytes) + T * k * 8
    return dict(flops=flops, weight_bytes=wbytes, bytes=wbytes + io,
                gate_up_flops=4 * d * f * a.rows, down_flops=2 * d * f * a.rows)


def level_rows_from_buckets(offsets_per_level: list, factor_of_per_level: list,
                            ranks: list) -> list:
    """LevelRows for every level from bucketing offsets (host arrays).

    ``factor_of_per_level[l]`` is None for the anchor level (every node does
    work) and the level's factor map otherwise.
    """
    out = []
    for li, off in enumerate(offsets_per_level):
        cnt = np.diff(np.asarray(off, dtype=np.int64))
        fo = factor_of_per_level[li]
        if fo is not None:
            cnt = np.where(np.asarray(fo) >= 0, cnt, 0)
        out.append(LevelRows(rank=int(ranks[li]), rows=int(cnt.sum()),
                             nodes_touched=int((cnt > 0).sum())))
    return out

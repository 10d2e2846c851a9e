"""Shared test helpers: tiny layers and tolerance checks (no method arithmetic)."""
from __future__ import annotations

import copy

import numpy as np

from lxsynth import Layer, Level, make_layer_flat, make_layer_tree


def rel_max_err(got, ref) -> float:
    """max|got - ref| / RMS(ref)."""
    ref = np.asarray(ref, dtype=np.float64)
    got = np.asarray(got, dtype=np.float64)
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 1.0
    if rms == 0.0:
        rms = 1.0
    return float(np.max(np.abs(got - ref))) / rms if ref.size else 0.0


def tiny_flat(E=6, C=2, d=8, f=16, r=3, dtype="f32", seed=5, shuffle=False):
    return make_layer_flat(E, C, d, f, r, dtype, seed, shuffle=shuffle)


def tiny_tree(E=8, d=8, f=8, n_roots=1, subs=2, r_sub=3, r_leaf=2, dtype="f32", seed=6):
    return make_layer_tree(E, d, f, n_roots, subs, r_sub, r_leaf, dtype, seed)


def dense_layer(wg, wu, wd, dtype="f32"):
    """L = 0 layer whose anchors are the experts (values already stored)."""
    E, f, d = wg.shape
    return Layer(E=E, d=d, f=f, dtype=dtype, anchor_gate=wg, anchor_up=wu,
                 anchor_down=wd, levels=[])


def random_routing(T, k, E, seed, allow_dupes=False, drop_frac=0.0, bad_frac=0.0):
    rng = np.random.default_rng(seed)
    if allow_dupes:
        ids = rng.integers(0, E, size=(T, k))
    else:
        ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]) if T else np.zeros((0, k), int)
    ids = ids.astype(np.int32)
    if drop_frac:
        ids[rng.random(ids.shape) < drop_frac] = -1
    if bad_frac:
        m = rng.random(ids.shape) < bad_frac
        ids[m] = rng.choice([-7, -2, E, E + 3], size=int(m.sum()))
    w = rng.random((T, k)).astype(np.float32) + np.float32(0.05)
    return ids, w


def clone(layer):
    return copy.deepcopy(layer)


def zero_level(layer, li):
    """Copy of layer with every node of correction level li set to no factor."""
    out = clone(layer)
    out.levels[li].factor_of = np.full_like(out.levels[li].factor_of, -1)
    return out


__all__ = ["rel_max_err", "tiny_flat", "tiny_tree", "dense_layer", "random_routing",
           "clone", "zero_level", "Level", "Layer"]

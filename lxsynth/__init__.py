"""Seeded synthetic inputs for the LorExperts / BTExperts MoE-layer forward.

This module is shared by the CPU oracle and the GPU path. It only draws numbers
and stores them; it holds none of the layer's arithmetic. Everything it produces
is a plain numpy array on the host:

* weights in the storage dtype of the layer: bf16 as ``np.uint16`` bit patterns
  (round-to-nearest-even from an fp32 draw) or fp32;
* ``x`` in the same storage dtype;
* routing: ``topk_ids`` int32 ``[T, k]`` and ``topk_weights`` fp32 ``[T, k]``.

The router (x times a router matrix, top-k over all experts, softmax over the
chosen logits) is the model's unchanged gate (Sec. 3 "Stage 1", Fig. overview:
every expert stays addressable). It is input generation here, not part of the
library: the library takes ids and weights as inputs.

Layer layout (one MoE layer):

* level 0 holds dense anchors: ``anchor_gate``/``anchor_up`` ``[N0, f, d]`` and
  ``anchor_down`` ``[N0, d, f]`` (nn.Linear layout, input dimension contiguous);
* levels 1..L each hold ``parent[N_l]`` (node index at level l-1),
  ``factor_of[N_l]`` (index into the level's factor arrays, -1 = no correction)
  and rank-``r_l`` factor pairs, output-side ``a_*`` and input-side ``b_*``:
  ``a_gate/a_up [M, f, r]``, ``b_gate/b_up [M, r, d]``, ``a_down [M, d, r]``,
  ``b_down [M, r, f]``;
* the nodes of level L are the experts.

A flat LorExperts layer (Sec. 3 "Representation") is L = 1: the anchors are the
cluster dominants, level 1 are the experts, ``parent`` is the cluster map and the
dominant expert of each cluster has ``factor_of = -1``. A BTExperts tree
(Sec. 5, Fig. tree) has L = 2 here: roots, sub-dominants, leaves. A dense MoE
(every expert stored in full) is L = 0 with one anchor per expert.
"""
from .gen import (  # noqa: F401
    CONFIGS,
    Layer,
    Level,
    Routing,
    Problem,
    f32_to_bf16_bits,
    make_problem,
    make_layer_flat,
    make_layer_tree,
    make_x,
    route_gaussian,
    route_community,
    route_coselect,
    make_router,
    config,
)

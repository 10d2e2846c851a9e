"""CPU oracle for the LorExperts / BTExperts MoE-layer forward.

THIS PACKAGE IS TEST INFRASTRUCTURE. Only the test suite, the smoke check and
the benchmark's CPU-baseline leg may import or run it. The product path (the
HIP library and its Python binding) never calls it and shares no code with it.

Contents:

* ``moe.moe_forward``            binding oracle: dense per-expert reconstruction
                                  and the per-token top-k SwiGLU MoE, fp64;
* ``moe.moe_forward_amortized``  the amortized formulation (shared anchor and
                                  ancestor terms computed once per token), fp64,
                                  used only to cross-check the binding oracle;
* ``moe.moe_forward_bruteforce`` scalar Python loops for tiny shapes;
* ``bucket.bucket``              the routing-bucketing arrays, from their
                                  definition (sort + unique), bit-exact target;
* ``bucket.bucket_bruteforce``   the same arrays from explicit loops;
* ``router.route_topk``          the unchanged top-k router (logits, top-k in
                                  descending order, renormalised softmax), fp64;
* ``cluster``                     firing / co-activation counts, the NPMI
                                  distance and frequency-seeded k-medoids with
                                  the dominant choice (Stages 1-2), fp64;
* ``stage3``                      neuron-alignment cost, exact assignment,
                                  aligned residual and randomized truncated
                                  SVD with the symmetric split (Stage 3), fp64.

Every function is pinned by ``tests/test_oracle_*.py`` against brute force,
closed forms, library routines and invariants of the method.
"""
from . import bucket, cluster, moe, router, stage3  # noqa: F401

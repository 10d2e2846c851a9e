"""lorex: the LorExperts / BTExperts MoE-layer forward on MI355X (gfx950).

The compute lives in ``liblorex.so`` (hand-written HIP kernels behind a C ABI,
declared in ``include/lorex.h``). ``paper_2608_07814_amd.lorex`` is the thin
Python binding; it loads the library on first use and raises if it is missing.
"""

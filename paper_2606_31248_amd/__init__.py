"""STRATA hot path on AMD Instinct MI355X (gfx950).

Neighbourhood attention over the (level, y, x) token grid of each tile with
StereoRoPE, and the overlapping-tile blend, as hand-written HIP kernels behind
a C ABI (include/strata.h).  ``binding`` wraps that ABI; ``pipeline`` chains
the calls of one face rollout step; ``inputs`` draws seeded synthetic inputs.
Submodules are imported on use so that the input generators load without the
HIP library.
"""
__all__ = ["binding", "pipeline", "inputs", "build"]

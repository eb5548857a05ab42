"""Reachable-state weighted FST composition on AMD MI355X (gfx950).

Implements the hot path of Argueta & Chiang, "Composing Finite State
Transducers on GPUs": the composition M1 o M2 restricted to state pairs
reachable from the start pair, with identical composed arcs merged by adding
their weights.  Every step runs in hand-written HIP kernels behind the C ABI
declared in ``include/fstc.h``; ``paper_1805_06383_amd.fstc`` is the thin
Python binding over it.

Submodules are imported on demand so that ``workloads`` (seeded synthetic
inputs) can be used without loading the GPU library.
"""

__all__ = ["fstc", "workloads"]

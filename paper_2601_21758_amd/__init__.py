"""EWSJF scheduler core for AMD Instinct MI355X (gfx950).

Refine-and-Prune partitioning, Dynamic Queue Routing, Density-Weighted
Scoring and top-B admission as HIP kernels behind the C ABI of
include/ewsjf.h (libewsjf.so).  `paper_2601_21758_amd.ewsjf` is the thin
PyTorch binding; `paper_2601_21758_amd.workloads` draws seeded synthetic
inputs.  Importing the package loads nothing; the first call into the
binding loads libewsjf.so and raises if it has not been built.
"""
__all__ = ["ewsjf", "workloads"]

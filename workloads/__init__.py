"""Seeded synthetic inputs shaped like the paper's heterogeneous-graph workloads.

This package is shared by the CPU oracle's tests and by the GPU path's tests and
benchmark.  It only draws random numbers and index arrays; it performs none of
the layers' arithmetic.
"""
from .synth import (  # noqa: F401
    CONFIGS, make_graph, make_tensors, tiny_graph, tiny_tensors, degree_stats,
)

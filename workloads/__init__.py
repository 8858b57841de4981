"""Seeded synthetic inputs for the dynamic graph-index workloads.

This package draws vectors, ids and operation streams only.  It holds none
of the index method's arithmetic (no distances, no search, no pruning), so
that both the GPU path and the CPU oracle can consume the same inputs
without sharing any code of the method.
"""
from .generators import (  # noqa: F401
    CONFIGS,
    PATTERNS,
    IndexConfig,
    PatternStream,
    Workload,
    make_workload,
)

"""Seeded synthetic workloads (gradients with a planted spectrum) for the
GreedyLore compression path.

This package is shared by the tests, the bench and the CPU oracle's callers.
It draws inputs only: it holds none of the compression method's arithmetic.
"""
from .gen import (  # noqa: F401
    Workload,
    WORKLOADS,
    get_workload,
    planted_factors,
    planted_matrix,
    gradient_batch,
    noise_level,
)

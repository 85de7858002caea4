"""Seeded synthetic operator graphs shaped like the paper's workloads.

This package is shared by the CPU oracle's tests and by the GPU path's tests and
benchmark.  It only *draws* inputs (graph structure, per-op costs, device
parameters and random perturbations); it contains none of the placement method's
arithmetic.
"""
from .graphs import (Workload, make_config, make_random_dag, perturb_placements,
                     from_edges, CONFIG_NAMES)

__all__ = ["Workload", "make_config", "make_random_dag", "perturb_placements",
           "from_edges", "CONFIG_NAMES"]

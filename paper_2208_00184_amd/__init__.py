"""MI355X (gfx950) implementation of the Celeritas placement hot path.

The computation lives in libcel.so (HIP kernels behind the C ABI of
include/cel.h); this package is its thin Python binding.
"""
from ._binding import (CelError, Devices, Graph, blevel, cluster, colocate, comm_sums, cpd_order, dfs_order,
                       kernel_stats, lib, makespan, makespan_info, makespan_relax, blevel_info, policy_iteration, topo_levels_info, cluster_info, step_latency, makespan_model, order_place, place, place_ext, timing,
                       topo_levels, version, CLUSTER_DP, CLUSTER_GREEDY, COMM_OFF, EXPORTS, LIB_PATH,
                       MODEL_INSERT, MODEL_COMM_TASKS, MODEL_COMM_BLOCK)

__all__ = ["CelError", "Devices", "Graph", "blevel", "cluster", "colocate", "comm_sums", "cpd_order", "dfs_order", "kernel_stats", "lib", "step_latency",
           "makespan_info", "makespan_relax", "blevel_info", "policy_iteration", "topo_levels_info", "cluster_info",
           "makespan", "makespan_model", "order_place", "place", "place_ext", "timing", "topo_levels", "version",
           "CLUSTER_DP", "CLUSTER_GREEDY", "COMM_OFF", "EXPORTS", "LIB_PATH", "MODEL_INSERT",
           "MODEL_COMM_TASKS", "MODEL_COMM_BLOCK"]

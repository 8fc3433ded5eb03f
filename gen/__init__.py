"""Seeded synthetic graph generators shared by the CPU oracle, the tests and the benchmark.

This package only produces inputs: symmetric CSR adjacency structures (row pointers,
column indices, optional positive edge weights) and the solve parameters of each
workload.  It holds none of the resistance-curvature arithmetic (no edge numbering,
no Laplacian, no projection, no solve), so the oracle and the GPU path can both
consume it without sharing any of the method's code.
"""
from .graphs import (  # noqa: F401
    CSRGraph,
    from_edges,
    complete_graph,
    cycle_graph,
    path_graph,
    star_graph,
    complete_bipartite,
    random_tree,
    barbell_graph,
    erdos_renyi,
    sbm,
    chung_lu,
    component_count,
    relabel,
)
from .configs import CONFIGS, SolveParams, Workload, make_graph, get_workload  # noqa: F401

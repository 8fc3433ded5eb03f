"""The synthetic workloads and their solve parameters.

Each workload is a seeded graph recipe shaped like one of the paper's evaluation
graphs (Section 4: the SBM of Table 2, ogbn-arxiv, Reddit and ogbn-products of
Table 3 and its text), plus the projection width K, the column block width, the
diagonal shift delta (the paper's epsilon in Eq. 5), the CG tolerance tau, the
working precision and the projection seed.  The datasets themselves are not used:
these graphs stand in for them.  ORDER lists the five performance workloads; sbm2k is
the smaller SBM of the curvature-agreement study (Table 2).
"""
from __future__ import annotations

import os
from dataclasses import dataclass, field

from . import graphs as G

__all__ = ["SolveParams", "Workload", "CONFIGS", "make_graph", "get_workload", "cache_dir"]


@dataclass(frozen=True)
class SolveParams:
    K: int               # total number of JL columns (projection dimension)
    k_block: int         # columns solved together in one block
    delta: float         # diagonal shift of L + delta*I
    tol: float           # relative residual tolerance per column
    dtype: str           # working precision of the CG vectors: "f64" or "f32"
    seed: int            # projection seed
    max_iter: int = 10000
    eta: float = 1e-12   # stabiliser of the node sampling weight


@dataclass(frozen=True)
class Workload:
    name: str
    description: str
    graph_kind: str
    graph_args: dict = field(default_factory=dict)
    params: SolveParams = None


CONFIGS = {
    "er2k": Workload(
        "er2k",
        "Erdos-Renyi G(2000, 8/1999), connected draw, unit weights; K=32, fp64",
        "er_connected", {"n": 2000, "p": 8.0 / 1999.0, "seed": 1},
        SolveParams(K=32, k_block=32, delta=1e-6, tol=1e-8, dtype="f64", seed=101)),
    "sbm20k": Workload(
        "sbm20k",
        "SBM, 10 blocks of 2000, in-degree 10, cross-degree 1, U(0.5,2) weights; K=64, fp32",
        "sbm", {"blocks": 10, "size": 2000, "p_in": 10.0 / 1999.0, "p_out": 1.0 / 18000.0,
                "seed": 2},
        SolveParams(K=64, k_block=64, delta=1e-5, tol=1e-6, dtype="f32", seed=102)),
    "cl170k": Workload(
        "cl170k",
        "Chung-Lu gamma=2.1, n=170k, ~1.2M edges, largest component, unit weights; "
        "K=128, fp32 (ogbn-arxiv-shaped)",
        "chung_lu", {"n": 170_000, "gamma": 2.1, "i0": 10.0, "m_target": 1_230_000, "seed": 3,
                     "weighted": False, "keep_largest": True},
        SolveParams(K=128, k_block=128, delta=1e-5, tol=1e-6, dtype="f32", seed=103)),
    "cl230k": Workload(
        "cl230k",
        "Chung-Lu gamma=2.1 dense hubs, n=230k, ~57M edges, unit weights; "
        "K=128 in blocks of 32, fp32 (Reddit-shaped)",
        "chung_lu", {"n": 230_000, "gamma": 2.1, "i0": 760.5, "m_target": 57_000_000, "seed": 4,
                     "weighted": False, "keep_largest": False},
        SolveParams(K=128, k_block=32, delta=1e-4, tol=1e-5, dtype="f32", seed=104)),
    "cl2400k": Workload(
        "cl2400k",
        "Chung-Lu gamma=2.3, n=2.4M, ~62M edges, U(0.5,2) weights; "
        "K=256 in blocks of 64, fp32 with fp64 dots (ogbn-products-shaped)",
        "chung_lu", {"n": 2_400_000, "gamma": 2.3, "i0": 398.2, "m_target": 62_000_000, "seed": 5,
                     "weighted": True, "keep_largest": False},
        SolveParams(K=256, k_block=64, delta=1e-4, tol=1e-5, dtype="f32", seed=105)),
    "sbm2k": Workload(
        "sbm2k",
        "SBM, 10 blocks of 200, in-degree 10, cross-degree 1, U(0.5,2) weights; K up to "
        "4096 in blocks of 64, fp32 (the curvature-agreement study of Table 2)",
        "sbm", {"blocks": 10, "size": 200, "p_in": 10.0 / 199.0, "p_out": 1.0 / 1800.0,
                "seed": 6},
        SolveParams(K=4096, k_block=64, delta=1e-5, tol=1e-6, dtype="f32", seed=106)),
}

ORDER = ["er2k", "sbm20k", "cl170k", "cl230k", "cl2400k"]


def cache_dir() -> str:
    d = os.environ.get("ERC_GRAPH_CACHE") or os.path.join(
        os.environ.get("TMPDIR", "/tmp"), "erc_graph_cache")
    os.makedirs(d, exist_ok=True)
    return d


def _build(kind: str, args: dict) -> G.CSRGraph:
    if kind == "er_connected":
        seed = args["seed"]
        while True:
            g = G.erdos_renyi(args["n"], args["p"], seed)
            if _connected(g):
                return g
            seed += 1
    if kind == "sbm":
        return G.sbm(args["blocks"], args["size"], args["p_in"], args["p_out"], args["seed"])
    if kind == "chung_lu":
        return G.chung_lu(**args)
    raise ValueError(kind)


def _connected(g: G.CSRGraph) -> bool:
    import numpy as np
    import scipy.sparse as sp
    from scipy.sparse.csgraph import connected_components

    A = sp.csr_matrix((np.ones(g.nnz, dtype=np.int8), g.col, g.rowptr), shape=(g.n, g.n))
    return connected_components(A, directed=False)[0] == 1


def make_graph(name: str, use_cache: bool = True, progress=None) -> G.CSRGraph:
    """Generate (or load the cached copy of) the graph of workload ``name``."""
    wl = CONFIGS[name]
    path = os.path.join(cache_dir(), f"{name}_v2.npz")
    if use_cache and os.path.exists(path):
        return G.CSRGraph.load(path)
    args = dict(wl.graph_args)
    if wl.graph_kind == "chung_lu":
        args["progress"] = progress
    g = _build(wl.graph_kind, args)
    if use_cache:
        g.save(path)
    return g


def get_workload(name: str) -> Workload:
    return CONFIGS[name]

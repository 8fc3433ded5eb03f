"""Seeded graph families, returned as symmetric CSR adjacency structures.

Every generator is deterministic for a given seed (NumPy ``PCG64`` via
``numpy.random.default_rng``).  Edges are undirected, without self-loops or
duplicates; the CSR stores both orientations, with the column indices of each row
sorted ascending.  Weights, when present, are positive ``float32`` values drawn once
per undirected edge, so both stored orientations carry the same value.
"""
from __future__ import annotations

import os
from dataclasses import dataclass
from typing import Optional

import numpy as np

__all__ = [
    "CSRGraph", "from_edges", "complete_graph", "cycle_graph", "path_graph",
    "star_graph", "complete_bipartite", "random_tree", "barbell_graph",
    "erdos_renyi", "sbm", "chung_lu", "component_count", "relabel",
]


@dataclass
class CSRGraph:
    """Symmetric CSR adjacency of an undirected graph.

    ``rowptr`` is int64 of length n+1, ``col`` int32 of length nnz (two entries per
    undirected edge), ``w`` is None (unit weights) or a float array of length nnz.
    """

    n: int
    rowptr: np.ndarray
    col: np.ndarray
    w: Optional[np.ndarray] = None

    @property
    def nnz(self) -> int:
        return int(self.rowptr[-1])

    @property
    def m(self) -> int:
        return self.nnz // 2

    def degrees(self) -> np.ndarray:
        return np.diff(self.rowptr)

    def summary(self) -> dict:
        deg = self.degrees()
        return {
            "n": int(self.n), "m": int(self.m), "nnz": int(self.nnz),
            "deg_min": int(deg.min()) if self.n else 0,
            "deg_median": float(np.median(deg)) if self.n else 0.0,
            "deg_max": int(deg.max()) if self.n else 0,
            "weighted": self.w is not None,
        }

    def save(self, path: str) -> None:
        tmp = path + ".tmp.npz"
        arrays = {"n": np.int64(self.n), "rowptr": self.rowptr, "col": self.col}
        if self.w is not None:
            arrays["w"] = self.w
        np.savez(tmp, **arrays)
        os.replace(tmp, path)

    @staticmethod
    def load(path: str) -> "CSRGraph":
        with np.load(path, allow_pickle=False) as f:
            w = f["w"] if "w" in f.files else None
            return CSRGraph(int(f["n"]), f["rowptr"], f["col"], w)


def from_edges(n: int, u, v, w=None, sorted_unique: bool = False) -> CSRGraph:
    """Build the symmetric CSR of an undirected edge list.

    Self-loops are rejected; repeated pairs keep the weight of their first
    occurrence.  With ``sorted_unique`` the pairs must already satisfy u < v and be
    strictly increasing in (u, v) order, which skips the deduplication sort.  Rows list
    their lower neighbours first, then their upper ones, which is ascending column
    order.
    """
    if sorted_unique:
        a = np.asarray(u, dtype=np.int64)
        b = np.asarray(v, dtype=np.int64)
        if w is not None:
            w = np.asarray(w)
    else:
        u = np.asarray(u, dtype=np.int64)
        v = np.asarray(v, dtype=np.int64)
        if u.shape != v.shape:
            raise ValueError("u and v differ in length")
        if np.any(u == v):
            raise ValueError("self-loops are not allowed")
        if u.size and (min(u.min(), v.min()) < 0 or max(u.max(), v.max()) >= n):
            raise ValueError("endpoint out of range")
        key = np.minimum(u, v) * np.int64(n) + np.maximum(u, v)
        key, first = np.unique(key, return_index=True)
        a = key // n
        b = key % n
        del key
        if w is not None:
            w = np.asarray(w)[first]
    m = a.size
    up = np.bincount(a, minlength=n).astype(np.int64)
    lo = np.bincount(b, minlength=n).astype(np.int64)
    rowptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(up + lo, out=rowptr[1:])
    col = np.empty(2 * m, dtype=np.int32)
    wcsr = None if w is None else np.empty(2 * m, dtype=w.dtype)
    # upper entries (row a, column b): edges are sorted by (a, b) already
    start = rowptr[:-1] + lo - np.concatenate([[0], np.cumsum(up)[:-1]])
    pos = start[a]
    pos += np.arange(m, dtype=np.int64)
    col[pos] = b
    if w is not None:
        wcsr[pos] = w
    # lower entries (row b, column a): stable sort by b keeps a ascending per row
    perm = np.argsort(b, kind="stable")
    start = rowptr[:-1] - np.concatenate([[0], np.cumsum(lo)[:-1]])
    pos = start[b[perm]]
    pos += np.arange(m, dtype=np.int64)
    col[pos] = a[perm]
    if w is not None:
        wcsr[pos] = w[perm]
    return CSRGraph(int(n), rowptr, col, wcsr)


def _weights(rng, m, lo=0.5, hi=2.0):
    """float32 weights uniform on [lo, hi), drawn per undirected edge."""
    u = rng.random(m, dtype=np.float32)
    return (np.float32(lo) + np.float32(hi - lo) * u).astype(np.float32)


def complete_graph(n: int, w=None) -> CSRGraph:
    a, b = np.triu_indices(n, 1)
    return from_edges(n, a, b, None if w is None else np.full(a.size, w))


def cycle_graph(n: int, w=None) -> CSRGraph:
    a = np.arange(n)
    b = (a + 1) % n
    return from_edges(n, a, b, None if w is None else np.asarray(w))


def path_graph(n: int, w=None) -> CSRGraph:
    a = np.arange(n - 1)
    return from_edges(n, a, a + 1, None if w is None else np.asarray(w))


def star_graph(n: int, w=None) -> CSRGraph:
    """Star on n nodes: centre 0 joined to the n-1 leaves 1..n-1."""
    b = np.arange(1, n)
    return from_edges(n, np.zeros(n - 1, dtype=np.int64), b,
                      None if w is None else np.asarray(w))


def complete_bipartite(a: int, b: int) -> CSRGraph:
    x, y = np.meshgrid(np.arange(a), np.arange(a, a + b), indexing="ij")
    return from_edges(a + b, x.ravel(), y.ravel())


def random_tree(n: int, seed: int, weighted: bool = False) -> CSRGraph:
    """Uniform random recursive tree: node i > 0 attaches to a uniform earlier node."""
    rng = np.random.default_rng(seed)
    child = np.arange(1, n)
    parent = (rng.random(n - 1) * child).astype(np.int64)
    w = _weights(rng, n - 1) if weighted else None
    return from_edges(n, parent, child, w)


def barbell_graph(k: int, bridge_len: int = 1, seed: Optional[int] = None) -> CSRGraph:
    """Two k-cliques joined by a path of ``bridge_len`` edges (each a bridge).

    With a seed the edge weights are random, otherwise unit.
    """
    a1, b1 = np.triu_indices(k, 1)
    nodes = 2 * k + bridge_len - 1
    off = k + bridge_len - 1
    us = [a1, a1 + off]
    vs = [b1, b1 + off]
    chain = np.arange(k - 1, k - 1 + bridge_len + 1)
    chain[-1] = off
    us.append(chain[:-1])
    vs.append(chain[1:])
    u = np.concatenate(us)
    v = np.concatenate(vs)
    w = None
    if seed is not None:
        w = _weights(np.random.default_rng(seed), u.size)
    return from_edges(nodes, u, v, w)


def erdos_renyi(n: int, p: float, seed: int, weighted: bool = False) -> CSRGraph:
    """G(n, p) by one Bernoulli draw per unordered pair (small n only)."""
    rng = np.random.default_rng(seed)
    a, b = np.triu_indices(n, 1)
    keep = rng.random(a.size) < p
    a, b = a[keep], b[keep]
    w = _weights(rng, a.size) if weighted else None
    return from_edges(n, a, b, w)


def _pairs_in_block(rng, size: int, p: float):
    a, b = np.triu_indices(size, 1)
    keep = rng.random(a.size) < p
    return a[keep], b[keep]


def sbm(blocks: int, size: int, p_in: float, p_out: float, seed: int,
        weighted: bool = True) -> CSRGraph:
    """Stochastic block model with equal blocks.

    In-block pairs are Bernoulli(p_in).  For each block pair the number of
    cross edges is Binomial(size^2, p_out); endpoints are uniform, repeats removed.
    """
    rng = np.random.default_rng(seed)
    us, vs = [], []
    for k in range(blocks):
        a, b = _pairs_in_block(rng, size, p_in)
        us.append(a + k * size)
        vs.append(b + k * size)
    for k in range(blocks):
        for l in range(k + 1, blocks):
            c = rng.binomial(size * size, p_out)
            us.append(rng.integers(0, size, c) + k * size)
            vs.append(rng.integers(0, size, c) + l * size)
    u = np.concatenate(us)
    v = np.concatenate(vs)
    n = blocks * size
    g = from_edges(n, u, v)
    if weighted:
        g = _reweight(g, rng)
    return g


def _reweight(g: CSRGraph, rng) -> CSRGraph:
    """Attach float32 U(0.5, 2) weights, one per undirected edge in (u<v) order."""
    rows = np.repeat(np.arange(g.n, dtype=np.int64), np.diff(g.rowptr))
    upper = rows < g.col
    u = rows[upper]
    v = g.col[upper].astype(np.int64)
    del rows, upper
    w = _weights(rng, u.size)
    return from_edges(g.n, u, v, w, sorted_unique=True)


def largest_component(g: CSRGraph) -> CSRGraph:
    """Induced subgraph on the largest connected component (node order kept)."""
    import scipy.sparse as sp
    from scipy.sparse.csgraph import connected_components

    A = sp.csr_matrix((np.ones(g.nnz, dtype=np.int8), g.col, g.rowptr), shape=(g.n, g.n))
    ncomp, label = connected_components(A, directed=False)
    if ncomp == 1:
        return g
    big = np.argmax(np.bincount(label))
    keep = label == big
    newid = np.full(g.n, -1, dtype=np.int64)
    newid[keep] = np.arange(int(keep.sum()))
    rows = np.repeat(np.arange(g.n, dtype=np.int64), np.diff(g.rowptr))
    upper = (rows < g.col) & keep[rows]
    u = newid[rows[upper]]
    v = newid[g.col[upper]]
    w = None if g.w is None else g.w[upper]
    return from_edges(int(keep.sum()), u, v, w, sorted_unique=True)


def component_count(g: CSRGraph) -> int:
    """Number of connected components (isolated nodes count as components)."""
    import scipy.sparse as sp
    from scipy.sparse.csgraph import connected_components

    A = sp.csr_matrix((np.ones(g.nnz, dtype=np.int8), g.col, g.rowptr), shape=(g.n, g.n))
    return int(connected_components(A, directed=False)[0])


def relabel(g: CSRGraph, perm) -> CSRGraph:
    """The same graph with node i renamed perm[i] (perm a permutation of 0..n-1); each
    stored entry keeps its weight, rows and their columns come out sorted."""
    perm = np.asarray(perm, dtype=np.int64)
    if perm.shape != (g.n,) or not np.array_equal(np.sort(perm), np.arange(g.n)):
        raise ValueError("perm must be a permutation of 0..n-1")
    rows = perm[np.repeat(np.arange(g.n, dtype=np.int64), np.diff(g.rowptr))]
    cols = perm[np.asarray(g.col, dtype=np.int64)]
    order = np.argsort(rows * g.n + cols, kind="stable")
    rowptr = np.zeros(g.n + 1, dtype=np.int64)
    np.cumsum(np.bincount(rows, minlength=g.n), out=rowptr[1:])
    col = cols[order].astype(np.int32)
    w = None if g.w is None else np.asarray(g.w)[order]
    return CSRGraph(g.n, rowptr, col, w)


def chung_lu(n: int, gamma: float, i0: float, m_target: int, seed: int,
             weighted: bool = False, keep_largest: bool = False,
             overdraw: float = 1.06, progress=None) -> CSRGraph:
    """Chung–Lu power-law graph with ``m_target`` distinct edges.

    Node i has weight (i + i0)^(-1/(gamma-1)).  Endpoints are drawn i.i.d. in
    proportion to the weights (a multinomial count per node, randomly permuted and
    paired), self-loops are dropped and repeats merged; more pairs are drawn until at
    least ``m_target`` distinct edges exist, and a uniformly random subset of exactly
    ``m_target`` of them is kept.  Node ids are in decreasing expected-degree order.
    ``progress`` (a callable taking a string) reports the stages of large draws.
    """
    say = progress or (lambda msg: None)
    rng = np.random.default_rng(seed)
    wt = (np.arange(n, dtype=np.float64) + i0) ** (-1.0 / (gamma - 1.0))
    prob = wt / wt.sum()
    keys = np.empty(0, dtype=np.int64)
    need = m_target
    rounds = 0
    while keys.size < m_target:
        draws = int(need * overdraw) + 1024
        ends = np.repeat(np.arange(n, dtype=np.int32), rng.multinomial(2 * draws, prob))
        rng.shuffle(ends)
        a = ends[0::2]
        b = ends[1::2]
        k = np.minimum(a, b).astype(np.int64)
        k *= n
        k += np.maximum(a, b)
        k = k[a != b]
        del ends, a, b
        keys = np.unique(np.concatenate([keys, k]))
        del k
        rounds += 1
        say(f"chung_lu: round {rounds}: {keys.size} distinct edges of {m_target}")
        need = max(1024, int((m_target - keys.size) * 1.5))
    if keys.size > m_target:
        r = rng.random(keys.size)
        sel = np.argpartition(r, m_target)[:m_target]
        del r
        sel.sort()
        keys = keys[sel]
        del sel
    u = keys // n
    v = keys % n
    del keys
    say("chung_lu: building CSR")
    if weighted and not keep_largest:
        # same draw as _reweight: one weight per edge in (u<v) order
        g = from_edges(n, u, v, _weights(rng, u.size), sorted_unique=True)
        del u, v
        return g
    g = from_edges(n, u, v, sorted_unique=True)
    del u, v
    if keep_largest:
        g = largest_component(g)
    if weighted:
        say("chung_lu: weights")
        g = _reweight(g, rng)
    return g

"""Canonical edges, oriented incidence matrix and Laplacian (Section 3.1.1).

The paper writes L = D - A = B^T W B with B an m x n oriented incidence matrix and
W = diag(w_e) of positive weights.  It does not fix the edge numbering or the
orientation; this oracle reads them as:

* edge e is the e-th pair (u, v), u < v, in lexicographic order;
* row e of B has +1 in column u and -1 in column v.

Effective resistance does not depend on either choice; the bits of Y = B^T W^{1/2} Q
do, which is why both are fixed here.
"""
from __future__ import annotations

import numpy as np
import scipy.sparse as sp


def check_graph(g) -> None:
    """Reject what the method is not defined for: asymmetry, self-loops, repeats, w <= 0."""
    n, rp, col = g.n, np.asarray(g.rowptr), np.asarray(g.col)
    if rp[0] != 0 or np.any(np.diff(rp) < 0):
        raise ValueError("row pointers must start at 0 and be non-decreasing")
    rows = np.repeat(np.arange(n), np.diff(rp))
    if col.size and (col.min() < 0 or col.max() >= n):
        raise ValueError("column index out of range")
    if np.any(rows == col):
        raise ValueError("self-loop")
    key = rows.astype(np.int64) * n + col
    if np.any(np.diff(key) <= 0):
        raise ValueError("columns must be strictly ascending in each row")
    tkey = col.astype(np.int64) * n + rows
    order = np.argsort(tkey)
    if not np.array_equal(tkey[order], key):
        raise ValueError("structure is not symmetric")
    if g.w is not None:
        w = np.asarray(g.w, dtype=np.float64)
        if not np.all(np.isfinite(w)) or np.any(w <= 0):
            raise ValueError("weights must be finite and positive")
        if not np.array_equal(w[order], w):
            raise ValueError("weights are not symmetric")


def entry_rows(g) -> np.ndarray:
    return np.repeat(np.arange(g.n, dtype=np.int64), np.diff(g.rowptr))


def canonical_edges(g):
    """Edge list (u < v, lexicographic) and the edge id of every stored CSR entry.

    Returns (eu, ev, eid) with eu, ev int64 arrays of length m and eid int64 of
    length nnz such that CSR entry (i, j) is edge (min(i,j), max(i,j)).
    """
    rows = entry_rows(g)
    col = np.asarray(g.col, dtype=np.int64)
    upper = rows < col
    eu = rows[upper]
    ev = col[upper]
    # keys of the edge list are strictly increasing by construction of a sorted CSR
    keys = eu * g.n + ev
    lo = np.minimum(rows, col)
    hi = np.maximum(rows, col)
    eid = np.searchsorted(keys, lo * g.n + hi)
    return eu, ev, eid


def edge_weights(g) -> np.ndarray:
    """w_e per canonical edge, as fp64 (unit when the graph is unweighted)."""
    rows = entry_rows(g)
    upper = rows < np.asarray(g.col)
    if g.w is None:
        return np.ones(int(upper.sum()), dtype=np.float64)
    return np.asarray(g.w, dtype=np.float64)[upper]


def incidence(g) -> sp.csr_matrix:
    """Oriented incidence matrix B (m x n): +1 at the smaller endpoint, -1 at the larger."""
    eu, ev, _ = canonical_edges(g)
    m = eu.size
    r = np.concatenate([np.arange(m), np.arange(m)])
    c = np.concatenate([eu, ev])
    v = np.concatenate([np.ones(m), -np.ones(m)])
    return sp.csr_matrix((v, (r, c)), shape=(m, g.n))


def laplacian(g) -> sp.csr_matrix:
    """L = B^T W B as an fp64 sparse matrix."""
    B = incidence(g)
    W = sp.diags(edge_weights(g))
    return (B.T @ W @ B).tocsr()


def dense_laplacian(g) -> np.ndarray:
    """L = D - A built directly from the adjacency (used to pin ``laplacian``)."""
    A = np.zeros((g.n, g.n))
    rows = entry_rows(g)
    w = np.ones(g.nnz) if g.w is None else np.asarray(g.w, dtype=np.float64)
    A[rows, np.asarray(g.col)] = w
    return np.diag(A.sum(axis=1)) - A


def components(g) -> int:
    from scipy.sparse.csgraph import connected_components

    A = sp.csr_matrix((np.ones(g.nnz), np.asarray(g.col), np.asarray(g.rowptr)),
                      shape=(g.n, g.n))
    return int(connected_components(A, directed=False)[0])

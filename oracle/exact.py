"""Exact references for small graphs, used to pin the oracle pipeline.

* ``pinv_resistance``: R_uv = b_uv^T L^+ b_uv with a dense Moore-Penrose
  pseudoinverse (Eq. 1).
* ``reg_resistance``: the diagonal-perturbation scheme of the authors' prior work
  (ERC-REG in Table 2): b^T (L + eps I)^{-1} b with a dense inverse.
* ``jl_dense_resistance``: the JL estimate of Eq. 6 with the same Q as the CG path
  but a dense direct solve of Eq. 5 (ERC-JL in Table 2).
* ``dense_rhs``: Y = B^T W^{1/2} Q as a plain matrix product (Section 3.1.2).
"""
from __future__ import annotations

import math

import numpy as np

from . import graph as GR
from . import hashing as H


def dense_Q(g, K: int, seed: int, col0: int = 0, ncols=None) -> np.ndarray:
    """Q[e, c] = sign(e, c) / sqrt(K), shape (m, ncols)."""
    ncols = K - col0 if ncols is None else ncols
    m = g.m
    return H.signs(seed, K, np.arange(m), np.arange(col0, col0 + ncols)) / math.sqrt(K)


def dense_rhs(g, K: int, seed: int, col0: int = 0, ncols=None) -> np.ndarray:
    B = GR.incidence(g).toarray()
    sw = np.sqrt(GR.edge_weights(g))
    return B.T @ (sw[:, None] * dense_Q(g, K, seed, col0, ncols))


def pinv_resistance(g) -> np.ndarray:
    L = GR.dense_laplacian(g)
    Lp = np.linalg.pinv(L, hermitian=True)
    eu, ev, _ = GR.canonical_edges(g)
    return Lp[eu, eu] + Lp[ev, ev] - 2.0 * Lp[eu, ev]


def reg_resistance(g, eps: float) -> np.ndarray:
    L = GR.dense_laplacian(g)
    M = np.linalg.inv(L + eps * np.eye(g.n))
    eu, ev, _ = GR.canonical_edges(g)
    return M[eu, eu] + M[ev, ev] - 2.0 * M[eu, ev]


def jl_dense_resistance(g, K: int, seed: int, delta: float) -> np.ndarray:
    L = GR.dense_laplacian(g)
    Y = dense_rhs(g, K, seed)
    Z = np.linalg.solve(L + delta * np.eye(g.n), Y)
    eu, ev, _ = GR.canonical_edges(g)
    d = Z[eu] - Z[ev]
    return np.einsum("ij,ij->i", d, d)

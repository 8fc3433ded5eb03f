"""The ERC-LG pipeline in plain fp64 (Section 3.1, Algorithm 1, Section 3.2).

Steps, in the paper's order:

1. Y = B^T W^{1/2} Q for a batch of columns of the projection Q (Section 3.1.2;
   Algorithm 1, forming Y^(t) from streamed Q^(t)).
2. Solve (L + eps*I) Z = Y column by column with CG to relative residual tau
   (Eq. 5; Section 3.1.3 "column-wise CG"; Algorithm 1).
3. R_e += ||Z_u - Z_v||^2 per edge (Eq. 6), accumulated over the column batches.
4. p_u = 1 - 1/2 sum_v w_uv R_uv and kappa_uv = 2 (p_u + p_v) / R_uv (Eq. 2).
5. Node weights (Eq. 7), edge weights (Eq. 8), each normalised by its sum
   (Section 3.2).

Readings where the paper is silent (each also listed in the design notes):
CG inner products are computed in twice the working precision (``accurate``);
CG starts from Z = 0 and stops on the recursively updated residual,
||r|| <= tau ||y|| per column; the sum in step 1 runs over each node's neighbours in
ascending order in fp64 and is rounded once to the working precision; a column whose
right-hand side is zero is converged at iteration 0; the JL scale is 1/sqrt(K) with
K the total projection dimension even when only a column range is solved.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

from . import graph as GR
from . import hashing as H
from .accurate import dot2_columns


def working_dtype(dtype: str):
    return {"f64": np.float64, "f32": np.float32}[dtype]


def rhs(g, K: int, col0: int, ncols: int, seed: int, dtype: str = "f64", rows=None,
        edges=None):
    """Y[i, c] = (1/sqrt(K)) * sum_{j in N(i)} B_{e(i,j), i} sqrt(w_e) sign(e, col0 + c).

    B_{e,i} is +1 when i is the smaller endpoint of e and -1 otherwise.  The sum over
    j runs in ascending neighbour order in fp64, then the product with 1/sqrt(K) is
    rounded once to the working precision.  ``rows`` restricts the output to a
    subset of nodes (in the given order); ``edges`` is ``canonical_edges(g)`` when the
    caller already holds it.
    """
    eu, ev, eid = GR.canonical_edges(g) if edges is None else edges
    sw = np.sqrt(GR.edge_weights(g))
    rp = np.asarray(g.rowptr)
    col = np.asarray(g.col, dtype=np.int64)
    rows = np.arange(g.n) if rows is None else np.asarray(rows, dtype=np.int64)
    cols = np.arange(col0, col0 + ncols, dtype=np.int64)
    start = rp[rows]
    deg = rp[rows + 1] - start
    acc = np.zeros((rows.size, ncols), dtype=np.float64)
    maxdeg = int(deg.max()) if rows.size else 0
    live = np.arange(rows.size)
    for t in range(maxdeg):
        live = live[deg[live] > t]
        pos = start[live] + t
        e = eid[pos]
        orient = np.where(rows[live] < col[pos], 1.0, -1.0)
        s = H.signs(seed, K, e, cols).astype(np.float64)
        acc[live] += (orient * sw[e])[:, None] * s
    inv_sqrt_k = 1.0 / math.sqrt(K)
    return (acc * inv_sqrt_k).astype(working_dtype(dtype))


def laplacian_apply(L, delta: float, X: np.ndarray) -> np.ndarray:
    """(L + delta I) X in fp64 (the matrix-free operator of Section 3.1.3)."""
    X = np.asarray(X, dtype=np.float64)
    return L @ X + delta * X


class CGBreakdown(RuntimeError):
    pass


@dataclass
class CGResult:
    Z: np.ndarray
    iters: np.ndarray
    converged: np.ndarray
    relres: np.ndarray


def cg_columns(L, delta: float, Y: np.ndarray, tol: float, max_iter: int) -> CGResult:
    """Independent Hestenes-Stiefel CG for every column of (L + delta I) Z = Y.

    Per column c: z = 0, r = y, p = r, rho = r.r.  Each iteration forms
    q = (L + delta I) p, alpha = rho / (p.q), z += alpha p, r -= alpha q,
    rho' = r.r; the column stops once rho' <= tol^2 * rho_0, else
    p = r + (rho'/rho) p.  A column with rho_0 = 0 is converged with z = 0.
    Inner products are evaluated in twice the working precision (``dot2_columns``).
    """
    Y = np.asarray(Y, dtype=np.float64)
    n, k = Y.shape
    Z = np.zeros((n, k))
    R = Y.copy()
    P = R.copy()
    rho = dot2_columns(R, R)
    rho0 = rho.copy()
    thr = tol * tol * rho0
    active = rho0 > 0
    iters = np.zeros(k, dtype=np.int64)
    for it in range(1, max_iter + 1):
        a = np.flatnonzero(active)
        if a.size == 0:
            break
        Pa = P[:, a]
        Qa = laplacian_apply(L, delta, Pa)
        pi = dot2_columns(Pa, Qa)
        if np.any(~np.isfinite(pi)) or np.any(pi <= 0):
            raise CGBreakdown(f"p.q <= 0 or non-finite at iteration {it}")
        alpha = rho[a] / pi
        Z[:, a] += alpha * Pa
        Ra = R[:, a] - alpha * Qa
        R[:, a] = Ra
        rho_new = dot2_columns(Ra, Ra)
        iters[a] = it
        done = rho_new <= thr[a]
        beta = rho_new / rho[a]
        keep = ~done
        P[:, a[keep]] = Ra[:, keep] + beta[keep] * Pa[:, keep]
        rho[a] = rho_new
        active[a[done]] = False
    relres = np.sqrt(np.divide(rho, rho0, out=np.zeros(k), where=rho0 > 0))
    return CGResult(Z, iters, ~active, relres)


def jacobi_inverse(L, delta: float) -> np.ndarray:
    """m_i = 1 / (L_ii + delta): the inverse diagonal of L + delta I, in fp64."""
    return 1.0 / (np.asarray(L.diagonal(), dtype=np.float64) + delta)


def pcg_columns(L, delta: float, Y: np.ndarray, tol: float, max_iter: int) -> CGResult:
    """Jacobi-preconditioned CG for every column of (L + delta I) Z = Y.

    A variant the paper does not use: textbook preconditioned CG (Saad, Iterative
    Methods for Sparse Linear Systems, 2nd ed., Algorithm 9.1) with M^-1 = diag(m),
    m_i = 1 / (L_ii + delta).  Per column c: z = 0, r = y, s = m * r, p = s,
    rho = r.s.  Each iteration forms q = (L + delta I) p, alpha = rho / (p.q),
    z += alpha p, r -= alpha q; the column stops once r.r <= tol^2 y.y (the stopping
    test of plain CG), else s = m * r, rho' = r.s and p = s + (rho'/rho) p.  Inner
    products in twice the working precision, as for plain CG.
    """
    Y = np.asarray(Y, dtype=np.float64)
    n, k = Y.shape
    m = jacobi_inverse(L, delta)[:, None]
    Z = np.zeros((n, k))
    R = Y.copy()
    S = m * R
    P = S.copy()
    rho = dot2_columns(R, S)
    rr0 = dot2_columns(R, R)
    rr = rr0.copy()
    thr = tol * tol * rr0
    active = rr0 > 0
    iters = np.zeros(k, dtype=np.int64)
    for it in range(1, max_iter + 1):
        a = np.flatnonzero(active)
        if a.size == 0:
            break
        Pa = P[:, a]
        Qa = laplacian_apply(L, delta, Pa)
        pi = dot2_columns(Pa, Qa)
        if np.any(~np.isfinite(pi)) or np.any(pi <= 0):
            raise CGBreakdown(f"p.q <= 0 or non-finite at iteration {it}")
        alpha = rho[a] / pi
        Z[:, a] += alpha * Pa
        Ra = R[:, a] - alpha * Qa
        R[:, a] = Ra
        rr[a] = dot2_columns(Ra, Ra)
        iters[a] = it
        done = rr[a] <= thr[a]
        Sa = m * Ra
        rho_new = dot2_columns(Ra, Sa)
        beta = rho_new / rho[a]
        keep = ~done
        P[:, a[keep]] = Sa[:, keep] + beta[keep] * Pa[:, keep]
        rho[a] = rho_new
        active[a[done]] = False
    relres = np.sqrt(np.divide(rr, rr0, out=np.zeros(k), where=rr0 > 0))
    return CGResult(Z, iters, ~active, relres)


def edge_distances(Z: np.ndarray, eu: np.ndarray, ev: np.ndarray, chunk: int = 1 << 20):
    """sum_c (Z[u, c] - Z[v, c])^2 per edge, subtracting and summing in fp64 (Eq. 6)."""
    Z = np.asarray(Z, dtype=np.float64)
    out = np.empty(eu.size)
    for s in range(0, eu.size, chunk):
        d = Z[eu[s:s + chunk]] - Z[ev[s:s + chunk]]
        out[s:s + chunk] = np.einsum("ij,ij->i", d, d)
    return out


@dataclass
class ResistanceInfo:
    iters: list = field(default_factory=list)        # per block: per-column iteration counts
    converged: list = field(default_factory=list)    # per block: per-column flags
    relres: list = field(default_factory=list)


def resistance(g, K: int, k_block: int, delta: float, tol: float, max_iter: int, seed: int,
               dtype: str = "f64", col_begin: int = 0, col_end=None, L=None,
               precond: str = "none", edges=None):
    """R_hat over columns [col_begin, col_end) of the K-column sketch (Algorithm 1).

    Columns are processed in batches of at most ``k_block``; each batch forms Y,
    runs CG (or, with precond="jacobi", the Jacobi-preconditioned variant) and adds
    its squared edge distances to R before the next batch starts.  A caller that
    passes the Laplacian ``L`` (and optionally ``canonical_edges(g)`` as ``edges``)
    has validated the graph already; otherwise it is validated here.
    """
    solve = {"none": cg_columns, "jacobi": pcg_columns}[precond]
    col_end = K if col_end is None else col_end
    if L is None:
        GR.check_graph(g)
        L = GR.laplacian(g)
    edges = GR.canonical_edges(g) if edges is None else edges
    eu, ev, _ = edges
    R = np.zeros(eu.size)
    info = ResistanceInfo()
    for c0 in range(col_begin, col_end, k_block):
        nc = min(k_block, col_end - c0)
        Y = rhs(g, K, c0, nc, seed, dtype, edges=edges)
        res = solve(L, delta, Y, tol, max_iter)
        R += edge_distances(res.Z, eu, ev)
        info.iters.append(res.iters)
        info.converged.append(res.converged)
        info.relres.append(res.relres)
    return R, info


def curvature(g, R: np.ndarray):
    """Node curvature p and edge curvature kappa from per-edge resistances (Eq. 2).

    p_u = 1 - 1/2 sum_{v in N(u)} w_uv R_uv (an isolated node has p = 1);
    kappa_uv = 2 (p_u + p_v) / R_uv.
    """
    eu, ev, eid = GR.canonical_edges(g)
    rows = GR.entry_rows(g)
    w = np.ones(g.nnz) if g.w is None else np.asarray(g.w, dtype=np.float64)
    s = np.bincount(rows, weights=w * R[eid], minlength=g.n)
    p = 1.0 - 0.5 * s
    kappa = 2.0 * (p[eu] + p[ev]) / R
    return p, kappa


def sampling_probs(g, kappa: np.ndarray, eta: float):
    """Node and edge sampling probabilities (Eqs. 7 and 8, normalised by their sums).

    q_u = sum_{v in N(u)} (kappa_uv - kappa_min) / (kappa_max - kappa_min + eta); if
    every q_u is zero the node distribution is uniform over nodes with degree > 0.
    q_uv = sqrt(max(2 kappa_max - kappa_uv, 0)) + 1.
    """
    _, _, eid = GR.canonical_edges(g)
    rows = GR.entry_rows(g)
    kmin = float(np.min(kappa)) if kappa.size else 0.0
    kmax = float(np.max(kappa)) if kappa.size else 0.0
    qn = np.bincount(rows, weights=(kappa[eid] - kmin) / (kmax - kmin + eta), minlength=g.n)
    tot = qn.sum()
    if tot == 0.0:
        qn = (np.diff(g.rowptr) > 0).astype(np.float64)
        tot = qn.sum()
    pn = qn / tot if tot > 0 else qn
    qe = np.sqrt(np.maximum(2.0 * kmax - kappa, 0.0)) + 1.0
    pe = qe / qe.sum() if qe.size else qe
    return pn, pe


@dataclass
class RunResult:
    R: np.ndarray
    p: np.ndarray
    kappa: np.ndarray
    node_prob: np.ndarray
    edge_prob: np.ndarray
    info: ResistanceInfo


def run(g, params) -> RunResult:
    """The whole path for one workload: resistance, curvature, sampling probabilities."""
    R, info = resistance(g, params.K, params.k_block, params.delta, params.tol,
                         params.max_iter, params.seed, params.dtype)
    p, kappa = curvature(g, R)
    pn, pe = sampling_probs(g, kappa, params.eta)
    return RunResult(R, p, kappa, pn, pe, info)

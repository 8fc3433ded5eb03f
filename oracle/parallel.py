"""Column-parallel driver of the oracle for the large workloads (test infrastructure).

The K right-hand sides of Algorithm 1 are independent, so a column range can be split
into contiguous sub-ranges solved by separate processes with the unchanged oracle
(each column's arithmetic is the same as in a serial run).  The per-range edge sums
are then added in range order, which equals the serial result up to the
reassociation of that final fp64 sum.
"""
from __future__ import annotations

import multiprocessing as mp
import os
import tempfile
import time

import numpy as np

from . import erc
from . import graph as GR

_G = None
_L = None
_E = None


def _work(args):
    c0, c1, prm, path = args
    t0 = time.time()
    R, info = erc.resistance(_G, prm["K"], prm["k_block"], prm["delta"], prm["tol"],
                             prm["max_iter"], prm["seed"], prm["dtype"], c0, c1, L=_L,
                             precond=prm["precond"], edges=_E)
    iters = np.concatenate(info.iters) if info.iters else np.zeros(0, np.int64)
    conv = np.concatenate(info.converged) if info.converged else np.zeros(0, bool)
    np.savez(path, R=R, iters=iters, conv=conv, seconds=time.time() - t0)
    return c0, c1, iters, conv


def solve_chunks(g, chunks, paths, K, k_block, delta, tol, max_iter, seed, dtype="f64",
                 procs=None, progress=None, precond="none"):
    """Solve each column range chunks[i] = (c0, c1) in a pool of ``procs`` processes and
    write its R, iteration counts and convergence flags to paths[i] (``.npz``).

    Chunks are independent and may come from several disjoint ranges; each file holds
    exactly what ``erc.resistance`` returns for that range alone.
    """
    global _G, _L, _E
    assert len(chunks) == len(paths)
    if not chunks:
        return
    GR.check_graph(g)
    _G = g
    _L = GR.laplacian(g)
    # built once here and shared with the forked workers, which then hold only their
    # columns' vectors
    _E = GR.canonical_edges(g)
    prm = dict(K=K, k_block=k_block, delta=delta, tol=tol, max_iter=max_iter, seed=seed,
               dtype=dtype, precond=precond)
    jobs = [(c0, c1, prm, path) for (c0, c1), path in zip(chunks, paths)]
    procs = max(1, min(procs or min(8, os.cpu_count() or 1), len(jobs)))
    try:
        ctx = mp.get_context("fork")
        with ctx.Pool(procs) as pool:
            for res in pool.imap_unordered(_work, jobs):
                if progress:
                    progress(f"oracle columns [{res[0]}, {res[1]}) done")
    finally:
        _G = None
        _L = None
        _E = None


def resistance_parallel(g, K, k_block, delta, tol, max_iter, seed, dtype="f64", col_begin=0,
                        col_end=None, procs=None, progress=None, precond="none"):
    """R over columns [col_begin, col_end), solved in `procs` column ranges.

    Returns (R, iters, converged) with per-column iteration counts and flags in column
    order.
    """
    col_end = K if col_end is None else col_end
    procs = procs or min(8, os.cpu_count() or 1)
    ncol = col_end - col_begin
    procs = max(1, min(procs, ncol))
    bounds = [col_begin + (ncol * k) // procs for k in range(procs + 1)]
    chunks = [(bounds[k], bounds[k + 1]) for k in range(procs)]
    with tempfile.TemporaryDirectory(prefix="erc_oracle_") as tmp:
        paths = [os.path.join(tmp, f"R{k}.npz") for k in range(procs)]
        solve_chunks(g, chunks, paths, K, k_block, delta, tol, max_iter, seed, dtype,
                     procs=procs, progress=progress, precond=precond)
        R = np.zeros(g.m)
        iters, conv = [], []
        for path in paths:
            with np.load(path) as f:
                R += f["R"]
                iters.append(f["iters"])
                conv.append(f["conv"])
    return R, np.concatenate(iters), np.concatenate(conv)

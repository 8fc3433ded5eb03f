"""How far two CG solves that differ only in rounding land apart, edge by edge.

    python tests/golden/make_rounding_spread.py

The power-law workloads have hub-hub edges whose resistance lies hundreds of times
below the typical edge's (two hubs share most of their neighbours).  Eq. 6 forms R_e as
the squared difference of two nearly equal rows of Z, so a perturbation of the iterate
that is small next to |Z| is large next to R_e there.  This script measures that on a
graph built like the 2.4M-node workload at 1/25 of its size (same exponent and weights,
n = 96,000): it solves the first 8 columns of the same projection with the oracle's CG
(fp64 vectors, inner products in twice fp64) and with CG variants that change only the
rounding of the same recurrence:

* "fp64, plain inner products": fp64 vectors, inner products summed in fp64;
* "fp32 vectors, fp64 inner products": the arithmetic of the fp32 path (iterate,
  residual and direction stored in fp32, the operator and the inner products in fp64).

For each it reports the difference in R from the oracle's, as a plain relative error and
over max(R_e, sqrt(R_e Rbar)) (Rbar the mean R), over all edges and over the hub-hub
edges (both endpoints among the 0.5 % highest degrees).  Writes
tests/golden/rounding_spread.json.  Calls the oracle and numpy only.
"""
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import gen  # noqa: E402
from oracle import erc as OE  # noqa: E402
from oracle import graph as OG  # noqa: E402

NAME = "cl2400k"
SHRINK = 25
COLUMNS = 8
OUT = os.path.join(HERE, "rounding_spread.json")


def variant_cg(L, delta, Y, tol, max_iter, vec_dtype, dot):
    """The CG of Algorithm 1 as the oracle runs it (z = 0, stop on the recursive
    residual), with the vectors stored in ``vec_dtype`` and inner products ``dot``."""
    f64 = np.float64
    n, k = Y.shape
    z = np.zeros((n, k), vec_dtype)
    r = Y.astype(vec_dtype)
    p = r.copy()
    rho = dot(r, r)
    thr = tol * tol * rho
    active = rho > 0
    iters = np.zeros(k, np.int64)
    for it in range(1, max_iter + 1):
        if not active.any():
            break
        p64 = p.astype(f64)
        q = np.asarray(L @ p64) + delta * p64
        pq = dot(p64, q)
        alpha = np.where(active, rho / np.where(active, pq, 1.0), 0.0)
        z = (z.astype(f64) + alpha * p64).astype(vec_dtype)
        r = (r.astype(f64) - alpha * q).astype(vec_dtype)
        rr = dot(r, r)
        iters[active] = it
        done = active & (rr <= thr)
        go = active & ~done
        beta = np.where(go, rr / np.where(active, rho, 1.0), 0.0)
        newp = (r.astype(f64) + beta * p.astype(f64)).astype(vec_dtype)
        p = np.where(go[None, :], newp, p)
        rho = np.where(active, rr, rho)
        active = go
    return z.astype(f64), iters


def plain_dot(a, b):
    return np.einsum("ij,ij->j", a.astype(np.float64), b.astype(np.float64))


def accurate_dot(a, b):
    from oracle.accurate import dot2_columns
    return dot2_columns(a.astype(np.float64), b.astype(np.float64))


def spread(R, R0, mask):
    rel = np.abs(R - R0) / R0
    scaled = np.abs(R - R0) / np.maximum(R0, np.sqrt(R0 * R0.mean()))

    def q(x):
        x = np.sort(x)
        return {"max": float(x[-1]), "p99.9": float(x[int(0.999 * (x.size - 1))]),
                "median": float(x[x.size // 2])}
    return {"R_rel": q(rel), "R_scaled": q(scaled), "hub_hub_R_rel": q(rel[mask]),
            "hub_hub_R_scaled": q(scaled[mask])}


def main():
    wl = gen.CONFIGS[NAME]
    p = wl.params
    args = dict(wl.graph_args)
    args.update(n=args["n"] // SHRINK, m_target=args["m_target"] // SHRINK,
                i0=args["i0"] / SHRINK)
    g = gen.graphs.chung_lu(**args)
    L = OG.laplacian(g).tocsr()
    eu, ev, _ = OG.canonical_edges(g)
    deg = np.diff(np.asarray(g.rowptr))
    hub = deg >= np.quantile(deg, 0.995)
    hub_hub = hub[eu] & hub[ev]
    Y = OE.rhs(g, p.K, 0, COLUMNS, p.seed, p.dtype)
    t0 = time.time()
    base = OE.cg_columns(L, p.delta, Y, p.tol, p.max_iter)
    R0 = OE.edge_distances(base.Z, eu, ev)
    out = {"workload": f"{NAME} generator at 1/{SHRINK}", "graph": g.summary(),
           "columns": [0, COLUMNS], "K": p.K, "delta": p.delta, "tol": p.tol,
           "hub_degree_min": int(deg[hub].min()), "hub_hub_edges": int(hub_hub.sum()),
           "R_median": float(np.median(R0)), "R_mean": float(R0.mean()),
           "hub_hub_R_median": float(np.median(R0[hub_hub])),
           "oracle_iters": [int(base.iters.min()), int(base.iters.max())], "variants": {}}
    for label, dt, dot in (("fp64, plain inner products", np.float64, plain_dot),
                           ("fp32 vectors, fp64 inner products", np.float32, accurate_dot)):
        Z, it = variant_cg(L, p.delta, Y, p.tol, p.max_iter, dt, dot)
        res = spread(OE.edge_distances(Z, eu, ev), R0, hub_hub)
        res["iters"] = [int(it.min()), int(it.max())]
        out["variants"][label] = res
        print(label, json.dumps(res), flush=True)
    out["seconds"] = round(time.time() - t0, 1)
    with open(OUT, "w") as f:
        json.dump(out, f, indent=1, sort_keys=True)
        f.write("\n")


if __name__ == "__main__":
    main()

"""The oracle's own truncation floor per workload: R from the CG stopped at the
workload's tolerance tau against R from the same CG run on to tau = 1e-11.

    python tests/golden/make_floor.py [er2k sbm20k cl170k cl230k cl2400k]

Both runs use the oracle only (same graph, sketch, shift and right-hand sides; the CG
of Algorithm 1 stopped on the relative residual), so their difference is what stopping
at tau costs by itself, before any GPU rounding enters: a GPU result can not be
expected to agree with the oracle much more closely than this.  The small workloads
are solved over their whole projection; the large ones over a leading column range
(COLUMNS), with the column chunks cached as in make_golden.py (the tau chunks are the
ones the stored parity values were built from).  R's relative difference does not
depend on how many columns are summed; p and kappa are reported only where the whole
projection is solved; R (again), p and kappa are also reported on the condition scales
of the parity tests.

Writes tests/golden/truncation_floor.json (one entry per workload).  With
ERC_FLOOR_PART=tau or =tight only that tolerance's column chunks are solved and cached
(two such runs can go side by side); a run without it then reads both from the cache.
"""
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)
sys.path.insert(0, HERE)

import gen  # noqa: E402
import make_golden as MG  # noqa: E402
from oracle import erc as OE  # noqa: E402
from oracle import graph as OG  # noqa: E402

TIGHT = 1e-11
# leading column range solved on the workloads whose whole projection is too long
COLUMNS = {"cl170k": 16, "cl230k": 8, "cl2400k": 4}
OUT = os.path.join(HERE, "truncation_floor.json")


def quantiles(x):
    x = np.sort(np.asarray(x, np.float64))
    return {"max": float(x[-1]), "p99.9": float(x[int(0.999 * (x.size - 1))]),
            "median": float(x[x.size // 2])}


def floor(name, procs):
    p = gen.CONFIGS[name].params
    g = gen.make_graph(name, progress=MG.log)
    ncols = COLUMNS.get(name, p.K)
    rng = (0, ncols)
    t0 = time.time()
    part = os.environ.get("ERC_FLOOR_PART", "")
    if part == "tau":  # solve (or find cached) only the chunks at the workload's tolerance
        MG.solve_ranges(g, name, name, [rng], "none", procs)
        return None
    if part == "tight":  # only the chunks at the tight tolerance
        MG.solve_ranges(g, name, f"{name}_tight", [rng], "none", procs, tol=TIGHT)
        return None
    (_, _, _, R, it, conv, _), = MG.solve_ranges(g, name, name, [rng], "none", procs)
    (_, _, _, Rt, itt, convt, _), = MG.solve_ranges(g, name, f"{name}_tight", [rng], "none",
                                                    procs, tol=TIGHT)
    rel = np.abs(R - Rt) / Rt
    # the same difference over max(R_e, sqrt(R_e Rbar)), Rbar the mean R (the R scale of
    # the parity tests)
    scaled = np.abs(R - Rt) / np.maximum(Rt, np.sqrt(Rt * Rt.mean()))
    out = {"workload": name, "graph": g.summary(), "columns": list(rng), "K": p.K,
           "tol": p.tol, "tight_tol": TIGHT, "dtype_rhs": p.dtype,
           "iters": [int(it.min()), int(it.max())], "iters_tight": [int(itt.min()), int(itt.max())],
           "converged": bool(conv.all() and convt.all()), "R_rel": quantiles(rel),
           "R_scaled": quantiles(scaled),
           "seconds": round(time.time() - t0, 1)}
    if ncols == p.K:
        eu, ev, eid = OG.canonical_edges(g)
        rows = OG.entry_rows(g)
        w = np.ones(g.nnz) if g.w is None else np.asarray(g.w, np.float64)
        s = 0.5 * np.bincount(rows, weights=w * Rt[eid], minlength=g.n)
        pp, kk = OE.curvature(g, R)
        pt, kt = OE.curvature(g, Rt)
        live = s > 0
        out["p_scaled"] = quantiles(np.abs(pp - pt)[live] / s[live])
        out["kappa_scaled"] = quantiles(np.abs(kk - kt) / (2.0 * (s[eu] + s[ev]) / Rt + np.abs(kt)))
    MG.log(f"{name}: floor {out}")
    return out


def main():
    procs = int(os.environ.get("ERC_ORACLE_PROCS", "8"))
    names = sys.argv[1:] or gen.configs.ORDER
    table = {}
    if os.path.exists(OUT):
        with open(OUT) as f:
            table = json.load(f)
    for name in names:
        res = floor(name, procs)
        if res is None:  # ERC_FLOOR_PART: one tolerance's chunks only, nothing to write
            continue
        table[name] = res
        with open(OUT, "w") as f:
            json.dump(table, f, indent=1, sort_keys=True)
            f.write("\n")


if __name__ == "__main__":
    main()

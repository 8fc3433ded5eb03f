"""Write the stored oracle values used by the large-workload parity tests.

    python tests/golden/make_golden.py cl170k [cl230k cl2400k cl2400k:jacobi cl170k:relabel ...]

Each run regenerates the seeded graph, runs the CPU oracle (column-parallel, see
oracle/parallel.py) over the workload's full projection, or over each column range
named in RANGES, then computes curvature and sampling probabilities from that R and
stores the values at seeded samples of edges and nodes in tests/golden/<name>.npz
(the first range) and tests/golden/<name>_c<begin>.npz (each further range).
A name with the suffix ":jacobi" solves with the oracle's Jacobi-preconditioned CG
instead and writes tests/golden/<name>_jacobi.npz; the suffix ":relabel" solves on a
copy of the graph with node ids randomly permuted (RELABEL_SEED) and writes
tests/golden/<name>_relabel.npz.
Only gen/ and oracle/ are used; nothing here touches the GPU library.  The oracle
solves columns in chunks of at most CHUNK columns, one process each, and caches every
chunk's R under $TMPDIR; a range's R is the sum of its chunks in column order, so
ranges sharing columns reuse them and stored fields can be recomputed without a solve.

The samples: SAMPLES seeded random edges and nodes, the two extreme-curvature edges,
and, so that the work paths of long rows (split over a block's waves or over several
blocks) are always checked, the NHUB highest-degree nodes and up to HUB_EDGES seeded
edges at each of them.

Besides the values, each file stores, per sampled entry, the first-order error bound
that a relative error `RTOL` in every edge curvature (measured on the condition scale
2 (s_u + s_v) / R + |kappa|, s_u = 1/2 sum_v w_uv R_uv) induces in the sampling
probabilities of Eqs. 7-8 and their normalisation:
  node:  b_u = RTOL [sum_v (S_uv + S_x) + 2 q_u S_x] / D,  |dP_u| <= (b_u + P_u sum b) / Q
  edge:  a_e = RTOL (2 S_x + S_e),  b_e = sqrt(x_e + a_e) - sqrt(max(x_e - a_e, 0)),
         |dP_e| <= (b_e + P_e sum b) / Q_e
with S the kappa scale, S_x the larger scale of the two extreme edges, D = kappa_max -
kappa_min + eta and x_e = 2 kappa_max - kappa_e.
"""
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import gen  # noqa: E402
from oracle import erc as OE  # noqa: E402
from oracle import graph as OG  # noqa: E402
from oracle.parallel import solve_chunks  # noqa: E402

# column ranges for workloads whose full sketch is too long for the CPU oracle: on the
# 2.4M-node graph one column-iteration of the fp64 oracle takes seconds and a column
# needs ~480 iterations, so the stored ranges are the first two 64-column blocks (sign
# words 0 and 1 of the hash), the last 16 columns (sign word 3, the fourth block) and
# the first 16 of the third block (sign word 2), all in the launch configuration of the
# benchmark (64-column blocks)
RANGES = {"cl2400k": [(0, 64), (240, 256), (64, 128), (128, 144)]}
# the Jacobi-preconditioned variant keeps its stored range
RANGES_JACOBI = {"cl2400k": [(0, 16)]}
# ":relabel" runs the workload on a copy with node ids permuted by RELABEL_SEED (no
# hub-first order), over these column ranges
RANGES_RELABEL = {"cl170k": [(0, 8)], "cl2400k": [(0, 8)]}
RELABEL_SEED = 7
# columns per oracle process (ERC_ORACLE_CHUNK overrides it: 11 put the 2.4M-node
# graph's first 80 stored columns on eight processes at once; its other two ranges were
# solved later in 8-column chunks on four)
CHUNK = int(os.environ.get("ERC_ORACLE_CHUNK", "8"))
SAMPLES = 8192
NHUB = 256
HUB_EDGES = 128
RTOL = 1e-4
ORACLE_VERSION = 2  # bump when the oracle's arithmetic changes


def log(msg):
    print(f"[golden] {msg}", flush=True)


def cache_dir():
    d = os.path.join(os.environ.get("TMPDIR", "/tmp"), "erc_golden_cache")
    os.makedirs(d, exist_ok=True)
    return d


def chunk_path(tag, c0, c1):
    return os.path.join(cache_dir(), f"{tag}_c{c0}-{c1}_v{ORACLE_VERSION}.npz")


def cached_chunks(tag):
    pat = re.compile(re.escape(tag) + r"_c(\d+)-(\d+)_v" + str(ORACLE_VERSION) + r"\.npz$")
    out = []
    for fn in os.listdir(cache_dir()):
        mt = pat.match(fn)
        if mt:
            out.append((int(mt.group(1)), int(mt.group(2))))
    return sorted(out)


def plan_chunks(tag, c0, c1):
    """Disjoint chunks covering [c0, c1): cached ones where they fit, new ones of at
    most CHUNK columns in the gaps.  Returns (chunks, is_new flags)."""
    chunks, new = [], []
    pos = c0
    for a, b in cached_chunks(tag) + [(c1, c1)]:
        if a < pos or b > c1:
            continue
        while pos < a:
            e = min(a, pos + CHUNK)
            chunks.append((pos, e))
            new.append(True)
            pos = e
        if a < b:
            chunks.append((a, b))
            new.append(False)
            pos = b
    return chunks, new


def sampling_bounds(g, R, kappa, s, node_prob, edge_prob, eta):
    eu, ev, eid = OG.canonical_edges(g)
    rows = OG.entry_rows(g)
    S = 2.0 * (s[eu] + s[ev]) / R + np.abs(kappa)
    kmin, kmax = float(kappa.min()), float(kappa.max())
    Sx = max(S[np.argmin(kappa)], S[np.argmax(kappa)])
    D = kmax - kmin + eta
    qn = np.bincount(rows, weights=(kappa[eid] - kmin) / D, minlength=g.n)
    bn = RTOL * (np.bincount(rows, weights=S[eid] + Sx, minlength=g.n) + 2.0 * qn * Sx) / D
    Q = qn.sum()
    bound_node = (bn + node_prob * bn.sum()) / Q
    x = 2.0 * kmax - kappa
    a = RTOL * (2.0 * Sx + S)
    be = np.sqrt(x + a) - np.sqrt(np.maximum(x - a, 0.0))
    qe = np.sqrt(np.maximum(x, 0.0)) + 1.0
    bound_edge = (be + edge_prob * be.sum()) / qe.sum()
    return S, bound_node, bound_edge, kmin, kmax


def hub_samples(g, rng):
    """Nodes: the NHUB highest-degree rows (ties by id).  Edges: up to HUB_EDGES
    seeded edges of each of them, as canonical edge ids."""
    _, _, eid = OG.canonical_edges(g)
    deg = np.diff(np.asarray(g.rowptr))
    hubs = np.sort(np.argsort(-deg, kind="stable")[:min(NHUB, g.n)])
    edges = []
    for u in hubs:
        lo, hi = int(g.rowptr[u]), int(g.rowptr[u + 1])
        pos = np.arange(lo, hi)
        if pos.size > HUB_EDGES:
            pos = np.sort(rng.choice(pos, size=HUB_EDGES, replace=False))
        edges.append(eid[pos])
    edges = np.concatenate(edges) if edges else np.zeros(0, np.int64)
    return hubs, edges


def solve_ranges(g, name, tag, ranges, precond, procs, tol=None):
    """R, iterations and flags per range, from cached or newly solved chunks (at the
    workload's tolerance, or at `tol`; the tag must then name that tolerance)."""
    p = gen.CONFIGS[name].params
    tol = p.tol if tol is None else tol
    plans = [plan_chunks(tag, c0, c1) for c0, c1 in ranges]
    todo = sorted({c for chunks, new in plans for c, fresh in zip(chunks, new) if fresh})
    if todo:
        log(f"{name}: solving chunks {todo} on {procs} processes")
        t0 = time.time()
        solve_chunks(g, todo, [chunk_path(tag, a, b) for a, b in todo], p.K, p.k_block,
                     p.delta, tol, p.max_iter, p.seed, p.dtype, procs=procs,
                     progress=log, precond=precond)
        log(f"{name}: chunks solved in {time.time() - t0:.0f}s")
    out = []
    for (c0, c1), (chunks, _) in zip(ranges, plans):
        R = np.zeros(g.m)
        iters, conv, secs = [], [], 0.0
        for a, b in chunks:
            with np.load(chunk_path(tag, a, b)) as f:
                R += f["R"]
                iters.append(f["iters"])
                conv.append(f["conv"])
                secs += float(f["seconds"]) if "seconds" in f else float(f.get("t_solve", 0.0))
        out.append((c0, c1, chunks, R, np.concatenate(iters), np.concatenate(conv), secs))
    return out


def make(spec, procs):
    name, _, variant = spec.partition(":")
    variant = variant or "none"
    precond = "jacobi" if variant == "jacobi" else "none"
    tag = name if variant == "none" else f"{name}_{variant}"
    wl = gen.CONFIGS[name]
    p = wl.params
    t0 = time.time()
    g = gen.make_graph(name, progress=log)
    relabel_seed = None
    if variant == "relabel":
        relabel_seed = RELABEL_SEED
        g = gen.relabel(g, np.random.default_rng(RELABEL_SEED).permutation(g.n))
    log(f"{tag}: graph {g.summary()} ({time.time() - t0:.0f}s)")
    table = {"none": RANGES, "jacobi": RANGES_JACOBI, "relabel": RANGES_RELABEL}[variant]
    ranges = table.get(name, [(0, p.K)])
    eu, ev, eid = OG.canonical_edges(g)
    rows = OG.entry_rows(g)
    w = np.ones(g.nnz) if g.w is None else np.asarray(g.w, np.float64)
    ncomp = OG.components(g)
    for k, (c0, c1, chunks, R, iters, conv, t_solve) in enumerate(
            solve_ranges(g, name, tag, ranges, precond, procs)):
        log(f"{name}: resistance over columns [{c0}, {c1}) from chunks {chunks}, "
            f"iters {iters.min()}..{iters.max()}, all converged {bool(conv.all())}")
        pn_p, kappa = OE.curvature(g, R)
        node_prob, edge_prob = OE.sampling_probs(g, kappa, p.eta)
        s = 0.5 * np.bincount(rows, weights=w * R[eid], minlength=g.n)
        S, bound_node, bound_edge, kmin, kmax = sampling_bounds(g, R, kappa, s, node_prob,
                                                                edge_prob, p.eta)
        rng = np.random.default_rng(12345)
        es = np.sort(rng.choice(g.m, size=min(SAMPLES, g.m), replace=False))
        ns = np.sort(rng.choice(g.n, size=min(SAMPLES, g.n), replace=False))
        hubs, hub_edges = hub_samples(g, np.random.default_rng(54321))
        # the extreme-curvature edges and the hub rows are always in the sample
        es = np.unique(np.concatenate([es, [np.argmin(kappa), np.argmax(kappa)], hub_edges]))
        ns = np.unique(np.concatenate([ns, hubs]))
        meta = {"workload": name, "graph": g.summary(), "col_begin": c0, "col_end": c1,
                "K": p.K, "k_block": p.k_block, "delta": p.delta, "tol": p.tol,
                "seed": p.seed, "dtype": p.dtype, "eta": p.eta,
                "oracle_version": ORACLE_VERSION, "rtol": RTOL, "precond": precond,
                "relabel_seed": relabel_seed,
                "chunks": chunks, "solve_process_seconds": round(t_solve, 1),
                "iters_min": int(iters.min()), "iters_max": int(iters.max()),
                "iters_total": int(iters.sum()), "converged": bool(conv.all()),
                "kappa_min": kmin, "kappa_max": kmax, "components": ncomp,
                "hub_nodes": int(hubs.size), "hub_edges": int(np.unique(hub_edges).size),
                "hub_degree_min": int(np.diff(np.asarray(g.rowptr))[hubs].min())}
        suffix = "" if k == 0 else f"_c{c0}"
        out = os.path.join(os.path.dirname(os.path.abspath(__file__)), f"{tag}{suffix}.npz")
        np.savez_compressed(
            out, meta=np.array(json.dumps(meta)), edge_idx=es, node_idx=ns,
            R=R[es], kappa=kappa[es], kappa_scale=S[es], edge_prob=edge_prob[es],
            edge_prob_bound=bound_edge[es], p=pn_p[ns], s_node=s[ns],
            node_prob=node_prob[ns], node_prob_bound=bound_node[ns], iters=iters,
            sum_wR=np.float64(np.sum(OG.edge_weights(g) * R)), sum_p=np.float64(pn_p.sum()))
        log(f"wrote {out}")


if __name__ == "__main__":
    procs = int(os.environ.get("ERC_ORACLE_PROCS", "8"))
    for name in sys.argv[1:]:
        make(name, procs)
